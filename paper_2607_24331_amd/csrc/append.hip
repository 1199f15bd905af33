// Latent write for new tokens: z = x [L_keys | L_value] (Sec. III-A write
// side; per-group L_g of Sec. III-C; whole-projection L_v of Sec. III-D),
// accumulated in fp32, rounded to nearest-even into the paged pool.
//
// Output column space of one token: [0, R_Kp + r_v)
//   c <  R_K          key column c           -> page key row, column c
//   R_K <= c < R_Kp   key-row padding         -> written as zero
//   c >= R_Kp         value column c - R_Kp   -> page value part, rank-major
#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

constexpr int kTileTok = 64;
constexpr int kTileCol = 64;
constexpr int kTileK = 16;

// Portable VALU kernel (fp32 latents, and bf16 when the MFMA path does not
// apply): 64 tokens x 64 columns per 256-thread block, 4x4 outputs a thread.
template <typename T>
__global__ __launch_bounds__(256) void append_valu(const T* __restrict__ x, const T* __restrict__ Lk,
                                                   const T* __restrict__ Lv,
                                                   const int64_t* __restrict__ slot,
                                                   T* __restrict__ pool, int n_tok, int m, int RK,
                                                   int RKp, int rv, int64_t page_elems,
                                                   int64_t value_base, int64_t num_pages) {
  __shared__ float xs[kTileK][kTileTok + 4];
  __shared__ float ls[kTileK][kTileCol + 4];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int tok0 = blockIdx.y * kTileTok;
  const int col0 = blockIdx.x * kTileCol;
  const int ncols = RKp + rv;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  for (int k0 = 0; k0 < m; k0 += kTileK) {
    for (int e = tid; e < kTileTok * kTileK; e += 256) {
      const int tt = e / kTileK, kk = e % kTileK;
      const int tok = tok0 + tt, k = k0 + kk;
      xs[kk][tt] = (tok < n_tok && k < m) ? to_f32(x[int64_t(tok) * m + k]) : 0.f;
    }
    for (int e = tid; e < kTileK * kTileCol; e += 256) {
      const int kk = e / kTileCol, cc = e % kTileCol;
      const int c = col0 + cc, k = k0 + kk;
      float v = 0.f;
      if (k < m) {
        if (c < RK)
          v = to_f32(Lk[int64_t(k) * RK + c]);
        else if (c >= RKp && c < ncols)
          v = to_f32(Lv[int64_t(k) * rv + (c - RKp)]);
      }
      ls[kk][cc] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kTileK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = xs[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = ls[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }

  const int64_t slot_end = num_pages * DCKV_PAGE_TOKENS;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = tok0 + ty * 4 + i;
    if (tok >= n_tok) continue;
    const int64_t sl = slot[tok];
    if (sl < 0 || sl >= slot_end) continue;
    T* pg = pool + (sl / DCKV_PAGE_TOKENS) * page_elems;
    const int s = int(sl % DCKV_PAGE_TOKENS);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = col0 + tx * 4 + j;
      if (c >= ncols) continue;
      if (c < RK)
        pg[int64_t(s) * RKp + c] = from_f32<T>(acc[i][j]);
      else if (c < RKp)
        pg[int64_t(s) * RKp + c] = from_f32<T>(0.f);
      else
        pg[value_base + int64_t(c - RKp) * DCKV_PAGE_TOKENS + s] = from_f32<T>(acc[i][j]);
    }
  }
}

template <typename T>
hipError_t launch_append_t(const dckv_plan& p, const void* x, int32_t n_tok, const void* Lk,
                           const void* Lv, const int64_t* slot, void* pool, int64_t num_pages,
                           hipStream_t stream) {
  const int ncols = p.RKp + p.rv;
  dim3 grid((ncols + kTileCol - 1) / kTileCol, (n_tok + kTileTok - 1) / kTileTok);
  hipLaunchKernelGGL(append_valu<T>, grid, dim3(256), 0, stream, static_cast<const T*>(x),
                     static_cast<const T*>(Lk), static_cast<const T*>(Lv), slot,
                     static_cast<T*>(pool), n_tok, p.m, p.RK, p.RKp, p.rv, p.page_elems,
                     p.value_base, num_pages);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_append(const dckv_plan& p, const void* x, int32_t n_tok, const void* L_keys,
                         const void* L_value, const int64_t* slot, void* pool, int64_t num_pages,
                         hipStream_t stream) {
  if (p.dtype == DCKV_F32)
    return launch_append_t<float>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
  return launch_append_t<bf16>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
}

}  // namespace dckv
