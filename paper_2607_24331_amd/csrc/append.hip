// Latent write for new tokens: z = x L (Sec. III-A write
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
      const int cc = e / kTileK, kk = e % kTileK;
      const int c = col0 + cc, k = k0 + kk;
      float v = 0.f;
      if (k < m) {
        if (c < RK)
          v = to_f32(Lk[int64_t(c) * m + k]);
        else if (c >= RKp && c < ncols)
          v = to_f32(Lv[int64_t(c - RKp) * m + k]);
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

// bf16 MFMA kernel (m a multiple of 32).  Output C[token][column] =
// sum_k x[token][k] * LT[column][k]: both operands are contiguous in k, so
// every MFMA operand lane reads its 8 consecutive k with one 16-byte load.
// Work-group tile 64 tokens x 128 columns, four waves of 32 x 64 (2 x 4
// tiles of 16 x 16), k-steps of 32 with the next step's operands loaded
// while the current one multiplies.  Rows past the token count or the
// column space are clamped to valid rows and their results discarded, so no
// load leaves its matrix.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kAM = 2;   // 16-token tiles a wave
constexpr int kAN = 4;   // 16-column tiles a wave

__global__ __launch_bounds__(256) void append_mfma(const bf16* __restrict__ x,
                                                   const bf16* __restrict__ LkT,
                                                   const bf16* __restrict__ LvT,
                                                   const int64_t* __restrict__ slot,
                                                   bf16* __restrict__ pool, int n_tok, int m, int RK,
                                                   int RKp, int rv, int64_t page_elems,
                                                   int64_t value_base, int64_t num_pages) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;
  const int ncols = RKp + rv;
  const int tok_w = blockIdx.y * 64 + (w >> 1) * 32;
  const int col_w = blockIdx.x * 128 + (w & 1) * 64;

  const bf16* arow[kAM];
#pragma unroll
  for (int i = 0; i < kAM; ++i) {
    const int t = min(tok_w + 16 * i + lr, n_tok - 1);
    arow[i] = x + int64_t(t) * m + 8 * lq;
  }
  const bf16* brow[kAN];
#pragma unroll
  for (int j = 0; j < kAN; ++j) {
    const int c = col_w + 16 * j + lr;
    const bf16* r;
    if (c < RK)
      r = LkT + int64_t(c) * m;
    else if (c < RKp)
      r = LkT;                                  // padding column: written as zero below
    else
      r = LvT + int64_t(min(c - RKp, rv - 1)) * m;
    brow[j] = r + 8 * lq;
  }

  floatx4_t acc[kAM][kAN];
#pragma unroll
  for (int i = 0; i < kAM; ++i)
#pragma unroll
    for (int j = 0; j < kAN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  u32x4_t a0[kAM], b0[kAN], a1[kAM], b1[kAN];
  auto load = [&](u32x4_t (&a)[kAM], u32x4_t (&b)[kAN], int k) {
#pragma unroll
    for (int i = 0; i < kAM; ++i) a[i] = *reinterpret_cast<const u32x4_t*>(arow[i] + k);
#pragma unroll
    for (int j = 0; j < kAN; ++j) b[j] = *reinterpret_cast<const u32x4_t*>(brow[j] + k);
  };
  auto mma = [&](const u32x4_t (&a)[kAM], const u32x4_t (&b)[kAN]) {
#pragma unroll
    for (int i = 0; i < kAM; ++i)
#pragma unroll
      for (int j = 0; j < kAN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[i]),
                                                            __builtin_bit_cast(bf16x8_t, b[j]),
                                                            acc[i][j], 0, 0, 0);
  };
  load(a0, b0, 0);
  int k = 0;
  for (; k + 64 <= m; k += 64) {
    load(a1, b1, k + 32);
    mma(a0, b0);
    if (k + 64 < m) load(a0, b0, k + 64);
    mma(a1, b1);
  }
  if (k < m) mma(a0, b0);                       // m = 32 (mod 64): one step left

  // stores: lane holds tokens 4*lq + v of each token tile, column lr of each column tile
  const int64_t slot_end = num_pages * DCKV_PAGE_TOKENS;
#pragma unroll
  for (int i = 0; i < kAM; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int t = tok_w + 16 * i + 4 * lq + v;
      if (t >= n_tok) continue;
      const int64_t sl = slot[t];
      if (sl < 0 || sl >= slot_end) continue;
      bf16* pg = pool + (sl / DCKV_PAGE_TOKENS) * page_elems;
      const int sp = int(sl % DCKV_PAGE_TOKENS);
#pragma unroll
      for (int j = 0; j < kAN; ++j) {
        const int c = col_w + 16 * j + lr;
        if (c >= ncols) continue;
        const float val = acc[i][j][v];
        if (c < RK)
          pg[int64_t(sp) * RKp + c] = static_cast<bf16>(val);
        else if (c < RKp)
          pg[int64_t(sp) * RKp + c] = static_cast<bf16>(0.f);
        else
          pg[value_base + int64_t(c - RKp) * DCKV_PAGE_TOKENS + sp] = static_cast<bf16>(val);
      }
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
  if (p.m % 32 == 0) {
    const int ncols = p.RKp + p.rv;
    dim3 grid((ncols + 127) / 128, (n_tok + 63) / 64);
    hipLaunchKernelGGL(append_mfma, grid, dim3(256), 0, stream, static_cast<const bf16*>(x),
                       static_cast<const bf16*>(L_keys), static_cast<const bf16*>(L_value), slot,
                       static_cast<bf16*>(pool), n_tok, p.m, p.RK, p.RKp, p.rv, p.page_elems,
                       p.value_base, num_pages);
    return hipGetLastError();
  }
  return launch_append_t<bf16>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
}

}  // namespace dckv
