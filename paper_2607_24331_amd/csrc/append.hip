// Latent write for new tokens: z = x L (Sec. III-A write
// side; per-group L_g of Sec. III-C; whole-projection L_v of Sec. III-D),
// accumulated in fp32, rounded to nearest-even into the paged pool.
//
// Output column space of one token: [0, R_Kp + r_v)
//   c <  R_K          key column c           -> page key part (chunk-major)
//   R_K <= c < R_Kp   key-row padding         -> written as zero
//   c >= R_Kp         value column c - R_Kp   -> page value part, rank-major
#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

// Chunk-major key part: column c of slot s at (c/32)*2048 + s*32 + c%32.
__device__ __forceinline__ int64_t key_elem(int s, int c) {
  return int64_t(c >> 5) * (32 * DCKV_PAGE_TOKENS) + s * 32 + (c & 31);
}

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
        pg[key_elem(s, c)] = from_f32<T>(acc[i][j]);
      else if (c < RKp)
        pg[key_elem(s, c)] = from_f32<T>(0.f);
      else
        pg[value_base + int64_t(c - RKp) * DCKV_PAGE_TOKENS + s] = from_f32<T>(acc[i][j]);
    }
  }
}

// bf16 MFMA kernel (m a multiple of 64).  Output C[token][column] =
// sum_k x[token][k] * LT[column][k]: both operands are contiguous in k.
// Work-group tile 128 tokens x 128 columns, four waves of 64 x 64 (4 x 4
// tiles of 16 x 16); k advances in stages of 64 staged through LDS (rows
// padded to 72 elements so the 16 rows an MFMA operand load touches fall in
// distinct banks), two stages in flight: the next stage's global loads are
// issued before the current stage multiplies.  Rows past the token count or
// the column space are clamped to valid rows and their results discarded,
// so no load leaves its matrix.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBM = 128;                  // tokens a work-group
constexpr int kBN = 128;                  // columns a work-group
constexpr int kBK = 64;                   // k a stage
constexpr int kLdsRow = kBK + 8;          // padded LDS row (elements)
constexpr int kStageElems = (kBM + kBN) * kLdsRow;

__global__ __launch_bounds__(256) void append_mfma(const bf16* __restrict__ x,
                                                   const bf16* __restrict__ LkT,
                                                   const bf16* __restrict__ LvT,
                                                   const int64_t* __restrict__ slot,
                                                   bf16* __restrict__ pool, int n_tok, int m, int RK,
                                                   int RKp, int rv, int64_t page_elems,
                                                   int64_t value_base, int64_t num_pages) {
  __shared__ __align__(16) bf16 lds[2 * kStageElems];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;
  const int ncols = RKp + rv;
  const int tok0 = blockIdx.y * kBM, col0 = blockIdx.x * kBN;

  // global rows this thread stages: rows tid/8 + 32*i (i < 4) of the A and
  // B tiles, 16-byte piece tid%8 of the stage's 64 k
  const int piece = tid & 7, prow = tid >> 3;
  const bf16* ga[4];
  const bf16* gb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = min(tok0 + prow + 32 * i, n_tok - 1);
    ga[i] = x + int64_t(t) * m + 8 * piece;
    const int c = col0 + prow + 32 * i;
    const bf16* r;
    if (c < RK)
      r = LkT + int64_t(c) * m;
    else if (c < RKp)
      r = LkT;                                // padding column: written as zero below
    else
      r = LvT + int64_t(min(c - RKp, rv - 1)) * m;
    gb[i] = r + 8 * piece;
  }
  u32x4_t ra[4], rb[4];
  auto gload = [&](int k) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = *reinterpret_cast<const u32x4_t*>(ga[i] + k);
      rb[i] = *reinterpret_cast<const u32x4_t*>(gb[i] + k);
    }
  };
  auto lstore = [&](int buf) {
    bf16* A = lds + buf * kStageElems;
    bf16* B = A + kBM * kLdsRow;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<u32x4_t*>(A + (prow + 32 * i) * kLdsRow + 8 * piece) = ra[i];
      *reinterpret_cast<u32x4_t*>(B + (prow + 32 * i) * kLdsRow + 8 * piece) = rb[i];
    }
  };

  floatx4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  const int wm = (w >> 1) * 64, wn = (w & 1) * 64;   // this wave's 64 x 64 sub-tile

  gload(0);
  lstore(0);
  __syncthreads();
  const int nst = m / kBK;
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    if (st + 1 < nst) gload((st + 1) * kBK);          // in flight while this stage multiplies
    const bf16* A = lds + buf * kStageElems;
    const bf16* B = A + kBM * kLdsRow;
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      u32x4_t a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        a[i] = *reinterpret_cast<const u32x4_t*>(A + (wm + 16 * i + lr) * kLdsRow + 32 * ks + 8 * lq);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        b[j] = *reinterpret_cast<const u32x4_t*>(B + (wn + 16 * j + lr) * kLdsRow + 32 * ks + 8 * lq);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[i]),
                                                              __builtin_bit_cast(bf16x8_t, b[j]),
                                                              acc[i][j], 0, 0, 0);
    }
    if (st + 1 < nst) lstore(buf ^ 1);
    __syncthreads();
  }

  // stores: lane holds tokens 4*lq + v of each token tile, column lr of each column tile
  const int64_t slot_end = num_pages * DCKV_PAGE_TOKENS;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int t = tok0 + wm + 16 * i + 4 * lq + v;
      if (t >= n_tok) continue;
      const int64_t sl = slot[t];
      if (sl < 0 || sl >= slot_end) continue;
      bf16* pg = pool + (sl / DCKV_PAGE_TOKENS) * page_elems;
      const int sp = int(sl % DCKV_PAGE_TOKENS);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = col0 + wn + 16 * j + lr;
        if (c >= ncols) continue;
        const float val = acc[i][j][v];
        if (c < RK)
          pg[key_elem(sp, c)] = static_cast<bf16>(val);
        else if (c < RKp)
          pg[key_elem(sp, c)] = static_cast<bf16>(0.f);
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
  if (p.m % kBK == 0) {
    const int ncols = p.RKp + p.rv;
    dim3 grid((ncols + kBN - 1) / kBN, (n_tok + kBM - 1) / kBM);
    hipLaunchKernelGGL(append_mfma, grid, dim3(256), 0, stream, static_cast<const bf16*>(x),
                       static_cast<const bf16*>(L_keys), static_cast<const bf16*>(L_value), slot,
                       static_cast<bf16*>(pool), n_tok, p.m, p.RK, p.RKp, p.rv, p.page_elems,
                       p.value_base, num_pages);
    return hipGetLastError();
  }
  return launch_append_t<bf16>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
}

}  // namespace dckv
