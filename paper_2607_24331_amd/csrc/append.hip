// Latent write for new tokens: z = x L (Sec. III-A write
// side; per-group L_g of Sec. III-C; whole-projection L_v of Sec. III-D),
// accumulated in fp32, rounded to nearest-even into the paged pool.
//
// Output column space of one token: [0, R_Kp + r_v)
//   c <  R_K          key column c           -> page key part (chunk-major)
//   R_K <= c < R_Kp   key-row padding         -> written as zero
//   c >= R_Kp         value column c - R_Kp   -> page value part, tile-major
#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

// Chunk-major key part: column c of slot s at (c/32)*2048 + s*32 + c%32.
__device__ __forceinline__ int64_t key_elem(int s, int c) {
  return int64_t(c >> 5) * (32 * DCKV_PAGE_TOKENS) + s * 32 + (c & 31);
}

// Tile-major value part (from the value base): column j of slot s at
// (j/16)*1024 + (s/32)*512 + (j%16)*32 + s%32.
__device__ __forceinline__ int64_t value_elem(int s, int j) {
  return int64_t(j >> 4) * (16 * DCKV_PAGE_TOKENS) + (s >> 5) * 512 + (j & 15) * 32 + (s & 31);
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
        pg[value_base + value_elem(s, c - RKp)] = from_f32<T>(acc[i][j]);
    }
  }
}

// bf16 MFMA kernel (m a multiple of 64).  Output C[token][column] =
// sum_k x[token][k] * LT[column][k]: both operands are contiguous in k.
// Work-group tile 128 tokens x 64 columns (so the long-context append of
// 512 tokens x 3584 columns fills 224 of the 256 CUs).  k advances in
// stages of 64.  Both tiles of a stage are staged through two LDS buffers
// (rows padded to 72 elements so the 16 rows an MFMA operand load touches
// fall in distinct banks) by loads that each cover 8 rows x 128 B, whole
// cache lines: a load in MFMA operand order (16 rows x 64 B) halves the L1
// throughput.  Every thread keeps the global loads of the next D stages in
// flight.  Eight waves, two a SIMD (one wave alone cannot keep the matrix
// pipe busy across the per-stage barrier): wave w owns tokens
// 32 (w % 4) .. +31 against all 64 columns (2 x 4 tiles of 16 x 16) and the
// k half w / 4 of every stage; at the end the upper k half's sums are added
// to the lower half's through LDS (a fixed order).  Work-group ids that are
// equal mod 8 run on one XCD; the id -> tile map gives each XCD a contiguous
// run of tiles with the token tiles of one column tile adjacent, so that
// column tile of L is fetched into the XCD's L2 once.  Rows past the token
// count or the column space are clamped to valid rows and their results
// discarded, so no load leaves its matrix.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBM = 128;                  // tokens a work-group
constexpr int kBN = 64;                   // columns a work-group
constexpr int kBK = 64;                   // k a stage
constexpr int kThreads = 512;
constexpr int kLdsRow = kBK + 8;          // padded LDS row (elements)
constexpr int kStageElems = (kBM + kBN) * kLdsRow;
constexpr int kPieces = kBK / 8;                    // 16-byte pieces a row a stage
constexpr int kRowsPerPass = kThreads / kPieces;      // rows one pass of all threads covers
constexpr int kALoads = kBM / kRowsPerPass;          // 16-byte x loads a thread a stage
constexpr int kBLoads = kBN / kRowsPerPass;          // 16-byte L loads a thread a stage
constexpr int kStageBytes = 2 * kStageElems * 2;    // both buffers
constexpr int kExchBytes = 4 * 2 * 4 * 64 * 16;     // k-half exchange: 4 waves x 8 tiles x 64 lanes
constexpr int kLdsBytes = kStageBytes > kExchBytes ? kStageBytes : kExchBytes;

template <int D>
__global__ __launch_bounds__(kThreads, 1) void append_mfma(const bf16* __restrict__ x,
                                                          const bf16* __restrict__ LkT,
                                                          const bf16* __restrict__ LvT,
                                                          const int64_t* __restrict__ slot,
                                                          bf16* __restrict__ pool, int n_tok, int m,
                                                          int RK, int RKp, int rv,
                                                          int64_t page_elems, int64_t value_base,
                                                          int64_t num_pages, int n_tok_tiles,
                                                          int n_tiles) {
  __shared__ __align__(16) unsigned char smem[kLdsBytes];
  bf16* lds = reinterpret_cast<bf16*>(smem);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;
  const int ncols = RKp + rv;

  // XCD-aware tile order: ids id, id + 8, ... (one XCD) take consecutive tiles
  const int id = blockIdx.x;
  const int xcd = id & 7, q = id >> 3;
  const int per = n_tiles >> 3, extra = n_tiles & 7;
  const int tile = xcd * per + min(xcd, extra) + q;
  const int tok0 = (tile % n_tok_tiles) * kBM;
  const int col0 = (tile / n_tok_tiles) * kBN;
  const int wm = 32 * (w & 3);                        // this wave's first token
  const int kh = w >> 2;                              // this wave's k half

  // staging: rows prow + kRowsPerPass i of both tiles, 16-byte piece
  // tid % kPieces (a wave covers 8 rows x 128 B)
  const int piece = tid % kPieces, prow = tid / kPieces;
  const bf16* ga[kALoads];
#pragma unroll
  for (int i = 0; i < kALoads; ++i) {
    const int t = min(tok0 + prow + kRowsPerPass * i, n_tok - 1);
    ga[i] = x + int64_t(t) * m + 8 * piece;
  }
  const bf16* gb[kBLoads];
#pragma unroll
  for (int i = 0; i < kBLoads; ++i) {
    const int c = col0 + prow + kRowsPerPass * i;
    const bf16* r;
    if (c < RK)
      r = LkT + int64_t(c) * m;
    else if (c < RKp)
      r = LkT;                                // padding column: written as zero below
    else
      r = LvT + int64_t(min(c - RKp, rv - 1)) * m;
    gb[i] = r + 8 * piece;
  }
  u32x4_t ra[D][kALoads], rb[D][kBLoads];
  const int nst = m / kBK;
  auto kof = [&](int st) { return min(st, nst - 1) * kBK; };   // past the end: re-read the last
  auto gload = [&](u32x4_t (&a)[kALoads], u32x4_t (&b)[kBLoads], int st) {
    const int k = kof(st);
#pragma unroll
    for (int i = 0; i < kALoads; ++i) a[i] = *reinterpret_cast<const u32x4_t*>(ga[i] + k);
#pragma unroll
    for (int i = 0; i < kBLoads; ++i) b[i] = *reinterpret_cast<const u32x4_t*>(gb[i] + k);
  };

  floatx4_t acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  // keep the prologue's stages in ring order, so that waiting for the
  // oldest stage never waits for the younger ones (vmcnt counts in order)
#pragma unroll
  for (int d = 0; d < D; ++d) {
    gload(ra[d], rb[d], d);
    __builtin_amdgcn_sched_barrier(0);
  }
  // nst is a multiple of D (the launcher picks D so), and D is even or 1
  for (int st0 = 0; st0 < nst; st0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int buf = (D == 1) ? (st0 & 1) : (d & 1);
      bf16* A = lds + buf * kStageElems;
      bf16* B = A + kBM * kLdsRow;
#pragma unroll
      for (int i = 0; i < kALoads; ++i)
        *reinterpret_cast<u32x4_t*>(A + (prow + kRowsPerPass * i) * kLdsRow + 8 * piece) = ra[d][i];
#pragma unroll
      for (int i = 0; i < kBLoads; ++i)
        *reinterpret_cast<u32x4_t*>(B + (prow + kRowsPerPass * i) * kLdsRow + 8 * piece) = rb[d][i];
      gload(ra[d], rb[d], st0 + d + D);
      __syncthreads();
#pragma unroll
      for (int ks = 0; ks < kBK / 64; ++ks) {
        const int kk = (kBK / 2) * kh + 32 * ks + 8 * lq;   // this wave's k half, step ks
        u32x4_t a[2], b[4];
#pragma unroll
        for (int i = 0; i < 2; ++i)
          a[i] = *reinterpret_cast<const u32x4_t*>(A + (wm + 16 * i + lr) * kLdsRow + kk);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          b[j] = *reinterpret_cast<const u32x4_t*>(B + (16 * j + lr) * kLdsRow + kk);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[i]),
                                                                __builtin_bit_cast(bf16x8_t, b[j]),
                                                                acc[i][j], 0, 0, 0);
      }
    }
  }

  // upper k half -> LDS, lower half adds it (lane-private slots, same order everywhere)
  floatx4_t* ex = reinterpret_cast<floatx4_t*>(smem);   // [4 waves][8 tiles][64 lanes]
  __syncthreads();                                       // staging buffers no longer read
  if (kh == 1) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) ex[((w & 3) * 8 + i * 4 + j) * 64 + lane] = acc[i][j];
  }
  __syncthreads();
  if (kh == 1) return;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] += ex[(w * 8 + i * 4 + j) * 64 + lane];

  // stores: lane holds tokens 4*lq + v of each token tile, column lr of each column tile
  const int64_t slot_end = num_pages * DCKV_PAGE_TOKENS;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
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
        const int c = col0 + 16 * j + lr;
        if (c >= ncols) continue;
        const float val = acc[i][j][v];
        if (c < RK)
          pg[key_elem(sp, c)] = static_cast<bf16>(val);
        else if (c < RKp)
          pg[key_elem(sp, c)] = static_cast<bf16>(0.f);
        else
          pg[value_base + value_elem(sp, c - RKp)] = static_cast<bf16>(val);
      }
    }
  }
}

template <int D>
hipError_t launch_append_mfma(const dckv_plan& p, const void* x, int32_t n_tok, const void* Lk,
                              const void* Lv, const int64_t* slot, void* pool, int64_t num_pages,
                              hipStream_t stream) {
  const int ncols = p.RKp + p.rv;
  const int n_tok_tiles = (n_tok + kBM - 1) / kBM;
  const int n_tiles = n_tok_tiles * ((ncols + kBN - 1) / kBN);
  hipLaunchKernelGGL(append_mfma<D>, dim3(n_tiles), dim3(kThreads), 0, stream,
                     static_cast<const bf16*>(x), static_cast<const bf16*>(Lk),
                     static_cast<const bf16*>(Lv), slot, static_cast<bf16*>(pool), n_tok, p.m,
                     p.RK, p.RKp, p.rv, p.page_elems, p.value_base, num_pages, n_tok_tiles, n_tiles);
  return hipGetLastError();
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
    const int nst = p.m / kBK;
    if (nst % 4 == 0)
      return launch_append_mfma<4>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
    if (nst % 2 == 0)
      return launch_append_mfma<2>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
    return launch_append_mfma<1>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
  }
  return launch_append_t<bf16>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
}

}  // namespace dckv
