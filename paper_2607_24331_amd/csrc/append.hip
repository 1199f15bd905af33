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
// stages of 64.  A stage (both tiles, 192 rows x 128 B) is copied from
// global memory straight into LDS by the loads' LDS path (no registers, no
// LDS store instructions): one wave instruction moves 8 rows x 128 B, whole
// cache lines, to 1 KB of LDS in lane order, and the lane -> 16-byte piece
// map is xor-swizzled by the row (LDS piece p of row r holds global piece
// p ^ (r % 8)) so that the 16 rows an MFMA operand load touches fall in
// distinct banks.  NB stage buffers: the loads run NB - 1 stages ahead, and
// one barrier a stage (after the wave's own loads of that stage and its LDS
// reads of the stage before have completed) both publishes the stage and
// frees the buffer the next loads refill.  Eight waves, two a SIMD (one wave
// alone cannot keep the matrix pipe busy across the per-stage barrier):
// wave w owns tokens 32 (w % 4) .. +31 against all 64 columns (2 x 4 tiles
// of 16 x 16) and the k half w / 4 of every stage; at the end the upper k
// half's sums are added to the lower half's through LDS (a fixed order).
// Work-group ids that are equal mod 8 run on one XCD; the id -> tile map
// gives each XCD a contiguous run of tiles with the token tiles of one
// column tile adjacent, so that column tile of L is fetched into the XCD's
// L2 once.  Rows past the token count or the column space are clamped to
// valid rows and their results discarded, so no load leaves its matrix.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBM = 128;                  // tokens a work-group
constexpr int kBN = 64;                   // columns a work-group
constexpr int kBK = 64;                   // k a stage (one 128-byte line a row)
constexpr int kThreads = 512;
constexpr int kNB = 4;                    // LDS stage buffers
constexpr int kBufBytes = (kBM + kBN) * kBK * 2;   // one stage: 24 blocks of 8 rows x 128 B
constexpr int kExchBytes = 4 * 2 * 4 * 64 * 16;     // k-half exchange: 4 waves x 8 tiles x 64 lanes
static_assert(kExchBytes <= kNB * kBufBytes, "the exchange fits the stage buffers");

template <int NB>
__global__ __launch_bounds__(kThreads, 1) void append_mfma(const bf16* __restrict__ x,
                                                          const bf16* __restrict__ LkT,
                                                          const bf16* __restrict__ LvT,
                                                          const int64_t* __restrict__ slot,
                                                          bf16* __restrict__ pool, int n_tok, int m,
                                                          int RK, int RKp, int rv,
                                                          int64_t page_elems, int64_t value_base,
                                                          int64_t num_pages, int n_tok_tiles,
                                                          int n_tiles) {
  __shared__ __align__(1024) unsigned char smem[NB * kBufBytes];
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

  // loads: wave w fills 8-row blocks 3w .. 3w + 2 of a stage (16 x blocks,
  // then 8 L blocks); lane: row lane / 8 of its block, LDS piece lane % 8,
  // which holds global piece (lane % 8) ^ (row % 8)
  const int lrow = lane >> 3, gpiece = (lane & 7) ^ lrow;
  const bf16* gsrc[3];
  int loff[3];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const int blk = 3 * w + j;
    loff[j] = blk * 1024;
    const bf16* r;
    if (blk < 16) {
      const int t = min(tok0 + 8 * blk + lrow, n_tok - 1);
      r = x + int64_t(t) * m;
    } else {
      const int c = col0 + 8 * (blk - 16) + lrow;
      if (c < RK)
        r = LkT + int64_t(c) * m;
      else if (c < RKp)
        r = LkT;                                // padding column: written as zero below
      else
        r = LvT + int64_t(min(c - RKp, rv - 1)) * m;
    }
    gsrc[j] = r + 8 * gpiece;
  }
  const int nst = m / kBK;
  auto issue = [&](int st, unsigned char* buf) {      // past the end: re-read the last stage
    const int k = min(st, nst - 1) * kBK;
#pragma unroll
    for (int j = 0; j < 3; ++j)
      __builtin_amdgcn_global_load_lds(gsrc[j] + k, buf + loff[j], 16, 0, 0);
  };

  floatx4_t acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  const int kp = 4 * kh + lq;                         // this lane's 16-byte k piece
  auto stage = [&](int st, unsigned char* cur, unsigned char* nxt) {
    // wait until this wave's loads of stage st (the oldest of the NB - 1
    // stages in flight, three loads each) and its LDS reads of the previous
    // stage are done, then meet the other waves; the asm is a compiler
    // barrier too, so no LDS access moves across it
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"i"(3 * (NB - 2)) : "memory");
    issue(st + NB - 1, nxt);
    u32x4_t a[2], b[4];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int row = wm + 16 * i + lr;
      a[i] = *reinterpret_cast<const u32x4_t*>(cur + row * 128 + 16 * (kp ^ (row & 7)));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = 16 * j + lr;
      b[j] = *reinterpret_cast<const u32x4_t*>(cur + 16 * 1024 + row * 128 + 16 * (kp ^ (row & 7)));
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[i]),
                                                            __builtin_bit_cast(bf16x8_t, b[j]),
                                                            acc[i][j], 0, 0, 0);
  };
#pragma unroll
  for (int u = 0; u < NB - 1; ++u) issue(u, smem + u * kBufBytes);
  if (nst % NB == 0) {
    for (int st0 = 0; st0 < nst; st0 += NB) {
#pragma unroll
      for (int u = 0; u < NB; ++u)
        stage(st0 + u, smem + u * kBufBytes, smem + ((u + NB - 1) % NB) * kBufBytes);
    }
  } else {
    for (int st0 = 0; st0 < nst; st0 += NB) {
#pragma unroll
      for (int u = 0; u < NB; ++u)
        if (st0 + u < nst) stage(st0 + u, smem + u * kBufBytes, smem + ((u + NB - 1) % NB) * kBufBytes);
    }
  }
  __builtin_amdgcn_s_waitcnt(0);                      // the re-reads past the end have landed

  // upper k half -> LDS, lower half adds it (lane-private slots, same order everywhere)
  floatx4_t* ex = reinterpret_cast<floatx4_t*>(smem);   // [4 waves][8 tiles][64 lanes]
  __syncthreads();                                       // stage buffers no longer read
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

template <int NB>
hipError_t launch_append_mfma(const dckv_plan& p, const void* x, int32_t n_tok, const void* Lk,
                              const void* Lv, const int64_t* slot, void* pool, int64_t num_pages,
                              hipStream_t stream) {
  const int ncols = p.RKp + p.rv;
  const int n_tok_tiles = (n_tok + kBM - 1) / kBM;
  const int n_tiles = n_tok_tiles * ((ncols + kBN - 1) / kBN);
  hipLaunchKernelGGL(append_mfma<NB>, dim3(n_tiles), dim3(kThreads), 0, stream,
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
  if (p.m % kBK == 0)
    return launch_append_mfma<kNB>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
  return launch_append_t<bf16>(p, x, n_tok, L_keys, L_value, slot, pool, num_pages, stream);
}

}  // namespace dckv
