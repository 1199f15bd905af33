// bf16 decode path on MFMA (gfx950).
//
// split_mfma: one 256-thread work-group (4 waves, one per SIMD) serves one
// slice of query heads (all heads when H_q <= 32) over one context split, so
// every latent byte of the split is read by exactly one work-group.  Per
// 64-token page:
//   scores   S^T[t][h] = sum_k Z_K[t][k] * Qblk[k][h], where Qblk is the
//            block-diagonal matrix holding head h's folded query q~_h in its
//            group's key columns (Sec. III-C: a head only meets its own group
//            latent).  MFMA 16x16x32 bf16 with fp32 accumulation; q~ is split
//            into bf16 hi + lo parts, so each score carries ~16 mantissa bits
//            of q~ and exact bf16 latents.
//   softmax  base-2 online softmax in fp32: per-head running max and sum,
//            tile maxima exchanged through LDS (two barriers a page).
//   values   acc^T[j][h] += sum_t Z_v^T[j][t] * p^T[t][h] on MFMA, p rounded
//            to bf16, accumulated in value-latent space (Sec. III-D: one value
//            latent shared by every head).
// Each wave streams its own operands with 16-byte loads straight into a
// 16-deep register ring, so 16 KB per wave stay in flight.
//
// merge_mfma: fixed ascending-split log-sum-exp merge of the partials into
// the normalised value-latent output a_h (fp32).
// The up-projection o_h = a_h R_v[:, kv(h) block] is launch_upproj (decode_pass.hip).
#include <cmath>

#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kPageSlots = 256;           // pages per split the LDS page list holds
constexpr int kPStride = 72;              // bf16 per head row of the p tile (64 + pad)
constexpr int kMergeRanks = 8;            // value ranks per merge work-group (16 for deep batches)
constexpr int kQblkLoads = 16;            // folded-query loads a thread issued at the split's start

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Word 3 of a raw buffer descriptor on gfx9-family parts (32-bit data
// format, no swizzle); loads at or past num_records return zero.
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kOutOfRange = 0x40000000;   // byte offset beyond any page
constexpr int kNonTemporal = 2;           // cache policy of streamed latents: nt

// One producer block: consecutive items of one page (KR keys or VR values),
// values (kind 2: past the split, every load reads zero).
struct ProdBlock {
  __amdgpu_buffer_rsrc_t rsrc;
  int kind;
  int base;    // byte offset of the block's first item, lane part excluded
  int idx0;    // index of the block's first item in the page's stream
  int nval;    // valid tokens of the page
};

__device__ __forceinline__ floatx4 mfma(u32x4 a, u32x4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ u32x4 load16(const bf16* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// Keep the first `n` (0..8) bf16 of a 16-byte vector, zero the rest.
__device__ __forceinline__ u32x4 keep_first(u32x4 v, int n) {
  u32x4 r;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t lo = (2 * d < n) ? 0x0000FFFFu : 0u;
    const uint32_t hi = (2 * d + 1 < n) ? 0xFFFF0000u : 0u;
    r[d] = v[d] & (lo | hi);
  }
  return r;
}

__device__ __forceinline__ float wave_max16(float v) {   // over lanes l, l^16, l^32, l^48
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}
__device__ __forceinline__ float wave_sum16(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

// ---------------------------------------------------------------------------
// fold_blocks: the folded queries q~_h = q_h R_{g,h}^T * log2(e)/sqrt(d_h)
// (Sec. III-A: q (z R)^T = (q R^T) z^T; Sec. III-C: head h meets only its
// group's factor), written straight into the split kernel's B-operand blocks.
// Block (slice, tile n, chunk c) holds, for head slot 16n + j and key column
// 32c + kk, q~ of that slot's head at column kk - koff_g when the column lies
// in the head's group latent, else zero; split as bf16 hi + lo parts.  B
// operand order: lane 16*(kk/8) + j, element kk%8.  One wave per (block,
// slot): 32 columns, two lanes a column (halves of d_h).
__global__ __launch_bounds__(64) void fold_blocks(const float* __restrict__ q,
                                                  const bf16* __restrict__ Rk,
                                                  u32x4* __restrict__ qblk_ws, float scale,
                                                  HeadTables tb, MfmaTables mt) {
  const int j = blockIdx.y, pr = blockIdx.z;           // (sequence, slice) on x: grid x is wide
  const int J = mt.n_slices;
  const int b = blockIdx.x / J, slice = blockIdx.x % J;
  const int nch0 = mt.kln[slice][0][0] + mt.kln[slice][0][1];
  const int npairs = nch0 + (mt.nt > 1 ? mt.kln[slice][1][0] + mt.kln[slice][1][1] : 0);
  if (pr >= npairs) return;
  const int n = pr < nch0 ? 0 : 1;
  const int ci = pr - (n ? nch0 : 0);                   // position in the tile's chunk list
  const int c = ci < mt.kln[slice][n][0] ? mt.kst[slice][n][0] + ci
                                         : mt.kst[slice][n][1] + (ci - mt.kln[slice][n][0]);
  const int row = mt.hord[slice][16 * n + j];           // query i * H_q + head h, or -1
  const int h = row < 0 ? -1 : row % tb.n_q_heads, qi = row < 0 ? 0 : row / tb.n_q_heads;
  const int lane = threadIdx.x, kk = lane & 31, half = lane >> 5;
  const int k = 32 * c + kk;
  const int dh = tb.head_dim, hd = dh / 2, d0 = half * hd;   // d_h is a multiple of 8
  float v = 0.f;
  if (h >= 0) {
    const int lo = tb.koff_of_q[h], r = tb.rank_of_q[h];
    if (k >= lo && k < lo + r) {
      const bf16* row = Rk + tb.roff_of_q[h] + int64_t(k - lo) * tb.rstride_of_q[h] + tb.rcol_of_q[h] + d0;
      const float* qh = q + ((int64_t(b) * tb.n_queries + qi) * tb.n_q_heads + h) * dh + d0;
      // 8 columns a step: one 8-byte-aligned load of R (4 x bf16 pairs) and two float4 of q
      for (int d = 0; d < hd; d += 8) {
        uint32_t w4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) w4[j] = *reinterpret_cast<const uint32_t*>(row + d + 2 * j);
        const float4 qa = *reinterpret_cast<const float4*>(qh + d);
        const float4 qb = *reinterpret_cast<const float4*>(qh + d + 4);
        const float qv[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v = fmaf(qv[2 * j], __uint_as_float(w4[j] << 16), v);
          v = fmaf(qv[2 * j + 1], __uint_as_float(w4[j] & 0xFFFF0000u), v);
        }
      }
    }
  }
  v += __shfl_xor(v, 32);
  if (half == 0) {
    v *= scale;
    const bf16 vh = static_cast<bf16>(v);
    const bf16 vl = static_cast<bf16>(v - static_cast<float>(vh));
    bf16* blk = reinterpret_cast<bf16*>(qblk_ws + (int64_t(b * J + slice) * mt.max_pairs + pr) * 128);
    const int l = 16 * (kk >> 3) + j, e = kk & 7;
    blk[l * 8 + e] = vh;
    blk[512 + l * 8 + e] = vl;
  }
}

// fold_mfma: the same blocks as fold_blocks, as one small product a (slice,
// slot, 32-column chunk): the batch's query rows of the slot's head (B x d_h)
// times the R rows of the chunk's columns (d_h x 32), on MFMA.  One wave;
// its B operands (R, bf16) are loaded once and serve every 16-sequence tile
// of the batch; the A operands are the fp32 query rows split into bf16 hi +
// lo parts (two products a k step), accumulated in fp32.  Columns outside
// the head's group latent, and slots without a head, are written as zero.
// d_h a multiple of 32 (KS = d_h / 32 k steps).
template <int KS>
__global__ __launch_bounds__(64) void fold_mfma(const float* __restrict__ q,
                                                const bf16* __restrict__ Rk,
                                                u32x4* __restrict__ qblk_ws, int batch, float scale,
                                                HeadTables tb, MfmaTables mt) {
  const int J = mt.n_slices;
  // 1-D grid, XCD-aware: the 16 slots of one (slice, chunk) write
  // interleaved 16-byte pieces of the same blocks, so they share an XCD
  // (work-group ids equal mod 8) and its L2 merges the pieces
  const int ngrp = J * mt.max_pairs;
  const int xcd = blockIdx.x & 7, pos = blockIdx.x >> 3;
  const int grp = 8 * (pos >> 4) + xcd, j = pos & 15;
  if (grp >= ngrp) return;
  const int slice = grp / mt.max_pairs, pr = grp % mt.max_pairs;
  const int nch0 = mt.kln[slice][0][0] + mt.kln[slice][0][1];
  const int npairs = nch0 + (mt.nt > 1 ? mt.kln[slice][1][0] + mt.kln[slice][1][1] : 0);
  if (pr >= npairs) return;
  const int n = pr < nch0 ? 0 : 1;
  const int ci = pr - (n ? nch0 : 0);
  const int c = ci < mt.kln[slice][n][0] ? mt.kst[slice][n][0] + ci
                                         : mt.kst[slice][n][1] + (ci - mt.kln[slice][n][0]);
  const int row = mt.hord[slice][16 * n + j];           // query i * H_q + head h, or -1
  const int h = row < 0 ? -1 : row % tb.n_q_heads, qi = row < 0 ? 0 : row / tb.n_q_heads;
  const int lane = threadIdx.x, lr = lane & 15, lq = lane >> 4;
  const int dh = tb.head_dim;
  const int lo = h < 0 ? 0 : tb.koff_of_q[h], rk = h < 0 ? 0 : tb.rank_of_q[h];
  // B operands: column 16 t + lr of the chunk, d = 32 ks + 8 lq .. +7
  u32x4 bR[2][KS];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int k = 32 * c + 16 * t + lr;
    const bool live = k >= lo && k < lo + rk;
    const bf16* src = live ? Rk + tb.roff_of_q[h] + int64_t(k - lo) * tb.rstride_of_q[h] + tb.rcol_of_q[h]
                           : Rk;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      bR[t][ks] = live ? load16(src + 32 * ks + 8 * lq) : u32x4{0u, 0u, 0u, 0u};
  }
  // output columns of this lane: 16 t + lr, t = 0, 1
  bool out_live[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int k = 32 * c + 16 * t + lr;
    out_live[t] = k >= lo && k < lo + rk;
  }
  const int hq = h < 0 ? 0 : h;
  float4 qa[KS][2], qn[KS][2];
  auto qload = [&](float4 (&d)[KS][2], int b0) {      // this lane's A row (clamped)
    const int ba = min(b0 + lr, batch - 1);
    const float* qh = q + ((int64_t(ba) * tb.n_queries + qi) * tb.n_q_heads + hq) * dh + 8 * lq;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      d[ks][0] = *reinterpret_cast<const float4*>(qh + 32 * ks);
      d[ks][1] = *reinterpret_cast<const float4*>(qh + 32 * ks + 4);
    }
  };
  qload(qa, 0);
  for (int b0 = 0; b0 < batch; b0 += 16) {
    if (b0 + 16 < batch) qload(qn, b0 + 16);           // the next tile's rows in flight
    floatx4 acc[2] = {floatx4{0.f, 0.f, 0.f, 0.f}, floatx4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const float f[8] = {qa[ks][0].x, qa[ks][0].y, qa[ks][0].z, qa[ks][0].w,
                          qa[ks][1].x, qa[ks][1].y, qa[ks][1].z, qa[ks][1].w};
      u32x4 ah, al;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16 h0 = static_cast<bf16>(f[2 * e]), h1 = static_cast<bf16>(f[2 * e + 1]);
        const bf16 l0 = static_cast<bf16>(f[2 * e] - static_cast<float>(h0));
        const bf16 l1 = static_cast<bf16>(f[2 * e + 1] - static_cast<float>(h1));
        ah[e] = uint32_t(__builtin_bit_cast(uint16_t, h0)) | (uint32_t(__builtin_bit_cast(uint16_t, h1)) << 16);
        al[e] = uint32_t(__builtin_bit_cast(uint16_t, l0)) | (uint32_t(__builtin_bit_cast(uint16_t, l1)) << 16);
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        acc[t] = mfma(ah, bR[t][ks], acc[t]);
        acc[t] = mfma(al, bR[t][ks], acc[t]);
      }
    }
    // lane holds sequences b0 + 4 lq + v of columns 16 t + lr
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int b = b0 + 4 * lq + v;
      if (b >= batch) continue;
      bf16* blk = reinterpret_cast<bf16*>(qblk_ws + (int64_t(b * J + slice) * mt.max_pairs + pr) * 128);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int kk = 16 * t + lr;
        const float x = out_live[t] ? acc[t][v] * scale : 0.f;
        const bf16 vh = static_cast<bf16>(x);
        const bf16 vl = static_cast<bf16>(x - static_cast<float>(vh));
        const int l = 16 * (kk >> 3) + j, e = kk & 7;
        blk[l * 8 + e] = vh;
        blk[512 + l * 8 + e] = vl;
      }
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qa[ks][0] = qn[ks][0];
      qa[ks][1] = qn[ks][1];
    }
  }
}

// ---------------------------------------------------------------------------
// W waves (4 or 8) a work-group; NT 16-head tiles; at most MTW value M-tiles
// (16 ranks) a wave; key ring blocks of KR loads, value ring blocks of VR
// (12 or 16, whichever holds the 2 MTW value items of a page without
// padding, or with the least).
// PW (the rotary decode's value pass): the split's softmax weights come
// ready from pw ([slot][split_tokens] bf16 per (sequence, slice, split),
// relative to the split maximum, with m and l already in part_ml), so there
// is no key phase and no online softmax: the whole split's weights are
// staged in LDS once, and the pages stream values only (KR == VR).
template <int W, int NT, int MTW, int KR, bool PW = false>
__global__ __launch_bounds__(W * 64, 1) void split_mfma(
    const u32x4* __restrict__ qblk_ws, const bf16* __restrict__ pool, int64_t num_pages,
    const int32_t* __restrict__ page_table, int max_pages, const int32_t* __restrict__ seq_lens,
    int max_context, int split_tokens, int n_split, int n_units, int RK, int rv,
    int64_t page_elems, int64_t value_base, float* __restrict__ part_ml, float* __restrict__ part,
    MfmaTables mt, const bf16* __restrict__ pw) {
  constexpr int NH = 16 * NT;                          // head slots of the slice
  constexpr int SW = (4 * NT < W) ? 4 * NT : W;        // waves holding score tiles
  constexpr int MPW = (4 * NT) / SW;                   // score M-tiles (16 tokens) a scoring wave
  constexpr int VR = ((2 * MTW) % 16 == 0) ? 16 : 12;  // value ring block
  constexpr int RING = KR > VR ? KR : VR;              // ring slots
  constexpr int NV = ((2 * MTW + VR - 1) / VR) * VR;   // value items a page (padded)
  static_assert(KR % 2 == 0 && KR % MPW == 0 && VR % 2 == 0, "blocks hold whole chunks and k-steps");
  static_assert(!PW || KR == VR, "the weighted value pass streams values only");
  static_assert(!PW || NV == 2 * MTW, "the weighted value pass has no padding items");
  extern __shared__ __align__(16) unsigned char smem[];

  const int J = mt.n_slices;
  const int Lid = blockIdx.x;
  const int grp = Lid / (8 * J), rr = Lid % (8 * J);
  const int slice = rr / 8;
  const int u = grp * 8 + (rr % 8);       // all slices of unit u share an XCD (ids equal mod 8)
  if (u >= n_units) return;               // n_units = batch * n_split (the grid is padded)
  const int b = u / n_split, split = u % n_split;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index, provably uniform
  const int lr = lane & 15, lq = lane >> 4;
  const int t0 = split * split_tokens;

  // ---- LDS carve-up
  const int nch0 = mt.kln[slice][0][0] + mt.kln[slice][0][1];
  const int npairs = PW ? 0 : nch0 + (NT > 1 ? mt.kln[slice][1][0] + mt.kln[slice][1][1] : 0);
  u32x4* qblk = reinterpret_cast<u32x4*>(smem);                         // [npairs][2][64]
  bf16* p_lds = reinterpret_cast<bf16*>(smem + size_t(npairs) * 2048);  // [32][kPStride]
  float* red_max = reinterpret_cast<float*>(p_lds + 32 * kPStride);     // [8][32]
  float* red_sum = red_max + 8 * 32;                                    // [8][32]
  int* pids = reinterpret_cast<int*>(red_sum + 8 * 32);                 // [kPageSlots]
  // PW: the split's weights [NH][split_tokens + 8] (16-byte row pad) after the page list
  const int pst = split_tokens + 8;
  bf16* p_all = reinterpret_cast<bf16*>(pids + kPageSlots);

  // ---- the prologue's loads go out together, none waiting on another:
  // this lane's query row (for the causal limit) and page-table entry, the
  // folded-query blocks (built by fold_blocks) into registers, then the
  // first page's table entry and the context length (scalar).  The vector
  // loads are issued in the order they are consumed, so each wait leaves
  // the later loads in flight.
  // (every load is unconditional at a clamped, valid address, so no branch
  // hides a load from the wait counting; unused values are dropped)
  constexpr int SWc = (4 * NT < W) ? 4 * NT : W;
  const int hrow_raw = mt.hord[slice][min(16 * ((min(w, SWc - 1) * ((4 * NT) / SWc)) / 4) + lr, kSliceHeads - 1)];
  const int hrow = w < SWc ? hrow_raw : -1;
  const int pg_lane = page_table[int64_t(b) * max_pages + min((t0 >> 6) + tid, max_pages - 1)];
  const u32x4* qsrc = qblk_ws + int64_t(b * J + slice) * mt.max_pairs * 128;
  const int n16 = npairs * 128;
  u32x4 qv[kQblkLoads];
  if constexpr (!PW) {
#pragma unroll
    for (int k = 0; k < kQblkLoads; ++k) qv[k] = qsrc[min(tid + k * W * 64, n16 - 1)];
  }
  int pid0 = (t0 >> 6) < max_pages ? page_table[int64_t(b) * max_pages + (t0 >> 6)] : -1;
  pid0 = __builtin_amdgcn_readfirstlane((pid0 >= 0 && pid0 < num_pages) ? pid0 : -1);
  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int t1 = min(t0 + split_tokens, T_b);
  if (t0 >= t1) return;                   // the merge only reads splits holding tokens
  const int np = (t1 - t0 + 63) / 64;

  static_assert(kPageSlots <= W * 64, "one page-table entry a thread");
  if (tid < np) pids[tid] = (pg_lane >= 0 && pg_lane < num_pages) ? pg_lane : -1;

  // ---- wave roles
  const bool scoring = w < SW;
  const int n_w = scoring ? (w * MPW) / 4 : 0;        // score N-tile
  const int mb_w = scoring ? (w * MPW) % 4 : 0;       // first score M-tile
  // the tile's key chunks: list position ci is chunk st0_w + ci below
  // ln0_w, else st1_w + (ci - ln0_w)
  const int st0_w = mt.kst[slice][n_w][0], ln0_w = mt.kln[slice][n_w][0];
  const int st1_w = mt.kst[slice][n_w][1];
  const int nch_w = ln0_w + mt.kln[slice][n_w][1];
  const int nk_real = (scoring && !PW) ? nch_w * MPW : 0;   // key items a page
  // key items padded to whole blocks; with two block sizes every wave has at
  // least one key block (all-dummy for a wave without score tiles), so the
  // last key block's change of length is on every wave's schedule
  const int NK = KR == VR ? (nk_real + KR - 1) / KR * KR : max(KR, (nk_real + KR - 1) / KR * KR);
  const int pair0_w = (n_w == 0) ? 0 : nch0;
  const int mt0_w = w * mt.mtw;
  const int mcnt_w = max(0, min(mt.mtw, mt.mt_v - mt0_w));
  // only the last chunk of the key latent can hold columns beyond r; its
  // list position in this tile, or -1
  const int kc_last = (RK - 1) / 32;
  const int ci_last = (kc_last >= st0_w && kc_last < st0_w + ln0_w) ? kc_last - st0_w
                    : (kc_last >= st1_w && kc_last < st1_w + nch_w - ln0_w) ? ln0_w + kc_last - st1_w
                    : -1;
  // causal limit of this lane's score column: query i of Q sits at position
  // T_b - Q + i and sees the positions before it and its own
  int lim = T_b;
  if (scoring && hrow >= 0) lim = T_b - mt.queries + hrow / mt.q_heads + 1;
  const int kvalid_last = min(8, max(0, RK - (32 * kc_last + 8 * lq)));

  // ---- producer.  The item stream of a page is NK key items (chunk-major,
  // M-tile minor) in blocks of KR, then NV value items (M-tile-major, k-step
  // minor) in blocks of VR.  The producer runs exactly one block ahead of the
  // consumer: while block b is consumed, slot s of block b + 1 is issued as
  // slot s of b is consumed; where b + 1 is longer, its extra slots (free,
  // as b does not use them) are issued before b is consumed, and where it is
  // shorter, b's last slots issue nothing.  Both lengths are whole blocks, so
  // a producer block never spans two pages or two kinds: its page and kind
  // are set once per block, and each issue is a single unconditional 16-byte
  // buffer load (out-of-range offsets read 0).
  const int lane_key = 2 * (lr * 32 + 8 * lq);        // byte offsets of this lane
  const int lane_val = 2 * (lr * 32 + 8 * lq);
  const int page_bytes = int(page_elems * 2);
  const int nkb = NK / KR;                            // key blocks a page
  const int blocks_pp = nkb + NV / VR;                // producer blocks a page
  int prod_block = 0;                                 // producer block counter over the split
  // the first block (page 0) takes its page from pid0: the LDS page list is
  // read only after the prologue's barrier
  auto setup = [&](int pblk, bool first = false) {
    ProdBlock r;
    const int page = pblk / blocks_pp;
    const int blk = pblk - page * blocks_pp;
    int pid = -1;
    if (first) pid = pid0;
    else if (page < np) pid = __builtin_amdgcn_readfirstlane(pids[page]);
    const bf16* base = pid >= 0 ? pool + int64_t(pid) * page_elems : pool;
    r.rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(base), 0,
                                               pid >= 0 ? page_bytes : 0, kRsrcWord3);
    r.nval = page < np ? min(64, (t1 - t0) - page * 64) : 0;
    r.idx0 = blk < nkb ? blk * KR : NK + (blk - nkb) * VR;   // first item of the block
    r.kind = page >= np ? 2 : (r.idx0 < NK ? 0 : 1);
    // key chunk c holds the 64 slots contiguously (2048 elements); M-tile m
    // of it is the 512-element run starting at m * 512.  Value tile u (16
    // ranks) holds the two 32-token halves as 512-element runs from u * 1024.
    r.base = r.kind == 0 ? 2 * (512 * mb_w)
           : PW          ? 2 * (int(value_base) + 1024 * mt0_w)
                         : 2 * (int(value_base) + 1024 * (mt0_w + (r.idx0 - NK) / 2));
    return r;
  };
  // issue item s (compile-time slot) of producer block pb
  auto issue = [&](const ProdBlock& pb, int s) -> u32x4 {
    int off = kOutOfRange;
    if (pb.kind == 0) {
      const int i = pb.idx0 + s;
      const int ci = i / MPW;
      const int c = ci < ln0_w ? st0_w + ci : st1_w + (ci - ln0_w);
      const int o = pb.base + 2 * (512 * (s % MPW) + 2048 * c) + lane_key;
      const bool ok = (i < nk_real) & (32 * c + 8 * lq < RK);     // no short-circuit branches
      off = ok ? o : kOutOfRange;
    } else if (pb.kind == 1) {
      if constexpr (PW) {
        // half-major: item j of the page is tile j % MTW of token half j / MTW
        const int j = pb.idx0 - NK + s;
        const int mtl = j % MTW, ks = j / MTW;
        const int o = pb.base + 2 * (1024 * mtl + 512 * ks) + lane_val;
        const bool ok = (mtl < mcnt_w) & (16 * (mt0_w + mtl) + lr < rv) & (32 * ks + 8 * lq < pb.nval);
        off = ok ? o : kOutOfRange;
      } else {
        const int mtl = (pb.idx0 - NK + s) >> 1;
        const int o = pb.base + 2 * (1024 * (s >> 1) + 512 * (s & 1)) + lane_val;
        const bool ok = (mtl < mcnt_w) & (16 * (mt0_w + mtl) + lr < rv) & (32 * (s & 1) + 8 * lq < pb.nval);
        off = ok ? o : kOutOfRange;
      }
    }
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(pb.rsrc, off, 0, kNonTemporal));
  };

  u32x4 ring[RING];
  {
    const ProdBlock pb0 = setup(prod_block++, true);     // page 0's first key block
#pragma unroll
    for (int s = 0; s < KR; ++s) ring[s] = issue(pb0, s);
  }

  if constexpr (PW) {
    // ---- the split's weights into LDS, four loads in flight a thread;
    // padding slots (no query head) get zero weights
    const bf16* src = pw + (int64_t(b * J + slice) * n_split + split) * NH * split_tokens;
    const int vrow = split_tokens / 8, nvec = NH * vrow;
    for (int base = tid; base < nvec; base += 4 * W * 64) {
      u32x4 v[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = *reinterpret_cast<const u32x4*>(src + 8 * min(base + k * W * 64, nvec - 1));
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int idx = base + k * W * 64;
        if (idx < nvec) {
          const int slot = idx / vrow, col = idx - slot * vrow;
          *reinterpret_cast<u32x4*>(p_all + slot * pst + 8 * col) =
              mt.hord[slice][slot] >= 0 ? v[k] : u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
  }
  // ---- block-diagonal folded query (hi/lo bf16 MFMA B operands): the
  // registers loaded above go to LDS (their loads precede the ring's, so
  // the ring stays in flight); a plan with more blocks than the registers
  // hold copies the rest here, eight loads in flight a thread.
  if constexpr (!PW) {
#pragma unroll
  for (int k = 0; k < kQblkLoads; ++k) {
    const int idx = tid + k * W * 64;
    if (idx < n16) qblk[idx] = qv[k];
  }
  }
  {
    for (int base = tid + kQblkLoads * W * 64; base < n16 && !PW; base += 8 * W * 64) {
      u32x4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int idx = base + k * W * 64;
        if (idx < n16) v[k] = qsrc[idx];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int idx = base + k * W * 64;
        if (idx < n16) qblk[idx] = v[k];
      }
    }
  }
  __syncthreads();

  floatx4 acc[MTW][NT];
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run[NT], l_run[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    m_run[n] = -INFINITY;
    l_run[n] = 0.f;
  }
  const int pmax_pair = pair0_w + max(nch_w, 1) - 1;    // clamp for padded key items

  for (int page = 0; page < np; ++page) {
    const int nval = min(64, (t1 - t0) - page * 64);
    const bool pvalid = pids[page] >= 0;
    u32x4 pB[NT][2];
    if constexpr (PW) {                   // weights ready in LDS: no keys, no softmax
#pragma unroll
      for (int n = 0; n < NT; ++n)        // the first token half's (the second's at mid-page)
        pB[n][0] = *reinterpret_cast<const u32x4*>(p_all + (16 * n + lr) * pst + 64 * page + 8 * lq);
    } else {

    // ---- scores: MPW M-tiles (16 tokens each) of this wave's N-tile
    floatx4 S[MPW];
#pragma unroll
    for (int m = 0; m < MPW; ++m) S[m] = floatx4{0.f, 0.f, 0.f, 0.f};
    // consume key slot s of the block at item kb
    u32x4 bhi = {0u, 0u, 0u, 0u}, blo = {0u, 0u, 0u, 0u};
    auto key_step = [&](int kb, int s) {
      const int c = (kb + s) / MPW;       // position in the tile's chunk list
      if (s % MPW == 0) {
        const int pr = min(pair0_w + c, pmax_pair);
        bhi = qblk[(pr * 2 + 0) * 64 + lane];
        blo = qblk[(pr * 2 + 1) * 64 + lane];
      }
      u32x4 a = ring[s];
      if (c == ci_last) a = keep_first(a, kvalid_last);
      S[s % MPW] = mfma(a, bhi, S[s % MPW]);
      S[s % MPW] = mfma(a, blo, S[s % MPW]);
    };
    if constexpr (KR == VR) {             // one block size: no block changes length
      for (int kb = 0; kb < NK; kb += KR) {
        const ProdBlock pbk = setup(prod_block++);
#pragma unroll
        for (int s = 0; s < KR; ++s) {
          key_step(kb, s);
          ring[s] = issue(pbk, s);
        }
      }
    } else {
      int kb = 0;
      for (; kb < NK - KR; kb += KR) {    // key block -> key block
        const ProdBlock pbk = setup(prod_block++);
#pragma unroll
        for (int s = 0; s < KR; ++s) {
          key_step(kb, s);
          ring[s] = issue(pbk, s);
        }
      }
      {                                   // last key block -> first value block
        const ProdBlock pbv = setup(prod_block++);
#pragma unroll
        for (int s = KR; s < VR; ++s) ring[s] = issue(pbv, s);
#pragma unroll
        for (int s = 0; s < KR; ++s) {
          key_step(kb, s);
          if (s < VR) ring[s] = issue(pbv, s);
        }
      }
    }

    // ---- softmax, part 1: tile maxima
    if (scoring) {
      float tmax = -INFINITY;
#pragma unroll
      for (int m = 0; m < MPW; ++m)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int tok = 16 * (mb_w + m) + 4 * lq + v;
          if (!pvalid || tok >= nval || t0 + 64 * page + tok >= lim) S[m][v] = -INFINITY;
          tmax = fmaxf(tmax, S[m][v]);
        }
      tmax = wave_max16(tmax);
      if (lane < 16) red_max[w * 32 + lane] = tmax;
    }
    __syncthreads();

    // ---- part 2: new maxima, p for own tokens, partial row sums
    float m_new[NT], alpha[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      float mx = m_run[n];
#pragma unroll
      for (int ww = 0; ww < SW; ++ww)
        if ((ww * MPW) / 4 == n) mx = fmaxf(mx, red_max[ww * 32 + lr]);
      m_new[n] = mx;
      alpha[n] = (mx == -INFINITY) ? 1.f : exp2f(m_run[n] - mx);
    }
    if (scoring) {
      float psum = 0.f;
      const float mw = (NT > 1 && n_w == 1) ? m_new[NT - 1] : m_new[0];   // no dynamic register index
#pragma unroll
      for (int m = 0; m < MPW; ++m) {
        uint32_t pk[2];
#pragma unroll
        for (int v2 = 0; v2 < 2; ++v2) {
          uint32_t word = 0;
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const float sc = S[m][2 * v2 + half];
            const float pv = (sc == -INFINITY) ? 0.f : exp2f(sc - mw);
            const bf16 pb = static_cast<bf16>(pv);
            psum += static_cast<float>(pb);
            word |= uint32_t(__builtin_bit_cast(uint16_t, pb)) << (16 * half);
          }
          pk[v2] = word;
        }
        const int tok = 16 * (mb_w + m) + 4 * lq;
        *reinterpret_cast<uint2*>(p_lds + (16 * n_w + lr) * kPStride + tok) = uint2{pk[0], pk[1]};
      }
      psum = wave_sum16(psum);
      if (lane < 16) red_sum[w * 32 + lane] = psum;
    }
    __syncthreads();

    // ---- part 3: running sums, rescale, p operands
    bool rescale = false;
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      float sum = 0.f;
#pragma unroll
      for (int ww = 0; ww < SW; ++ww)
        if ((ww * MPW) / 4 == n) sum += red_sum[ww * 32 + lr];
      l_run[n] = l_run[n] * alpha[n] + sum;
      m_run[n] = m_new[n];
      rescale = rescale || alpha[n] != 1.f;
    }
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        pB[n][ks] = *reinterpret_cast<const u32x4*>(p_lds + (16 * n + lr) * kPStride + 32 * ks + 8 * lq);
    if (__any(rescale)) {                 // the running maximum moved for some head
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int n = 0; n < NT; ++n) acc[i][n] *= alpha[n];
    }
    }                                     // !PW
    // token masks of the two k-steps on a partial page
    const int keep0 = min(8, max(0, nval - 8 * lq));
    const int keep1 = min(8, max(0, nval - 32 - 8 * lq));

    // ---- values: acc^T[rank][head] += Z_v^T[rank][tok] p^T[tok][head]
#pragma unroll
    for (int vb = 0; vb < NV; vb += VR) {
      const ProdBlock pbn = setup(prod_block++);   // next block: values, or the next page's keys
      const bool to_keys = vb + VR == NV;
      if (to_keys) {
#pragma unroll
        for (int s = VR; s < KR; ++s) ring[s] = issue(pbn, s);
      }
#pragma unroll
      for (int s = 0; s < VR; ++s) {
        const int i = vb + s;
        const int mtl = PW ? i % MTW : i >> 1, ks = PW ? i / MTW : i & 1;
        if constexpr (PW) {
          if (i == MTW) {
#pragma unroll
            for (int n = 0; n < NT; ++n)
              pB[n][1] = *reinterpret_cast<const u32x4*>(p_all + (16 * n + lr) * pst + 64 * page + 32 + 8 * lq);
          }
        }
        u32x4 a = ring[s];
        if (nval < 64) a = keep_first(a, ks ? keep1 : keep0);
        if (mtl < MTW) {
#pragma unroll
          for (int n = 0; n < NT; ++n) acc[mtl][n] = mfma(a, pB[n][ks], acc[mtl][n]);
        }
        if (!to_keys || s < KR) ring[s] = issue(pbn, s);
      }
    }
  }

  // ---- partials: (m[NH], l[NH]) compact per split, acc[rank][NH] (head slot fastest)
  const int64_t prow = (int64_t(b) * J + slice) * n_split + split;
  if (w == 0 && lane < 16) {
    float* pml = part_ml + prow * (2 * NH);
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      // PW: the key-rebuild kernel wrote the slots of real heads
      if (!PW || mt.hord[slice][16 * n + lane] < 0) {
        pml[16 * n + lane] = m_run[n];
        pml[NH + 16 * n + lane] = l_run[n];
      }
    }
  }
  float* pa = part + prow * int64_t(NH) * rv;
#pragma unroll
  for (int i = 0; i < MTW; ++i) {
    if (i < mcnt_w) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int rank = 16 * (mt0_w + i) + 4 * lq + v;
        if (rank < rv) {
#pragma unroll
          for (int n = 0; n < NT; ++n) pa[int64_t(rank) * NH + 16 * n + lr] = acc[i][n][v];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Merge: a[b][h][r] = sum_s 2^(m_s - M) acc_s[r] / sum_s 2^(m_s - M) l_s.
// Grid (batch * slices, value-rank chunks of MR), 256 threads; MR = 8, or 16
// when the grid would hold 2048 work-groups or more (deep batches: fewer,
// larger work-groups, each reading the (m, l) rows once for more ranks).
// Pass 1: per head slot the maximum M and the weighted sum L over splits,
// read from the compact (m, l) rows, up to 32 (16 pairs) independent loads
// a thread for long merges, eight for short ones.
// Pass 2: a split row of the chunk is MR * NH contiguous floats;
// TPR threads cover it with float4 loads (4 head slots each) and the
// 256 / TPR thread groups take the splits round-robin, sixteen splits in
// flight for long merges, four for short ones.
// Fixed order: group g sums splits g, g + G, ... ascending, then the G group
// sums are added in order.
template <int NH, bool LONG, int MR>
__global__ __launch_bounds__(256) void merge_mfma(const float* __restrict__ part_ml,
                                                  const float* __restrict__ part,
                                                  const int32_t* __restrict__ seq_lens,
                                                  int max_context, int split_tokens, int n_split,
                                                  int rv, float* __restrict__ amerged,
                                                  HeadTables tb, MfmaTables mt) {
  constexpr int TPR = MR * NH / 4;            // threads a split row
  constexpr int G = 256 / TPR;                // split groups
  constexpr int SUB = 256 / NH;               // split groups of pass 1
  const int bj = blockIdx.x;                  // (sequence, slice) on x: grid x is wide
  const int rc = blockIdx.y;
  const int J = mt.n_slices;
  const int b = bj / J, slice = bj % J;
  const int tid = threadIdx.x;
  __shared__ float red[256];
  __shared__ float sM[NH], sInvL[NH];
  __shared__ float4 racc[256];
  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int ns = (T_b + split_tokens - 1) / split_tokens;
  const float* ml = part_ml + (int64_t(b) * J + slice) * n_split * (2 * NH);
  const float* pb = part + (int64_t(b) * J + slice) * n_split * int64_t(NH) * rv;

  // pass 1
  {
    const int h = tid % NH, sub = tid / NH;
    float mx = -INFINITY;
    int s = sub;
    for (; LONG && s + 31 * SUB < ns; s += 32 * SUB) {   // long merges: 32 loads in flight
      float v[32];
#pragma unroll
      for (int k = 0; k < 32; ++k) v[k] = ml[(s + k * SUB) * (2 * NH) + h];
#pragma unroll
      for (int k = 0; k < 32; ++k) mx = fmaxf(mx, v[k]);
    }
    for (; s + 7 * SUB < ns; s += 8 * SUB) {
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = ml[(s + k * SUB) * (2 * NH) + h];
#pragma unroll
      for (int k = 0; k < 8; ++k) mx = fmaxf(mx, v[k]);
    }
    for (; s < ns; s += SUB) mx = fmaxf(mx, ml[s * (2 * NH) + h]);
    red[tid] = mx;
    __syncthreads();
    if (tid < NH) {
      float M = -INFINITY;
      for (int k = 0; k < SUB; ++k) M = fmaxf(M, red[k * NH + tid]);
      sM[tid] = M;
    }
    __syncthreads();
    const float M = sM[h];
    float l = 0.f;
    if (M != -INFINITY) {
      s = sub;
      for (; LONG && s + 15 * SUB < ns; s += 16 * SUB) {   // long merges: 16 pairs in flight
        float mv[16], lv[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          mv[k] = ml[(s + k * SUB) * (2 * NH) + h];
          lv[k] = ml[(s + k * SUB) * (2 * NH) + NH + h];
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) l += exp2f(mv[k] - M) * lv[k];
      }
      for (; s + 7 * SUB < ns; s += 8 * SUB) {
        float mv[8], lv[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          mv[k] = ml[(s + k * SUB) * (2 * NH) + h];
          lv[k] = ml[(s + k * SUB) * (2 * NH) + NH + h];
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) l += exp2f(mv[k] - M) * lv[k];
      }
      for (; s < ns; s += SUB) l += exp2f(ml[s * (2 * NH) + h] - M) * ml[s * (2 * NH) + NH + h];
    }
    red[tid] = l;
    __syncthreads();
    if (tid < NH) {
      float L = 0.f;
      for (int k = 0; k < SUB; ++k) L += red[k * NH + tid];
      sInvL[tid] = L > 0.f ? 1.f / L : 0.f;
    }
    __syncthreads();
  }

  // pass 2
  const int g = tid / TPR, e = tid % TPR;
  const int rl = e / (NH / 4);                 // rank inside the chunk
  const int hq = (e % (NH / 4)) * 4;           // first of four head slots
  const int r = rc * MR + rl;
  const float4 M4 = make_float4(sM[hq], sM[hq + 1], sM[hq + 2], sM[hq + 3]);
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
  if (r < rv) {
    const float* src = pb + int64_t(r) * NH + hq;
    const int64_t stride = int64_t(NH) * rv;
    int s = g;
    for (; LONG && s + 15 * G < ns; s += 16 * G) {   // long merges: 16 splits in flight
      float4 mv[16], av[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        mv[k] = *reinterpret_cast<const float4*>(ml + (s + k * G) * (2 * NH) + hq);
        av[k] = *reinterpret_cast<const float4*>(src + (s + k * G) * stride);
      }
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        a.x = fmaf(exp2f(mv[k].x - M4.x), av[k].x, a.x);
        a.y = fmaf(exp2f(mv[k].y - M4.y), av[k].y, a.y);
        a.z = fmaf(exp2f(mv[k].z - M4.z), av[k].z, a.z);
        a.w = fmaf(exp2f(mv[k].w - M4.w), av[k].w, a.w);
      }
    }
    for (; s + 3 * G < ns; s += 4 * G) {
      float4 mv[4], av[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        mv[k] = *reinterpret_cast<const float4*>(ml + (s + k * G) * (2 * NH) + hq);
        av[k] = *reinterpret_cast<const float4*>(src + (s + k * G) * stride);
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        a.x = fmaf(exp2f(mv[k].x - M4.x), av[k].x, a.x);
        a.y = fmaf(exp2f(mv[k].y - M4.y), av[k].y, a.y);
        a.z = fmaf(exp2f(mv[k].z - M4.z), av[k].z, a.z);
        a.w = fmaf(exp2f(mv[k].w - M4.w), av[k].w, a.w);
      }
    }
    for (; s < ns; s += G) {
      const float4 mv = *reinterpret_cast<const float4*>(ml + s * (2 * NH) + hq);
      const float4 av = *reinterpret_cast<const float4*>(src + s * stride);
      a.x = fmaf(exp2f(mv.x - M4.x), av.x, a.x);
      a.y = fmaf(exp2f(mv.y - M4.y), av.y, a.y);
      a.z = fmaf(exp2f(mv.z - M4.z), av.z, a.z);
      a.w = fmaf(exp2f(mv.w - M4.w), av.w, a.w);
    }
  }
  racc[tid] = a;
  __syncthreads();
  if (g == 0 && r < rv) {
    float4 t = racc[e];
    for (int k = 1; k < G; ++k) {
      const float4 u = racc[k * TPR + e];
      t.x += u.x;
      t.y += u.y;
      t.z += u.z;
      t.w += u.w;
    }
    const float tv[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = mt.hord[slice][hq + k];           // query i * H_q + head h
      if (row >= 0)
        amerged[(int64_t(b) * tb.n_queries * tb.n_q_heads + row) * rv + r] =
            sM[hq + k] == -INFINITY ? 0.f : tv[k] * sInvL[hq + k];
    }
  }
}

template <int W, int NT, int MTW, int KR>
hipError_t launch_split(const dckv_plan& p, const DecodeShape& sh, const u32x4* qblk,
                        const void* pool, int64_t num_pages, const int32_t* page_table,
                        int32_t max_pages, const int32_t* seq_lens, float* part_ml, float* part,
                        size_t lds, hipStream_t stream, const bf16* pw = nullptr) {
  if (pw) {                               // the rotary decode's value pass
    if constexpr (KR == (((2 * MTW) % 16 == 0) ? 16 : 12)) {
      auto kern = split_mfma<W, NT, MTW, KR, true>;
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(kern, dim3(sh.n_units * p.mfma.n_slices), dim3(W * 64), lds, stream, qblk,
                         static_cast<const bf16*>(pool), num_pages, page_table, max_pages, seq_lens,
                         sh.max_context, sh.split_tokens, sh.n_split, sh.batch * sh.n_split, p.RK,
                         p.rv, p.page_elems, p.value_base, part_ml, part, p.mfma, pw);
      return hipGetLastError();
    }
    return hipErrorInvalidValue;
  }
  auto kern = split_mfma<W, NT, MTW, KR>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  const int grid = sh.n_units * p.mfma.n_slices;
  if (p.prof_before && p.prof_after)   // events stamped by the kernel's own dispatch
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(W * 64), uint32_t(lds), stream, p.prof_before,
                          p.prof_after, 0u, qblk, static_cast<const bf16*>(pool), num_pages,
                          page_table, max_pages, seq_lens, sh.max_context, sh.split_tokens,
                          sh.n_split, sh.batch * sh.n_split, p.RK, p.rv, p.page_elems,
                          p.value_base, part_ml, part, p.mfma, static_cast<const bf16*>(nullptr));
  else
    hipLaunchKernelGGL(kern, dim3(grid), dim3(W * 64), lds, stream, qblk,
                       static_cast<const bf16*>(pool), num_pages, page_table, max_pages, seq_lens,
                       sh.max_context, sh.split_tokens, sh.n_split, sh.batch * sh.n_split, p.RK,
                       p.rv, p.page_elems, p.value_base, part_ml, part, p.mfma,
                       static_cast<const bf16*>(nullptr));
  return hipGetLastError();
}

template <int W, int NT, int MTW>
hipError_t launch_split_r(const dckv_plan& p, const DecodeShape& sh, const u32x4* qt,
                          const void* pool, int64_t num_pages, const int32_t* page_table,
                          int32_t max_pages, const int32_t* seq_lens, float* part_ml, float* part,
                          size_t lds, hipStream_t stream) {
  if constexpr (MTW <= 12) {               // the plan mixes block sizes only here
    if (p.mfma.ring == 12)
      return launch_split<W, NT, MTW, 12>(p, sh, qt, pool, num_pages, page_table, max_pages,
                                          seq_lens, part_ml, part, lds, stream);
    if (p.mfma.ring == 14)
      return launch_split<W, NT, MTW, 14>(p, sh, qt, pool, num_pages, page_table, max_pages,
                                          seq_lens, part_ml, part, lds, stream);
  }
  if (p.mfma.ring != 16) return hipErrorInvalidValue;
  return launch_split<W, NT, MTW, 16>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens,
                                      part_ml, part, lds, stream);
}

template <int W, int NT>
hipError_t launch_split_w(const dckv_plan& p, const DecodeShape& sh, const u32x4* qt,
                          const void* pool, int64_t num_pages, const int32_t* page_table,
                          int32_t max_pages, const int32_t* seq_lens, float* part_ml, float* part,
                          size_t lds, hipStream_t stream) {
#define DCKV_SPLIT(M)                                                                   \
  return launch_split_r<W, NT, M>(p, sh, qt, pool, num_pages, page_table, max_pages, \
                                  seq_lens, part_ml, part, lds, stream)
  switch (p.mfma.mtw_t) {
    case 6: DCKV_SPLIT(6);
    case 8: DCKV_SPLIT(8);
    case 12: DCKV_SPLIT(12);
    case 16: DCKV_SPLIT(16);
    case 32: DCKV_SPLIT(NT == 1 ? 32 : 16);   // the plan takes 32 only with one head tile
  }
#undef DCKV_SPLIT
  return hipErrorInvalidValue;
}

// The rotary decode's value pass: the split kernel with weights from the
// workspace, its value ring block fixed by the value tiles a wave.
template <int W, int NT>
hipError_t launch_split_pw(const dckv_plan& p, const DecodeShape& sh, const void* pool,
                           int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                           const int32_t* seq_lens, float* part_ml, float* part, const bf16* pw,
                           size_t lds, hipStream_t stream) {
#define DCKV_PW(M)                                                                             \
  return launch_split<W, NT, M, ((2 * (M)) % 16 == 0 ? 16 : 12)>(                              \
      p, sh, nullptr, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, lds, \
      stream, pw)
  switch (p.mfma.mtw_t) {
    case 6: DCKV_PW(6);
    case 8: DCKV_PW(8);
    case 12: DCKV_PW(12);
    case 16: DCKV_PW(16);
    case 32: DCKV_PW(NT == 1 ? 32 : 16);
  }
#undef DCKV_PW
  return hipErrorInvalidValue;
}

// Merge of the splits' partials and the up-projection by R_v, shared by the
// position-free and the rotary decode.
hipError_t launch_merge_upproj(const dckv_plan& p, const DecodeShape& sh, const int32_t* seq_lens,
                               const float* part_ml, const float* part, float* amerged,
                               const void* R_value, float* out, hipStream_t stream) {
  // the deep-batch merge only for long split lists: its registers would cost
  // the short merges (many small work-groups) their occupancy
  const bool lng = sh.n_split >= 128;
  auto kern = sh.merge_ranks == 16
                  ? (p.mfma.nt == 1 ? (lng ? merge_mfma<16, true, 16> : merge_mfma<16, false, 16>)
                                    : (lng ? merge_mfma<32, true, 16> : merge_mfma<32, false, 16>))
                  : (p.mfma.nt == 1 ? (lng ? merge_mfma<16, true, 8> : merge_mfma<16, false, 8>)
                                    : (lng ? merge_mfma<32, true, 8> : merge_mfma<32, false, 8>));
  hipLaunchKernelGGL(kern, dim3(sh.batch * p.mfma.n_slices, sh.n_rchunks), dim3(256), 0, stream,
                     part_ml, part, seq_lens, sh.max_context, sh.split_tokens, sh.n_split, p.rv,
                     amerged, p.tables, p.mfma);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_upproj(p, sh.batch * p.Q, amerged, R_value, out, stream);
}

}  // namespace

hipError_t launch_fold(const dckv_plan& p, const MfmaTables& mt, int32_t batch, const float* q,
                       const void* R_keys, void* qblk, hipStream_t stream) {
  const float scale = kLog2e / std::sqrt(float(p.dh));
  // d_h 64 or 128: one wave a (slice, slot, chunk) for all sequences, on
  // MFMA; other head sizes: one wave a (sequence, slice, slot, chunk)
  if (p.dh == 64 || p.dh == 128) {
    auto kern = p.dh == 64 ? fold_mfma<2> : fold_mfma<4>;
    const int ngrp = mt.n_slices * mt.max_pairs;
    hipLaunchKernelGGL(kern, dim3(8 * 16 * ((ngrp + 7) / 8)), dim3(64), 0, stream, q,
                       static_cast<const bf16*>(R_keys), static_cast<u32x4*>(qblk), batch, scale,
                       p.tables, mt);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(fold_blocks, dim3(batch * mt.n_slices, 16, mt.max_pairs), dim3(64), 0, stream, q,
                     static_cast<const bf16*>(R_keys), static_cast<u32x4*>(qblk), scale, p.tables,
                     mt);
  return hipGetLastError();
}

size_t mfma_split_lds_bytes(const dckv_plan& p) {
  return size_t(p.mfma.max_pairs) * 2048 + 32 * kPStride * 2 + 2 * 8 * 32 * 4 + kPageSlots * 4;
}

int mfma_merge_ranks(const dckv_plan& p, int32_t batch) {
  const int64_t groups = int64_t(batch) * p.mfma.n_slices * ((p.rv + kMergeRanks - 1) / kMergeRanks);
  return groups >= 2048 ? 2 * kMergeRanks : kMergeRanks;
}

int mfma_max_split_tokens() { return kPageSlots * DCKV_PAGE_TOKENS; }

hipError_t launch_decode_mfma(const dckv_plan& p, const DecodeShape& sh, const float* q,
                              const void* pool, int64_t num_pages, const int32_t* page_table,
                              int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                              const void* R_value, float* out, void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  u32x4* qt = reinterpret_cast<u32x4*>(ws + sh.off_qt);
  float* part_ml = reinterpret_cast<float*>(ws + sh.off_ml);
  float* part = reinterpret_cast<float*>(ws + sh.off_acc);
  float* amerged = reinterpret_cast<float*>(ws + sh.off_opart);
  const size_t lds = mfma_split_lds_bytes(p);
  hipError_t e = launch_fold(p, p.mfma, sh.batch, q, R_keys, qt, stream);
  if (e != hipSuccess) return e;
  if (p.mfma.waves == 4)
    e = p.mfma.nt == 1
            ? launch_split_w<4, 1>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, lds, stream)
            : launch_split_w<4, 2>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, lds, stream);
  else
    e = p.mfma.nt == 1
            ? launch_split_w<8, 1>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, lds, stream)
            : launch_split_w<8, 2>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, lds, stream);
  if (e != hipSuccess) return e;
  return launch_merge_upproj(p, sh, seq_lens, part_ml, part, amerged, R_value, out, stream);
}

size_t rope_value_lds_bytes(const dckv_plan& p, int32_t split_tokens) {
  // the split kernel's fixed carve-up without query blocks, then the weights
  return size_t(32) * kPStride * 2 + 2 * 8 * 32 * 4 + kPageSlots * 4 +
         size_t(16) * p.mfma.nt * (split_tokens + 8) * 2;
}

hipError_t launch_decode_rope(const dckv_plan& p, const DecodeShape& sh, const float* q,
                              const void* pool, int64_t num_pages, const int32_t* page_table,
                              int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                              const void* R_value, double rope_base, float* out, void* workspace,
                              hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  void* rt = ws + sh.off_rt;
  bf16* pw = reinterpret_cast<bf16*>(ws + sh.off_p);
  float* part_ml = reinterpret_cast<float*>(ws + sh.off_ml);
  float* part = reinterpret_cast<float*>(ws + sh.off_acc);
  float* amerged = reinterpret_cast<float*>(ws + sh.off_opart);
  hipError_t e = launch_rope_factors(p, R_keys, rt, stream);
  if (e != hipSuccess) return e;
  e = launch_rope_scores(p, sh, q, pool, num_pages, page_table, max_pages, seq_lens, rt, rope_base,
                         pw, part_ml, stream);
  if (e != hipSuccess) return e;
  const size_t lds = rope_value_lds_bytes(p, sh.split_tokens);
  if (p.mfma.waves == 4)
    e = p.mfma.nt == 1
            ? launch_split_pw<4, 1>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, pw, lds, stream)
            : launch_split_pw<4, 2>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, pw, lds, stream);
  else
    e = p.mfma.nt == 1
            ? launch_split_pw<8, 1>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, pw, lds, stream)
            : launch_split_pw<8, 2>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, part_ml, part, pw, lds, stream);
  if (e != hipSuccess) return e;
  return launch_merge_upproj(p, sh, seq_lens, part_ml, part, amerged, R_value, out, stream);
}

}  // namespace dckv
