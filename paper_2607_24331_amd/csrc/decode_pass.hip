// Two-pass bf16 decode on MFMA (gfx950) for one query a sequence and at most
// 32 query heads.  The same attention as split_mfma (Sec. III-A: scores
// against the key latents with the query folded into each group's latent
// space, Sec. III-C; the weighted sum kept in value-latent space, Sec.
// III-D), with the work cut so that no pass writes per-split partials of
// the whole value rank:
//
// score_pages: one work-group per (sequence, range of pages); each wave takes
//   its own pages, with no barrier between waves.  Per 64-token page and
//   16-head tile: S = Z_K q~^T on MFMA (q~ as bf16 hi + lo parts, fp32
//   accumulate), then the page's own softmax weights relative to an integer
//   exponent e = ceil(max_t S): p_t = 2^(S_t - e) rounded to bf16, and
//   l = sum_t p_t (of the rounded weights).  Weights go out in the value
//   MFMA's operand order, (e, l) beside them.
// value_pages: one work-group per (sequence, context chunk, group of 16-rank
//   value tiles); each wave takes its own pages of the chunk and accumulates
//   acc^T[rank][head] += Z_v^T p' on MFMA, where p' = p 2^(e - E) rescales a
//   page's weights to the wave's running exponent E.  Exponents are
//   integers, so every rescaling (of weights, sums and accumulators) is an
//   exact power of two.  The waves' accumulators are combined in a fixed
//   order.  Partials: (E, L) and acc of the chunk's rank group.
// merge_chunks: the chunks of each (sequence, head) merged in ascending order
//   into the normalised value-latent row a_h.
// upproj_wide / upproj_rows / upproj_mfma: o_h = a_h R_v[:, kv(h) block]
//   (Sec. III-A z R, Sec. III-D R_v), by the number of rows a KV head.
#include <algorithm>
#include <cmath>

#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer descriptor on gfx9-family parts (32-bit data
// format, no swizzle); loads at or past num_records return zero.
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kOutOfRange = 0x40000000;   // byte offset beyond any page
constexpr int kNonTemporal = 2;           // cache policy of streamed latents: nt
constexpr int kMaxChunkPages = 512;       // pages of a value chunk: 64 a wave
constexpr int kMaxSharedChunkPages = 64;  // pages of a chunk walked by all waves together
constexpr int kScoreMinLds = 82 * 1024;   // one score work-group a compute unit
constexpr int kQblkLoads = 20;            // folded-query loads a thread: 80 blocks (the LDS limit)

__device__ __forceinline__ floatx4 mfma(u32x4 a, u32x4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
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

// 2^(e - E) for integer-valued e <= E (E finite whenever e is): an exact
// power of two, 0 for e = -inf.
__device__ __forceinline__ float pow2_rel(float e, float E) {
  return e == -INFINITY ? 0.f : ldexpf(1.f, int(fmaxf(e - E, -256.f)));
}

// Eight bf16 times f, f a power of two or zero: exact, so the truncation
// back to bf16 is the exact product.
__device__ __forceinline__ u32x4 scale8(u32x4 v, float f) {
  u32x4 r;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const float lo = __uint_as_float(v[d] << 16) * f;
    const float hi = __uint_as_float(v[d] & 0xFFFF0000u) * f;
    r[d] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
  }
  return r;
}

// ---------------------------------------------------------------------------
// Score pass.  Work-group u: sequence u / units_per_seq, pages
// [ur * kUnitPages, (ur + 1) * kUnitPages) of it.  The eight waves serve
// PP = 2 / NT pages at a time: wave w takes head tile n = (w / 4) % NT and
// 16-token row block m = w % 4 of pages pl, pl + PP, ... (pl = w / (4 NT)),
// so the waves of a work-group stream the same pages side by side.  A
// wave's items are, page after page, the 1 KB operands of its 16 tokens in
// the key chunks of its tile's groups; a ring of RING loads runs ahead
// across page boundaries.  Each wave keeps its pages' weights in LDS,
// relative to the integer exponent of its 16 tokens; once every page is
// scored, the work-group's exponent of a row is e = ceil(max over the unit's
// scores) (the largest of those), and each wave writes its weights rescaled
// to it by exact powers of two.  One exponent for the unit's pages lets the
// value pass use the weights as stored, rescaling its accumulators only
// where the exponent changes.
//
// With several queries a sequence the rows are cut into J slices (as for
// the single-pass kernel): work-group (unit, slice) loads the key chunks of
// its slice's groups, and a row of query i sees positions before
// T_b - Q + i + 1.
//
// Outputs per (sequence b, page pg of it): a block of RT x 2560 bytes (RT =
// J NT row tiles) at (b * npm + pg) * RT * 2560 holding, for row tile t =
// slice * NT + n,
//   at t * 2 KB: the weights as the value MFMA's B operand, 16 rows x 64
//          tokens: k-step ks (tokens 32ks..32ks+31) at ks * 1024 bytes, lane
//          L = 16 * (token%32 / 8) + row at L * 16, 8 tokens a lane
//   at RT * 2 KB + t * 512: e and l of row slot j and row block m at floats
//          8j + m and 8j + 4 + m: e the unit's exponent of the row (the same
//          for every block and page of the unit; -inf for a row with no
//          visible token in the unit), l the sum of the block's weights as
//          stored
template <int NT, int RING, bool MASK>
__global__ __launch_bounds__(512, 1) void score_pages(
    const u32x4* __restrict__ qblk_ws, const bf16* __restrict__ pool, int64_t num_pages,
    const int32_t* __restrict__ page_table, int max_pages, const int32_t* __restrict__ seq_lens,
    int max_context, int units_per_seq, int n_units, int npm, int RK, int64_t page_elems,
    uint32_t* __restrict__ pw, MfmaTables mt) {
  constexpr int PP = 2 / NT;                   // pages side by side
  constexpr int unit_pages = kUnitPages;
  extern __shared__ __align__(16) unsigned char smem[];
  // the J slices of a page range run side by side on one XCD (block ids
  // equal mod 8), so a key chunk two slices load comes the second time from
  // that XCD's L2
  const int J = mt.n_slices;
  const int qd = blockIdx.x >> 3, slice = qd % J;
  const int u = 8 * (qd / J) + (blockIdx.x & 7);
  if (u >= n_units) return;
  const int b = u / units_per_seq, ur = u - b * units_per_seq;
  const int RT = J * NT;                       // row tiles of a page's outputs
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;
  const int pl = w / (4 * NT), n = (w >> 2) % NT, m = w & 3;

  // The prologue's loads go out together, none waiting on another: the
  // wave's page-table entries (lane i: its i-th page), the folded-query
  // blocks, the context length.  Nothing before the ring's first issue
  // depends on the context length, and a work-group past its sequence's end
  // does no work but does not leave early, so that no branch holds a load
  // back.
  const int p0 = ur * unit_pages;
  const int pt = page_table[int64_t(b) * max_pages + min(p0 + pl + PP * lane, max_pages - 1)];
  const int nch0 = mt.kln[slice][0][0] + mt.kln[slice][0][1];
  const int npairs = nch0 + (NT > 1 ? mt.kln[slice][1][0] + mt.kln[slice][1][1] : 0);
  u32x4* qblk = reinterpret_cast<u32x4*>(smem);                // [npairs][2][64]
  const u32x4* qsrc = qblk_ws + (int64_t(b) * J + slice) * mt.max_pairs * 128;
  const int n16 = npairs * 128;
  u32x4 qv[kQblkLoads];
#pragma unroll
  for (int k = 0; k < kQblkLoads; ++k) qv[k] = qsrc[min(tid + 512 * k, n16 - 1)];
  int T_b = seq_lens[b];

  const int st0 = mt.kst[slice][n][0], ln0 = mt.kln[slice][n][0], st1 = mt.kst[slice][n][1];
  const int nch = ln0 + mt.kln[slice][n][1];   // key chunks of this wave's tile
  // this lane's row (query i, head h) sees positions before T_b - Q + i + 1
  const int hrow = mt.hord[slice][16 * n + lr];
  const int pair0 = n ? nch0 : 0;
  // lane i: the physical page of this wave's i-th page (-1: invalid)
  const int pid_tbl = (pt >= 0 && pt < num_pages) ? pt : -1;

  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int np = (T_b + 63) >> 6;
  const int p1 = min(np, p0 + unit_pages);
  const int nmine = max(0, (p1 - p0 - pl + PP - 1) / PP);       // this wave's pages (<= 8)
  const int total = nmine * nch;
  const int lim = hrow < 0 ? 0 : T_b - mt.queries + hrow / mt.q_heads + 1;

  const int page_bytes = int(page_elems * 2);
  const int lane_key = 2 * (lr * 32 + 8 * lq) + 2 * 512 * m;
  const int kc_last = (RK - 1) >> 5;
  const int kvalid_last = min(8, max(0, RK - (32 * kc_last + 8 * lq)));

  // producer: page prod_k of this wave, chunk prod_c of the tile's list
  int prod_k = 0, prod_c = 0;
  __amdgpu_buffer_rsrc_t prod_rsrc;
  auto set_page = [&](int k) {
    const int pid = __builtin_amdgcn_readlane(pid_tbl, min(k, 63));
    const bool ok = k < nmine && pid >= 0;
    prod_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(ok ? pool + int64_t(pid) * page_elems : pool), 0, ok ? page_bytes : 0,
        kRsrcWord3);
  };
  set_page(0);
  // every call issues exactly one load (past the wave's last page the
  // descriptor covers nothing and the load reads zero), so the number of
  // loads in flight is the same on every path and each wait is for one slot
  auto issue = [&]() -> u32x4 {
    if (prod_c == nch) {
      prod_c = 0;
      set_page(++prod_k);
    }
    const int c = prod_c < ln0 ? st0 + prod_c : st1 + (prod_c - ln0);
    ++prod_c;
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                         prod_rsrc, 2 * 2048 * c + lane_key, 0, kNonTemporal));
  };

  u32x4 ring[RING];
#pragma unroll
  for (int s = 0; s < RING; ++s) ring[s] = issue();

  if (p1 > p0) {
#pragma unroll
    for (int k = 0; k < kQblkLoads; ++k)
      if (tid + 512 * k < n16) qblk[tid + 512 * k] = qv[k];
  }
  __syncthreads();

  int con_k = 0, con_c = 0;
  floatx4 S = floatx4{0.f, 0.f, 0.f, 0.f};
  u32x4 bhi = qblk[(pair0 * 2 + 0) * 64 + lane], blo = qblk[(pair0 * 2 + 1) * 64 + lane];

  // LDS after the query blocks: per wave and page (at most kUnitPages) the
  // weights, 8 bytes a lane, then per wave, page and row the exponent and sum
  const size_t stage0 = size_t(mt.max_pairs) * 2048;
  uint2* pst = reinterpret_cast<uint2*>(smem + stage0) + w * kUnitPages * 64;
  float* est = reinterpret_cast<float*>(smem + stage0 + 8 * kUnitPages * 512);
  float* lst = est + 8 * kUnitPages * 16;
  if (lq == 0) {
#pragma unroll
    for (int k = 0; k < kUnitPages; ++k) est[(w * kUnitPages + k) * 16 + lr] = -INFINITY;
  }

  // the weights of this wave's 16 tokens of page k, from S, relative to
  // their own exponent, into LDS
  auto epilogue = [&](int k) {
    const int pg = p0 + pl + PP * k;
    const bool pvalid = __builtin_amdgcn_readlane(pid_tbl, min(k, 63)) >= 0;
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int t = 64 * pg + 16 * m + 4 * lq + v;     // position; t < lim <= T_b
      if (!pvalid || t >= lim) S[v] = -INFINITY;
      mx = fmaxf(mx, S[v]);
    }
    mx = wave_max16(mx);
    const float e = mx == -INFINITY ? -INFINITY : ceilf(mx);
    float psum = 0.f;
    uint32_t pk[2];
#pragma unroll
    for (int v2 = 0; v2 < 2; ++v2) {
      uint32_t word = 0;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const float sc = S[2 * v2 + hf];
        const float pv = sc == -INFINITY ? 0.f : exp2f(sc - e);
        const bf16 pb = static_cast<bf16>(pv);
        psum += static_cast<float>(pb);
        word |= uint32_t(__builtin_bit_cast(uint16_t, pb)) << (16 * hf);
      }
      pk[v2] = word;
    }
    pst[k * 64 + lane] = uint2{pk[0], pk[1]};
    psum = wave_sum16(psum);
    if (lq == 0) {
      est[(w * kUnitPages + k) * 16 + lr] = e;
      lst[(w * kUnitPages + k) * 16 + lr] = psum;
    }
    S = floatx4{0.f, 0.f, 0.f, 0.f};
  };

  auto consume = [&](u32x4 a) {
    const int c = con_c < ln0 ? st0 + con_c : st1 + (con_c - ln0);
    // MASK: R_K is not a multiple of 32, so the last key chunk holds padding
    // columns (zero when written by the append, but masked all the same);
    // without it the check and its selects are compiled out
    if (MASK && c == kc_last) a = keep_first(a, kvalid_last);
    S = mfma(a, bhi, S);
    S = mfma(a, blo, S);
    // the next item's query blocks
    const int cn = con_c + 1 == nch ? 0 : con_c + 1;
    bhi = qblk[((pair0 + cn) * 2 + 0) * 64 + lane];
    blo = qblk[((pair0 + cn) * 2 + 1) * 64 + lane];
    if (++con_c == nch) {
      epilogue(con_k);
      con_c = 0;
      ++con_k;
    }
  };
  // whole ring blocks: every slot consumed, then reloaded
  int base = 0;
  for (; base + RING <= total; base += RING) {
#pragma unroll
    for (int s = 0; s < RING; ++s) {
      consume(ring[s]);
      ring[s] = issue();
    }
  }
  // the last, partial block: nothing left to load
#pragma unroll
  for (int s = 0; s < RING; ++s)
    if (base + s < total) consume(ring[s]);

  // the unit's exponent of this lane's row: the largest over the waves of
  // its tile and their pages
  __syncthreads();
  float eu = -INFINITY;
#pragma unroll
  for (int ww = 0; ww < 8; ++ww) {
    if (((ww >> 2) % NT) == n) {
#pragma unroll
      for (int k = 0; k < kUnitPages; ++k) eu = fmaxf(eu, est[(ww * kUnitPages + k) * 16 + lr]);
    }
  }
  // this wave's pages, rescaled to it: tokens 16m + 4lq .. +3 go to k-step
  // m/2, operand lane 16 * (2(m%2) + lq/2) + lr
  const int L = 16 * (2 * (m & 1) + (lq >> 1)) + lr;
  for (int k = 0; k < nmine; ++k) {
    const int pg = p0 + pl + PP * k;
    const float ep = est[(w * kUnitPages + k) * 16 + lr];
    const float f = pow2_rel(ep, eu);                  // 0 for a page with no visible token
    const uint2 v = pst[k * 64 + lane];
    uint32_t pk[2] = {v.x, v.y};
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const float lo = __uint_as_float(pk[d] << 16) * f;
      const float hi = __uint_as_float(pk[d] & 0xFFFF0000u) * f;
      pk[d] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
    }
    uint32_t* pblk = pw + (int64_t(b) * npm + pg) * RT * 640;   // 2560 bytes a row tile
    const int ti = slice * NT + n;
    *reinterpret_cast<uint2*>(pblk + ti * 512 + (m >> 1) * 256 + L * 4 + 2 * (lq & 1)) =
        uint2{pk[0], pk[1]};
    if (lq == 0) {
      float* rec = reinterpret_cast<float*>(pblk + RT * 512 + ti * 128);
      rec[8 * lr + m] = eu;
      rec[8 * lr + 4 + m] = lst[(w * kUnitPages + k) * 16 + lr] * f;
    }
  }
}

// ---------------------------------------------------------------------------
// Value pass.  Work-group (sequence b, chunk c, rank group g): the pages
// [c * chunk_pages, (c + 1) * chunk_pages) of b, value tiles [g * RGT,
// (g + 1) * RGT); wave w takes pages w, w + W, ... of the chunk.  A page's
// items, one ring block: per head tile the (e, l) records of the lane's head
// (two 16-byte loads), the weight operands (two k-steps a head tile), then
// the RGT x 2 value operands (16 ranks x 32 tokens each).  The n_rg
// work-groups of one (sequence, chunk) share an XCD (ids equal mod 8), so
// the weights they all read come from that XCD's L2.
//
// Partials per (sequence, chunk): vel [2][NH] (E, L) written by rank group
// 0, vpart [NH][r_v] the chunk's sums relative to 2^E.
template <int W, int NT, int RGT>
__global__ __launch_bounds__(W * 64, 1) void value_pages(
    const bf16* __restrict__ pool, int64_t num_pages, const int32_t* __restrict__ page_table,
    int max_pages, const int32_t* __restrict__ seq_lens, int max_context, int chunk_pages,
    int n_chunks, int n_rg, int batch, int npm, int rv, int mt_v, int64_t page_elems,
    int64_t value_base, const u32x4* __restrict__ pw, float* __restrict__ vpart,
    float* __restrict__ vel) {
  constexpr int NH = 16 * NT;
  constexpr int P0 = 2 * NT;                        // first weight item
  constexpr int V0 = 4 * NT;                        // first value item
  constexpr int IPP = V0 + 2 * RGT;                 // items a page
  extern __shared__ __align__(16) unsigned char smem[];
  const int L = blockIdx.x;
  const int xcd = L & 7, qd = L >> 3;
  const int rg = qd % n_rg;
  const int cidx = 8 * (qd / n_rg) + xcd;          // sequence * n_chunks + chunk
  if (cidx >= batch * n_chunks) return;
  const int b = cidx / n_chunks, chunk = cidx - b * n_chunks;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;

  // the page-table entries (lane i: this wave's i-th page) and the context
  // length are loaded together
  const int g0 = chunk * chunk_pages;
  const int pt = page_table[int64_t(b) * max_pages + min(g0 + w + W * lane, max_pages - 1)];
  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int np = (T_b + 63) >> 6;
  // a chunk past the sequence's end has no pages and writes nothing (the
  // merge reads chunks holding tokens only); its work-group does not leave
  // early, so that no branch holds the loads above back
  const int g1 = min(np, g0 + chunk_pages);
  const int nmine = max(0, (g1 - g0 - w + W - 1) / W);   // this wave's pages (<= 64)
  const int mt0 = rg * RGT;
  const int pid_tbl = (pt >= 0 && pt < num_pages) ? pt : -1;   // -1: invalid

  const int page_bytes = int(page_elems * 2);
  const int lane_val = 2 * (lr * 32 + 8 * lq);
  const int64_t seq_page0 = int64_t(b) * npm;

  // producer: page k of this wave, items s = 0 .. IPP-1 (slot = item)
  __amdgpu_buffer_rsrc_t prsrc;
  int ppg = 0, pnval = 0;
  auto set_page = [&](int k) {
    const int pid = __builtin_amdgcn_readlane(pid_tbl, min(k, 63));
    const bool ok = k < nmine && pid >= 0;
    ppg = k < nmine ? g0 + w + W * k : g0;        // past the wave's pages: a valid page, unused
    pnval = k < nmine ? min(64, T_b - 64 * ppg) : 0;
    prsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(ok ? pool + int64_t(pid) * page_elems : pool), 0, ok ? page_bytes : 0,
        kRsrcWord3);
  };
  auto issue = [&](int s) -> u32x4 {
    const u32x4* pblk = pw + (seq_page0 + ppg) * NT * 160;
    if (s < P0) return pblk[NT * 128 + (s >> 1) * 32 + 2 * lr + (s & 1)];
    if (s < V0) {
      const int n = (s - P0) >> 1, ks = (s - P0) & 1;
      return pblk[n * 128 + ks * 64 + lane];
    }
    const int i = (s - V0) >> 1, ks = (s - V0) & 1;
    const int o = 2 * (int(value_base) + 1024 * (mt0 + i) + 512 * ks) + lane_val;
    const bool ok = (mt0 + i < mt_v) & (16 * (mt0 + i) + lr < rv) & (32 * ks + 8 * lq < pnval);
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                         prsrc, ok ? o : kOutOfRange, 0, kNonTemporal));
  };

  u32x4 ring[IPP];
  set_page(0);
#pragma unroll
  for (int s = 0; s < IPP; ++s) ring[s] = issue(s);

  floatx4 acc[RGT][NT];
#pragma unroll
  for (int i = 0; i < RGT; ++i)
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};
  float E_run[NT], L_run[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    E_run[n] = -INFINITY;
    L_run[n] = 0.f;
  }

  for (int k = 0; k < nmine; ++k) {
    const int pg = g0 + w + W * k;
    const int nval = min(64, T_b - 64 * pg);
    set_page(k + 1);                    // the next page's loads go into each slot as it is consumed
    float fks[NT][2];                   // weight scale of this lane's tokens, per head tile and k-step
    {
      bool resc = false;
      float fa[NT];
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const float4 ev = __builtin_bit_cast(float4, ring[2 * n]);       // (e0, e1, e2, e3)
        const float4 lv = __builtin_bit_cast(float4, ring[2 * n + 1]);   // (l0, l1, l2, l3)
        const float em = fmaxf(fmaxf(ev.x, ev.y), fmaxf(ev.z, ev.w));
        const float En = fmaxf(E_run[n], em);
        fa[n] = E_run[n] == -INFINITY ? 1.f : pow2_rel(E_run[n], En);
        const float f0 = pow2_rel(ev.x, En), f1 = pow2_rel(ev.y, En);
        const float f2 = pow2_rel(ev.z, En), f3 = pow2_rel(ev.w, En);
        L_run[n] = L_run[n] * fa[n] + (((lv.x * f0 + lv.y * f1) + lv.z * f2) + lv.w * f3);
        E_run[n] = En;
        // lane quarter lq holds tokens 32 ks + 8 lq ..: row block 2 ks + lq / 2
        fks[n][0] = (lq >> 1) ? f1 : f0;
        fks[n][1] = (lq >> 1) ? f3 : f2;
        resc = resc || fa[n] != 1.f;
      }
      if (__any(resc)) {
#pragma unroll
        for (int i = 0; i < RGT; ++i)
#pragma unroll
          for (int n = 0; n < NT; ++n) acc[i][n] *= fa[n];
      }
#pragma unroll
      for (int s = 0; s < P0; ++s) ring[s] = issue(s);
    }
    u32x4 pB[NT][2];
#pragma unroll
    for (int s = P0; s < V0; ++s) {
      const int n = (s - P0) >> 1, ks = (s - P0) & 1;
      pB[n][ks] = scale8(ring[s], fks[n][ks]);
      ring[s] = issue(s);
    }
    const int keep0 = min(8, max(0, nval - 8 * lq));
    const int keep1 = min(8, max(0, nval - 32 - 8 * lq));
#pragma unroll
    for (int s = V0; s < IPP; ++s) {
      const int i = (s - V0) >> 1, ks = (s - V0) & 1;
      u32x4 a = ring[s];
      if (nval < 64) a = keep_first(a, ks ? keep1 : keep0);
#pragma unroll
      for (int n = 0; n < NT; ++n) acc[i][n] = mfma(a, pB[n][ks], acc[i][n]);
      ring[s] = issue(s);
    }
  }

  // ---- combine the waves in a fixed order
  float* sE = reinterpret_cast<float*>(smem);                       // [W][NH]
  float* sL = sE + W * NH;                                          // [W][NH]
  floatx4* red = reinterpret_cast<floatx4*>(sL + W * NH);           // [W][RGT][NT][64]
  if (lq == 0) {
#pragma unroll
    for (int n = 0; n < NT; ++n) sE[w * NH + 16 * n + lr] = E_run[n];
  }
  __syncthreads();
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    float Eg = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < W; ++ww) Eg = fmaxf(Eg, sE[ww * NH + 16 * n + lr]);
    const float f = pow2_rel(E_run[n], Eg);
    L_run[n] *= f;
#pragma unroll
    for (int i = 0; i < RGT; ++i) acc[i][n] *= f;
    if (lq == 0) sL[w * NH + 16 * n + lr] = L_run[n];
  }
#pragma unroll
  for (int i = 0; i < RGT; ++i)
#pragma unroll
    for (int n = 0; n < NT; ++n) red[((w * RGT + i) * NT + n) * 64 + lane] = acc[i][n];
  __syncthreads();
  if (g0 >= g1) return;
  float* vp = vpart + int64_t(cidx) * NH * rv;
  for (int e = tid; e < RGT * NT * 64; e += W * 64) {
    floatx4 t = red[e];
#pragma unroll
    for (int ww = 1; ww < W; ++ww) t += red[ww * RGT * NT * 64 + e];
    const int ln = e & 63, n = (e >> 6) % NT, i = (e >> 6) / NT;
    const int head = 16 * n + (ln & 15);
    const int r0 = 16 * (mt0 + i) + 4 * (ln >> 4);
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (r0 + v < rv) vp[int64_t(head) * rv + r0 + v] = t[v];
  }
  if (rg == 0 && tid < NH) {
    float Eg = -INFINITY, Lg = 0.f;
    for (int ww = 0; ww < W; ++ww) Eg = fmaxf(Eg, sE[ww * NH + tid]);
    for (int ww = 0; ww < W; ++ww) Lg += sL[ww * NH + tid];
    vel[int64_t(cidx) * 2 * NH + tid] = Eg;
    vel[int64_t(cidx) * 2 * NH + NH + tid] = Lg;
  }
}

// ---------------------------------------------------------------------------
// Value pass for several row slices (several queries a sequence).  Work-group
// (sequence b, chunk c, rank group g): the W waves walk the chunk's pages
// together, wave w owning value tiles g * W * RGTW + w * RGTW .. + RGTW - 1
// against all RT row tiles, so each value latent byte is read once.  A
// page's weights and records are staged in LDS as stored (two buffers, one
// barrier a page); a wave's value loads and the next page's staging loads
// run DP pages ahead.  The weights of a row are relative to 2^e, e its exponent on
// that page (one for all pages of a score unit).  A wave keeps per row slot
// a base exponent B, its accumulators and the sum L being relative to 2^B:
// a page with another exponent moves B to it, the accumulators and L
// multiplied by 2^(B_old - B), an exact power of two above or below 1.  B
// stays within 64 of the largest exponent met, so the accumulators stay far
// from overflow: a page whose exponent is further below (all its weights
// under 2^-64 of the row's largest) is left out for that row, its weights
// zeroed in LDS before use.  All waves take the same B from the same
// records.
// Partials as value_pages, over NS = 16 RT row slots; no sums across waves.
template <int W, int RTMAX, int RGTW, int DP>
__global__ __launch_bounds__(W * 64, 1) void value_shared(
    const bf16* __restrict__ pool, int64_t num_pages, const int32_t* __restrict__ page_table,
    int max_pages, const int32_t* __restrict__ seq_lens, int max_context, int chunk_pages,
    int n_chunks, int n_rg, int batch, int npm, int rv, int mt_v, int64_t page_elems,
    int64_t value_base, int RT, const u32x4* __restrict__ pw, float* __restrict__ vpart,
    float* __restrict__ vel) {
  constexpr int NTH = W * 64;
  // launched with RT = RTMAX only (the plan's row-tile count picks the
  // instantiation); the check also lets the compiler take the count as
  // fixed, which keeps the page loop free of spills
  if (RT != RTMAX) return;
  constexpr int IP = 2 * RGTW;                      // value loads a page a wave
  constexpr int SV = (RTMAX * 160 + NTH - 1) / NTH; // staged 16-byte loads a thread a page
  extern __shared__ __align__(16) unsigned char smem[];
  const int Lb = blockIdx.x;
  const int xcd = Lb & 7, qd = Lb >> 3;
  const int rg = qd % n_rg;
  const int cidx = 8 * (qd / n_rg) + xcd;          // sequence * n_chunks + chunk
  if (cidx >= batch * n_chunks) return;
  const int b = cidx / n_chunks, chunk = cidx - b * n_chunks;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;
  const int NS = 16 * RT;

  // lane i: the physical page of the chunk's i-th page (chunk_pages <= 64)
  const int g0 = chunk * chunk_pages;               // < npm
  const int pt = page_table[int64_t(b) * max_pages + min(g0 + lane, max_pages - 1)];
  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int np = (T_b + 63) >> 6;
  const int npg = max(0, min(np, g0 + chunk_pages) - g0);   // the chunk's pages
  const int last = max(npg - 1, 0);
  const int pid_tbl = (pt >= 0 && pt < num_pages) ? pt : -1;
  const int mt0 = rg * W * RGTW + w * RGTW;          // this wave's first value tile

  // a staged page: weights [RT][2][64] then records [NS][8] (e0..e3, l0..l3)
  const int nst = RT * 160;
  u32x4* lbuf = reinterpret_cast<u32x4*>(smem);     // two pages
  // the sequence's weight blocks (RT * 2560 bytes a page) through a buffer
  // descriptor: one offset register a staged item, the page in soffset
  const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(pw + int64_t(b) * npm * RT * 160), 0, npm * RT * 2560, kRsrcWord3);
  // the holder of a slot's l record keeps the slot's base exponent, largest
  // exponent and sum (the same rule as the waves', on the same records)
  float sB[SV], sE[SV], sL[SV];
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    sB[k] = -INFINITY;
    sE[k] = -INFINITY;
    sL[k] = 0.f;
  }
  auto stage_item = [&](int k, int pg) -> u32x4 {   // pg < npm
    const int i = min(tid + NTH * k, nst - 1);
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(prs, 16 * i, pg * RT * 2560, 0));
  };
  auto stage_store = [&](const u32x4* sv, int buf) {
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      const int i = tid + NTH * k;
      // element i ^ 1 is held by lane ^ 1: for an l record, the e record
      const float ep = __shfl_xor(__uint_as_float(sv[k].x), 1);
      if (i < nst) {
        lbuf[buf * nst + i] = sv[k];
        if (i >= RT * 128 && (i & 1) && ep != -INFINITY) {
          const float4 lv = __builtin_bit_cast(float4, sv[k]);
          const float sum = (lv.x + lv.y) + (lv.z + lv.w);
          if (ep == sB[k]) {
            sL[k] += sum;
          } else {
            const float em = fmaxf(sE[k], ep);
            if (ep >= em - 64.f) {
              const float fa = sB[k] == -INFINITY ? 1.f : pow2_rel(sB[k], ep);
              sL[k] = sL[k] * fa + sum;
              sB[k] = ep;
              sE[k] = em;
            }
          }
        }
      }
    }
  };

  const int page_bytes = int(page_elems * 2);
  const int lane_val = 2 * (lr * 32 + 8 * lq);
  __amdgpu_buffer_rsrc_t rsrc;
  int pnval = 0;
  auto set_page = [&](int k) {                      // value loads of the chunk's page k
    const int pid = __builtin_amdgcn_readlane(pid_tbl, min(k, 63));
    const bool ok = k < npg && pid >= 0;
    pnval = k < npg ? min(64, T_b - 64 * (g0 + k)) : 0;
    rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(ok ? pool + int64_t(pid) * page_elems : pool), 0, ok ? page_bytes : 0,
        kRsrcWord3);
  };
  auto issue = [&](int s) -> u32x4 {                // item s: value tile s / 2, k-step s % 2
    const int i = s >> 1, ks = s & 1;
    const int o = 2 * (int(value_base) + 1024 * (mt0 + i) + 512 * ks) + lane_val;
    const bool ok = (mt0 + i < mt_v) & (16 * (mt0 + i) + lr < rv) & (32 * ks + 8 * lq < pnval);
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                         rsrc, ok ? o : kOutOfRange, 0, kNonTemporal));
  };

  // ring slot d (page k = d mod DP): the value loads of page k and the
  // staging loads of page k + 1, both issued DP pages ahead
  u32x4 ring[DP][IP + SV];
  auto fill = [&](int d, int k) {
    set_page(k);
#pragma unroll
    for (int s = 0; s < IP; ++s) ring[d][s] = issue(s);
    const int pg = g0 + min(k + 1, last);
#pragma unroll
    for (int s = 0; s < SV; ++s) ring[d][IP + s] = stage_item(s, pg);
  };
  {
    u32x4 s0[SV];
#pragma unroll
    for (int s = 0; s < SV; ++s) s0[s] = stage_item(s, g0);
#pragma unroll
    for (int d = 0; d < DP; ++d) fill(d, d);
    if (npg > 0) stage_store(s0, 0);
  }
  __syncthreads();

  floatx4 acc[RGTW][RTMAX];
#pragma unroll
  for (int i = 0; i < RGTW; ++i)
#pragma unroll
    for (int t = 0; t < RTMAX; ++t) acc[i][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float Bx[RTMAX], Em[RTMAX];                      // base and largest exponent per row slot
#pragma unroll
  for (int t = 0; t < RTMAX; ++t) {
    Bx[t] = -INFINITY;
    Em[t] = -INFINITY;
  }

  // page k of the chunk, ring slot d = k mod DP, staged in buffer k % 2
  auto page = [&](int k, int d) {
    const int cur = k & 1;
    const u32x4* lb = lbuf + cur * nst;
    const float* rec = reinterpret_cast<const float*>(lb + RT * 128);
    // the page's exponents of this lane's row slots, read together; the
    // usual page (the same exponents as the last: a score unit spans eight
    // pages) changes nothing
    float ev[RTMAX];
#pragma unroll
    for (int t = 0; t < RTMAX; ++t) ev[t] = rec[(16 * min(t, RT - 1) + lr) * 8];
    bool same = true;
#pragma unroll
    for (int t = 0; t < RTMAX; ++t) same = same && (t >= RT || ev[t] == Bx[t]);
    uint32_t dropped = 0;                           // row tiles left out
    if (!__all(same)) {
      bool resc = false;
      float fa[RTMAX];
#pragma unroll
      for (int t = 0; t < RTMAX; ++t) {
        fa[t] = 1.f;
        const float ep = ev[t];
        if (t < RT && ep != -INFINITY) {            // else the row's weights are zero
          const float em = fmaxf(Em[t], ep);
          if (ep >= em - 64.f) {
            fa[t] = Bx[t] == -INFINITY ? 1.f : pow2_rel(Bx[t], ep);
            Bx[t] = ep;
            Em[t] = em;
          } else {
            dropped |= 1u << t;                     // below 2^-64 of the row's largest weights
          }
        }
        resc = resc || fa[t] != 1.f;
      }
      if (__any(resc)) {
#pragma unroll
        for (int i = 0; i < RGTW; ++i)
#pragma unroll
          for (int t = 0; t < RTMAX; ++t) acc[i][t] *= fa[t];
      }
    }
    if (__any(dropped != 0)) {
      // each wave zeroes its own lanes' operand elements of the dropped rows
      // before reading them (all waves write the same zeros, and a lane's
      // read follows its own write)
      u32x4* lw = lbuf + cur * nst;
#pragma unroll
      for (int t = 0; t < RTMAX; ++t) {
        if (t < RT && ((dropped >> t) & 1u)) {
          lw[t * 128 + lane] = u32x4{0u, 0u, 0u, 0u};
          lw[t * 128 + 64 + lane] = u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
    const int nval = min(64, T_b - 64 * (g0 + k));
    const int keep0 = min(8, max(0, nval - 8 * lq));
    const int keep1 = min(8, max(0, nval - 32 - 8 * lq));
    // weight operands (k-step, row tile) in order, BQ LDS reads ahead of
    // their products
    constexpr int NB = 2 * RTMAX, BQ = 3;
    auto bload = [&](int j) { return lb[min(j % RTMAX, RT - 1) * 128 + (j / RTMAX) * 64 + lane]; };
    u32x4 bq[BQ];
#pragma unroll
    for (int j = 0; j < BQ; ++j) bq[j] = bload(j);
    u32x4 a[RGTW];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int ks = j / RTMAX, t = j % RTMAX;
      if (t == 0) {
#pragma unroll
        for (int i = 0; i < RGTW; ++i) {
          a[i] = ring[d][2 * i + ks];
          if (nval < 64) a[i] = keep_first(a[i], ks ? keep1 : keep0);
        }
      }
      const u32x4 B = bq[j % BQ];
      if (j + BQ < NB) bq[j % BQ] = bload(j + BQ);
      if (t < RT) {
#pragma unroll
        for (int i = 0; i < RGTW; ++i) acc[i][t] = mfma(a[i], B, acc[i][t]);
      }
    }
    if (k + 1 < npg) stage_store(&ring[d][IP], cur ^ 1);   // page k + 1, loaded DP pages back
    fill(d, k + DP);
    __syncthreads();
  };
  int k0 = 0;
  for (; k0 + DP <= npg; k0 += DP) {
#pragma unroll
    for (int d = 0; d < DP; ++d) page(k0 + d, d);
  }
#pragma unroll
  for (int d = 0; d < DP; ++d)
    if (k0 + d < npg) page(k0 + d, d);

  if (npg == 0) return;
  float* vp = vpart + int64_t(cidx) * NS * rv;
#pragma unroll
  for (int i = 0; i < RGTW; ++i) {
    const int r0 = 16 * (mt0 + i) + 4 * lq;
#pragma unroll
    for (int t = 0; t < RTMAX; ++t) {
      if (t < RT && mt0 + i < mt_v) {
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (r0 + v < rv) vp[int64_t(16 * t + lr) * rv + r0 + v] = acc[i][t][v];
      }
    }
  }
  if (rg == 0) {
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      const int i = tid + NTH * k;
      if (i < nst && i >= RT * 128 && (i & 1)) {
        const int slot = (i - RT * 128) >> 1;
        vel[int64_t(cidx) * 2 * NS + slot] = sB[k];
        vel[int64_t(cidx) * 2 * NS + NS + slot] = sL[k];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Merge of the chunks: a[b][row][r] = sum_c 2^(E_c - M) acc_c[r] / sum_c
// 2^(E_c - M) L_c, chunks in ascending order, with the running maximum
// rescaled by exact powers of two.  Grid (batch * NS row slots, rank blocks
// of 256); slot 16 t + j is row hord[t / NT][16 (t % NT) + j] (query i, head
// h as i * H_q + h).
__global__ __launch_bounds__(256) void merge_chunks(const float* __restrict__ vpart,
                                                    const float* __restrict__ vel,
                                                    const int32_t* __restrict__ seq_lens,
                                                    int max_context, int chunk_pages, int n_chunks,
                                                    int rv, int NS, float* __restrict__ amerged,
                                                    MfmaTables mt) {
  const int b = blockIdx.x / NS, j = blockIdx.x % NS;
  const int nh = 16 * mt.nt;
  const int row = mt.hord[j / nh][j % nh];
  if (row < 0) return;
  const int r = blockIdx.y * 256 + threadIdx.x;
  if (r >= rv) return;
  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int np = (T_b + 63) >> 6;
  const int nc = (np + chunk_pages - 1) / chunk_pages;
  const float* e_b = vel + int64_t(b) * n_chunks * 2 * NS + j;
  const float* a_b = vpart + (int64_t(b) * n_chunks * NS + j) * rv + r;
  float M = -INFINITY, a = 0.f, l = 0.f;
  int c = 0;
  for (; c + 8 <= nc; c += 8) {
    float ev[8], lv[8], av[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      ev[k] = e_b[(c + k) * 2 * NS];
      lv[k] = e_b[(c + k) * 2 * NS + NS];
      av[k] = a_b[int64_t(c + k) * NS * rv];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float Mn = fmaxf(M, ev[k]);
      const float fo = pow2_rel(M, Mn), fn = pow2_rel(ev[k], Mn);
      a = a * fo + av[k] * fn;
      l = l * fo + lv[k] * fn;
      M = Mn;
    }
  }
  for (; c < nc; ++c) {
    const float ev = e_b[c * 2 * NS], lv = e_b[c * 2 * NS + NS];
    const float av = a_b[int64_t(c) * NS * rv];
    const float Mn = fmaxf(M, ev);
    const float fo = pow2_rel(M, Mn), fn = pow2_rel(ev, Mn);
    a = a * fo + av * fn;
    l = l * fo + lv * fn;
    M = Mn;
  }
  amerged[(int64_t(b) * mt.queries * mt.q_heads + row) * rv + r] =
      (M == -INFINITY || !(l > 0.f)) ? 0.f : a / l;
}

// ---------------------------------------------------------------------------
// Up-projection o[b][h][:] = a[b][h][:] R_v[:, kv(h) block].  Grid (row
// blocks of 8 over (sequence, query, head of the KV head), KV heads, column
// tiles of CT).  Thread t: 8 columns (one 16-byte load a rank), rank group
// t / CG (ranks t / CG + RGS * k).  The merged rows are staged in LDS with
// float4 loads issued together with the thread's first batch of R_v loads
// (one memory round trip for both); the rank groups' sums are then added in
// ascending group order from LDS.
template <int CT>
__global__ __launch_bounds__(256) void upproj_rows(const float* __restrict__ amerged,
                                                   const bf16* __restrict__ Rv,
                                                   float* __restrict__ out, int batch, int rv,
                                                   HeadTables tb) {
  constexpr int RB = 8;                        // query rows a work-group
  constexpr int CG = CT / 8;                   // column groups of 8
  constexpr int RGS = 256 / CG;                // rank groups
  constexpr int U = 16;                        // R_v loads a batch
  constexpr int SV = 8;                        // staging float4 loads a thread a batch
  constexpr int RS = RB * CT + 1;              // LDS stride of a rank group's sums (odd: no bank conflicts)
  const int rbk = blockIdx.x, kv = blockIdx.y, ct = blockIdx.z;
  const int tid = threadIdx.x;
  const int dh = tb.head_dim, n = tb.n_kv_heads * dh, qpk = tb.q_per_kv;
  const int rows = batch * qpk;
  const int row0 = rbk * RB;
  const int nrow = min(RB, rows - row0);
  if (nrow <= 0) return;
  extern __shared__ float sa[];                // [RB][rv]; later [RGS][RS] rank-group sums
  const int c8 = tid % CG, rgp = tid / CG;
  const int col = ct * CT + 8 * c8;            // first of eight output columns
  // d_h is a multiple of 8: threads past d_h load a valid column group and
  // discard their sums
  const bf16* src = Rv + int64_t(kv) * dh + min(col, dh - 8);
  u32x4 v[U];
  auto issue = [&](int rbase) {
#pragma unroll
    for (int k = 0; k < U; ++k)
      v[k] = *reinterpret_cast<const u32x4*>(src + int64_t(min(rbase + RGS * k, rv - 1)) * n);
  };
  auto arow = [&](int q) {                     // merged row of local row q
    const int row = row0 + q;
    return amerged + (int64_t(row / qpk) * tb.n_q_heads + kv * qpk + row % qpk) * rv;
  };
  if ((rv & 3) == 0) {
    const int rv4 = rv >> 2, nvec = nrow * rv4;
    float4 sv[SV];
    // loads at clamped indices, unconditionally: no branch holds one back
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      const int i = min(tid + 256 * k, nvec - 1);
      sv[k] = reinterpret_cast<const float4*>(arow(i / rv4))[i % rv4];
    }
    issue(rgp);
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      const int i = tid + 256 * k;
      if (i < nvec) reinterpret_cast<float4*>(sa)[i] = sv[k];
    }
    for (int base = 256 * SV; base < nvec; base += 256 * SV) {
#pragma unroll
      for (int k = 0; k < SV; ++k) {
        const int i = min(base + tid + 256 * k, nvec - 1);
        sv[k] = reinterpret_cast<const float4*>(arow(i / rv4))[i % rv4];
      }
#pragma unroll
      for (int k = 0; k < SV; ++k) {
        const int i = base + tid + 256 * k;
        if (i < nvec) reinterpret_cast<float4*>(sa)[i] = sv[k];
      }
    }
  } else {
    issue(rgp);
    for (int i = tid; i < nrow * rv; i += 256) sa[i] = arow(i / rv)[i % rv];
  }
  __syncthreads();
  float acc[RB][8];
#pragma unroll
  for (int q = 0; q < RB; ++q)
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) acc[q][jj] = 0.f;
  for (int r = rgp; r < rv; r += RGS * U) {
    u32x4 cur[U];
#pragma unroll
    for (int k = 0; k < U; ++k) cur[k] = v[k];
    if (r + RGS * U < rv) issue(r + RGS * U);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int rr = r + RGS * k;
      if (rr < rv) {
        float f[8];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          f[2 * jj] = __uint_as_float(cur[k][jj] << 16);
          f[2 * jj + 1] = __uint_as_float(cur[k][jj] & 0xFFFF0000u);
        }
#pragma unroll
        for (int q = 0; q < RB; ++q) {
          if (q < nrow) {
            const float aq = sa[q * rv + rr];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) acc[q][jj] = fmaf(aq, f[jj], acc[q][jj]);
          }
        }
      }
    }
  }
  __syncthreads();                             // the staged rows are read; their space is reused
  float* red = sa;
#pragma unroll
  for (int q = 0; q < RB; ++q)
    if (q < nrow) {
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) red[rgp * RS + q * CT + 8 * c8 + jj] = acc[q][jj];
    }
  __syncthreads();
  for (int e = tid; e < nrow * CT; e += 256) {
    const int q = e / CT, cc = e % CT;
    if (ct * CT + cc >= dh) continue;
    float part[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) part[k] = 0.f;
    for (int g = 0; g < RGS; g += 8) {
#pragma unroll
      for (int k = 0; k < 8; ++k) part[k] += red[(g + k) * RS + q * CT + cc];
    }
    const float t = ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
    const int row = row0 + q;
    const int bb = row / qpk, h = kv * qpk + row % qpk;
    out[(int64_t(bb) * tb.n_q_heads + h) * dh + ct * CT + cc] = t;
  }
}

// ---------------------------------------------------------------------------
// Up-projection for the few rows (at most RB) of one KV head, a product of
// those rows with the head's r_v x d_h block of R_v that reads each of the
// block's rank rows as whole 128-byte pieces.  Grid (64-column tiles, KV
// heads), sixteen waves.  Lane: columns 8 (lane % 8) .. +7 of the tile, rank
// group g = 8 w + lane / 8 of 128 (ranks g, g + 128, ...), sixteen 16-byte
// R_v loads in flight.  The merged rows are staged in LDS first.  Fixed
// order of the sums: each lane sums its ranks in ascending order, a wave's
// eight rank groups are added by xor shuffles over lane bits 3, 4 and 5, and
// the sixteen waves' sums are added in wave order.
template <int RB>
__global__ __launch_bounds__(1024) void upproj_wide(const float* __restrict__ amerged,
                                                    const bf16* __restrict__ Rv,
                                                    float* __restrict__ out, int rows, int rv,
                                                    HeadTables tb) {
  constexpr int U = 16;                        // R_v loads a batch
  constexpr int RG = 128;                      // rank groups
  const int ct = blockIdx.x, kv = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c8 = lane & 7, rg = 8 * w + (lane >> 3);
  const int dh = tb.head_dim, n = tb.n_kv_heads * dh, qpk = tb.q_per_kv;
  extern __shared__ float sa[];                // [rows][rv]; later [16 waves][RB * 64]
  const bf16* src = Rv + (int64_t(kv) * dh + ct * 64);   // uniform base; lane offsets below
  u32x4 v[U];
  auto issue = [&](int rbase) {
#pragma unroll
    for (int k = 0; k < U; ++k)
      v[k] = *reinterpret_cast<const u32x4*>(src + (min(rbase + RG * k, rv - 1) * n + 8 * c8));
  };
  auto arow = [&](int q) {                     // merged row of local row q
    return amerged + (int64_t(q / qpk) * tb.n_q_heads + kv * qpk + q % qpk) * rv;
  };
  issue(rg);                                   // the first batch travels with the staging
  if ((rv & 3) == 0) {
    const int rv4 = rv >> 2, nvec = rows * rv4;
    for (int i0 = tid; i0 < nvec; i0 += 2048) {   // two loads in flight
      const int i1 = min(i0 + 1024, nvec - 1);
      const float4 s0 = reinterpret_cast<const float4*>(arow(i0 / rv4))[i0 % rv4];
      const float4 s1 = reinterpret_cast<const float4*>(arow(i1 / rv4))[i1 % rv4];
      reinterpret_cast<float4*>(sa)[i0] = s0;
      if (i0 + 1024 < nvec) reinterpret_cast<float4*>(sa)[i0 + 1024] = s1;
    }
  } else {
    for (int i = tid; i < rows * rv; i += 1024) sa[i] = arow(i / rv)[i % rv];
  }
  __syncthreads();
  float acc[RB][8];
#pragma unroll
  for (int q = 0; q < RB; ++q)
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) acc[q][jj] = 0.f;
  // one batch covers 128 U ranks (all of r_v = 2048 at U = 16)
  for (int r = rg; r < rv; r += RG * U) {
    if (r != rg) issue(r);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int rr = r + RG * k;
      if (rr < rv) {
        float f[8];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          f[2 * jj] = __uint_as_float(v[k][jj] << 16);
          f[2 * jj + 1] = __uint_as_float(v[k][jj] & 0xFFFF0000u);
        }
#pragma unroll
        for (int q = 0; q < RB; ++q) {
          if (q < rows) {
            const float aq = sa[q * rv + rr];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) acc[q][jj] = fmaf(aq, f[jj], acc[q][jj]);
          }
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < RB; ++q)
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      float x = acc[q][jj];
      x += __shfl_xor(x, 8);
      x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      acc[q][jj] = x;
    }
  __syncthreads();                             // the staged rows are read; their space is reused
  float* red = sa;
  if (lane < 8) {
#pragma unroll
    for (int q = 0; q < RB; ++q)
      if (q < rows) {
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) red[w * (RB * 64) + q * 64 + 8 * c8 + jj] = acc[q][jj];
      }
  }
  __syncthreads();
  if (tid < rows * 64) {
    const int q = tid >> 6, cc = tid & 63;
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) t += red[k * (RB * 64) + tid];
    const int bb = q / qpk, h = kv * qpk + q % qpk;
    out[(int64_t(bb) * tb.n_q_heads + h) * dh + ct * 64 + cc] = t;
  }
}

// ---------------------------------------------------------------------------
// Up-projection on MFMA: o[row][c] = sum_r a[row][r] R_v[r][kv d_h + c] for
// the rows of one KV head (sequence, query, head of the KV head).  One
// work-group of W waves (4, or 8 when a wave would otherwise walk 32 rank
// steps or more) a (column tile of CT, KV head, group of 64 rows).  The work-group's R_v block (r_v x CT bf16) is loaded once, in 8 x 8 units
// transposed in registers, and stored in LDS rank-contiguous per column:
// the MFMA's B operand takes 8 consecutive ranks of one column a lane.  The
// waves are the row group's 16-row tiles (1, 2 or 4) times KS = W / tiles
// rank ranges; a wave's A operand is its 16 merged rows (fp32 split into
// bf16 hi + lo parts) read from global memory in operand order, KA rank
// steps ahead.  The rank ranges' sums are added through LDS in a fixed
// order.
constexpr int kUpWavesMax = 8;                 // waves of the MFMA up-projection, at most

template <int CT, int W>
__global__ __launch_bounds__(W * 64) void upproj_mfma(const float* __restrict__ amerged,
                                                   const bf16* __restrict__ Rv,
                                                   float* __restrict__ out, int rows, int rv,
                                                   HeadTables tb) {
  constexpr int NC = CT / 16;                  // column tiles of a wave
  constexpr int KA = W == 8 ? 8 : 4;           // rank steps of A loads in flight
  constexpr int NTH = W * 64;
  constexpr int UB = 2;                        // R_v units (8 x 8) a thread a batch
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* rt = reinterpret_cast<bf16*>(smem);    // [CT][stride]
  // 1-D grid, XCD-aware: work-group ids equal mod 8 run on one XCD, and all
  // column tiles of one (KV head, row group) share an XCD, so its merged rows
  // are fetched into that XCD's L2 once
  const int nct = tb.head_dim / CT, ngr = tb.n_kv_heads * ((rows + 63) / 64);
  const int xcd = blockIdx.x & 7, pos = blockIdx.x >> 3;
  const int grp = 8 * (pos / nct) + xcd, ctile = pos % nct;
  if (grp >= ngr) return;
  const int kv = grp % tb.n_kv_heads, row0 = (grp / tb.n_kv_heads) * 64;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lq = lane >> 4;
  const int dh = tb.head_dim, n = tb.n_kv_heads * dh, qpk = tb.q_per_kv;
  const int nrow = min(64, rows - row0);
  const int tiles = nrow <= 16 ? 1 : (nrow <= 32 ? 2 : 4);
  const int KS = W / tiles;
  const int mt = w % tiles, ks = w / tiles;
  const int nstep = (rv + 31) >> 5;            // 32-rank steps
  const int stride = 32 * nstep + 8;           // LDS row of one column (elements)
  const int col0 = kv * dh + ctile * CT;

  // this lane's A row (clamped; results of rows past the end are dropped)
  const int lrow = row0 + 16 * mt + lr;
  const int crow = min(lrow, rows - 1);
  const float* arow = amerged + (int64_t(crow / qpk) * tb.n_q_heads + kv * qpk + crow % qpk) * rv;
  const int s0 = ks * nstep / KS, s1 = (ks + 1) * nstep / KS;   // this wave's rank steps
  float4 av[KA][2];
  auto aload = [&](int st, float4 (&d)[2]) {   // ranks 32 st + 8 lq .. +7, zero past r_v
    const int r = 32 * min(st, nstep - 1) + 8 * lq;
    if ((rv & 3) == 0 && r + 8 <= rv) {          // 16-byte aligned rows
      d[0] = *reinterpret_cast<const float4*>(arow + r);
      d[1] = *reinterpret_cast<const float4*>(arow + r + 4);
    } else {
      float t[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) t[j] = r + j < rv ? arow[r + j] : 0.f;
      d[0] = make_float4(t[0], t[1], t[2], t[3]);
      d[1] = make_float4(t[4], t[5], t[6], t[7]);
    }
  };
#pragma unroll
  for (int k = 0; k < KA; ++k) aload(s0 + k, av[k]);

  // the R_v block in units of 8 ranks x 8 columns (unit u: ranks 8 (u / (CT
  // / 8)) .., columns 8 (u % (CT / 8)) ..), UB units a thread a batch: eight
  // 16-byte row loads, transposed in registers into eight rank-contiguous
  // 16-byte column pieces; ranks past r_v are stored as zero
  const int nunit = 4 * nstep * (CT / 8);
  for (int base = 0; base < nunit; base += NTH * UB) {
    u32x4 v[UB][8];
#pragma unroll
    for (int k = 0; k < UB; ++k) {
      const int u = min(base + tid + NTH * k, nunit - 1);
      const int r0 = 8 * (u / (CT / 8)), c8 = 8 * (u % (CT / 8));
#pragma unroll
      for (int i = 0; i < 8; ++i)
        v[k][i] = *reinterpret_cast<const u32x4*>(Rv + int64_t(min(r0 + i, rv - 1)) * n + col0 + c8);
    }
#pragma unroll
    for (int k = 0; k < UB; ++k) {
      const int u = base + tid + NTH * k;
      if (u < nunit) {
        const int r0 = 8 * (u / (CT / 8)), c8 = 8 * (u % (CT / 8));
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (r0 + i >= rv) v[k][i] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          u32x4 t;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t a = v[k][2 * j][c >> 1], b = v[k][2 * j + 1][c >> 1];
            t[j] = (c & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
          }
          *reinterpret_cast<u32x4*>(rt + (c8 + c) * stride + r0) = t;
        }
      }
    }
  }
  __syncthreads();

  floatx4 acc[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) acc[c] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int sb = s0; sb < s1; sb += KA) {
#pragma unroll
    for (int k = 0; k < KA; ++k) {
      const int st = sb + k;
      if (st < s1) {
        const float f[8] = {av[k][0].x, av[k][0].y, av[k][0].z, av[k][0].w,
                            av[k][1].x, av[k][1].y, av[k][1].z, av[k][1].w};
        aload(st + KA, av[k]);
        u32x4 hi, lo;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bf16 h0 = static_cast<bf16>(f[2 * j]), h1 = static_cast<bf16>(f[2 * j + 1]);
          const bf16 l0 = static_cast<bf16>(f[2 * j] - static_cast<float>(h0));
          const bf16 l1 = static_cast<bf16>(f[2 * j + 1] - static_cast<float>(h1));
          hi[j] = uint32_t(__builtin_bit_cast(uint16_t, h0)) | (uint32_t(__builtin_bit_cast(uint16_t, h1)) << 16);
          lo[j] = uint32_t(__builtin_bit_cast(uint16_t, l0)) | (uint32_t(__builtin_bit_cast(uint16_t, l1)) << 16);
        }
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const u32x4 B = *reinterpret_cast<const u32x4*>(rt + (16 * c + lr) * stride + 32 * st + 8 * lq);
          acc[c] = mfma(hi, B, acc[c]);
          acc[c] = mfma(lo, B, acc[c]);
        }
      }
    }
  }

  // rank ranges ks > 0 -> LDS; ks = 0 adds them in ascending order and stores
  __syncthreads();                             // the R_v block is no longer read
  floatx4* red = reinterpret_cast<floatx4*>(smem);   // [wave][NC][64]
  if (ks > 0) {
#pragma unroll
    for (int c = 0; c < NC; ++c) red[(w * NC + c) * 64 + lane] = acc[c];
  }
  __syncthreads();
  if (ks > 0) return;
  for (int k2 = 1; k2 < KS; ++k2) {
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[c] += red[((k2 * tiles + mt) * NC + c) * 64 + lane];
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int row = row0 + 16 * mt + 4 * lq + v;
    if (row < rows) {
      const int bb = row / qpk, h = kv * qpk + row % qpk;
#pragma unroll
      for (int c = 0; c < NC; ++c)
        out[(int64_t(bb) * tb.n_q_heads + h) * dh + ctile * CT + 16 * c + lr] = acc[c][v];
    }
  }
}

}  // namespace

size_t pass_score_lds_bytes(const dckv_plan& p) {
  // query blocks, then each wave's pages: 512 B of weights and 128 B of
  // exponents and sums a page
  return std::max<size_t>(size_t(p.pass.max_pairs) * 2048 + 8 * kUnitPages * (512 + 128), kScoreMinLds);
}

size_t pass_value_lds_bytes(const dckv_plan& p, int rgt) {
  if (p.pass.n_slices > 1)   // two pages' weights and records, 2.5 KB a row tile
    return size_t(2) * p.pass.n_slices * p.pass.nt * 2560;
  const int nh = 16 * p.pass.nt, W = 8;
  return size_t(2) * W * nh * 4 + size_t(W) * rgt * p.pass.nt * 64 * 16;
}

size_t upproj_lds_bytes(const dckv_plan& p, int ct) {
  // the staged rows, or the rank groups' sums: (256 / (ct / 8)) x (8 ct + 1)
  return std::max<size_t>(size_t(8) * p.rv, size_t(2048 / ct) * (8 * ct + 1)) * 4;
}

int pass_max_chunk_pages(const dckv_plan& p) {
  return p.pass.n_slices > 1 ? kMaxSharedChunkPages : kMaxChunkPages;
}

template <int NT, int RGT>
hipError_t launch_value(const dckv_plan& p, const DecodeShape& sh, const void* pool,
                        int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                        const int32_t* seq_lens, const u32x4* pw, float* vpart, float* vel,
                        hipStream_t stream) {
  auto kern = value_pages<8, NT, RGT>;
  const size_t lds = pass_value_lds_bytes(p, RGT);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  const int bc = sh.batch * sh.n_chunks;
  const dim3 grid(unsigned(8 * sh.n_rgroups * ((bc + 7) / 8)));
  if (p.prof_before && p.prof_after)
    hipExtLaunchKernelGGL(kern, grid, dim3(512), uint32_t(lds), stream, p.prof_before, p.prof_after,
                          0u, static_cast<const bf16*>(pool), num_pages, page_table, max_pages,
                          seq_lens, sh.max_context, sh.chunk_pages, sh.n_chunks, sh.n_rgroups,
                          sh.batch, sh.npm, p.rv, p.pass.mt_v, p.page_elems, p.value_base, pw,
                          vpart, vel);
  else
    hipLaunchKernelGGL(kern, grid, dim3(512), lds, stream, static_cast<const bf16*>(pool),
                       num_pages, page_table, max_pages, seq_lens, sh.max_context, sh.chunk_pages,
                       sh.n_chunks, sh.n_rgroups, sh.batch, sh.npm, p.rv, p.pass.mt_v,
                       p.page_elems, p.value_base, pw, vpart, vel);
  return hipGetLastError();
}

template <int W, int RTMAX, int RGTW, int DP>
hipError_t launch_shared(const dckv_plan& p, const DecodeShape& sh, const void* pool,
                         int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                         const int32_t* seq_lens, const u32x4* pw, float* vpart, float* vel,
                         hipStream_t stream) {
  auto kern = value_shared<W, RTMAX, RGTW, DP>;
  const size_t lds = pass_value_lds_bytes(p, RGTW);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  const int bc = sh.batch * sh.n_chunks;
  const dim3 grid(unsigned(8 * sh.n_rgroups * ((bc + 7) / 8)));
  const int RT = p.pass.n_slices * p.pass.nt;
  if (p.prof_before && p.prof_after)
    hipExtLaunchKernelGGL(kern, grid, dim3(W * 64), uint32_t(lds), stream, p.prof_before, p.prof_after,
                          0u, static_cast<const bf16*>(pool), num_pages, page_table, max_pages,
                          seq_lens, sh.max_context, sh.chunk_pages, sh.n_chunks, sh.n_rgroups,
                          sh.batch, sh.npm, p.rv, p.pass.mt_v, p.page_elems, p.value_base, RT, pw,
                          vpart, vel);
  else
    hipLaunchKernelGGL(kern, grid, dim3(W * 64), lds, stream, static_cast<const bf16*>(pool), num_pages,
                       page_table, max_pages, seq_lens, sh.max_context, sh.chunk_pages, sh.n_chunks,
                       sh.n_rgroups, sh.batch, sh.npm, p.rv, p.pass.mt_v, p.page_elems, p.value_base,
                       RT, pw, vpart, vel);
  return hipGetLastError();
}

// The shared-weights value pass for the plan's RT = 2J row tiles (J >= 2
// slices of two tiles), RGTW = sh.rgt value tiles a wave; each row-tile
// count has its own instantiation.
hipError_t launch_value_shared(const dckv_plan& p, const DecodeShape& sh, const void* pool,
                               int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                               const int32_t* seq_lens, const u32x4* pw, float* vpart,
                               float* vel, hipStream_t stream) {
  const int RT = p.pass.n_slices * p.pass.nt;
#define DCKV_SHARED(RTC, RGTW, DP) \
  launch_shared<kSharedWaves, RTC, RGTW, DP>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, pw, vpart, vel, stream)
  // the deepest ring of each shape that the compiler keeps out of scratch
  switch (RT) {
    case 4: return sh.rgt == 2 ? DCKV_SHARED(4, 2, 3) : DCKV_SHARED(4, 1, 4);
    case 6: return sh.rgt == 2 ? DCKV_SHARED(6, 2, 2) : DCKV_SHARED(6, 1, 4);
    case 8: return sh.rgt == 2 ? DCKV_SHARED(8, 2, 4) : DCKV_SHARED(8, 1, 8);
    case 10: return DCKV_SHARED(10, 1, 6);
    case 12: return DCKV_SHARED(12, 1, 4);
    case 14: return DCKV_SHARED(14, 1, 3);
    case 16: return DCKV_SHARED(16, 1, 3);
  }
#undef DCKV_SHARED
  return hipErrorInvalidValue;
}

template <int NT, int RING>
hipError_t launch_score_r(const dckv_plan& p, const DecodeShape& sh, const u32x4* qblk,
                          const void* pool, int64_t num_pages, const int32_t* page_table,
                          int32_t max_pages, const int32_t* seq_lens, uint32_t* pw,
                          hipStream_t stream) {
  auto kern = p.RK % 32 ? score_pages<NT, RING, true> : score_pages<NT, RING, false>;
  const size_t lds = pass_score_lds_bytes(p);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  const int n_units = sh.batch * sh.units_per_seq;
  hipLaunchKernelGGL(kern, dim3(8 * p.pass.n_slices * ((n_units + 7) / 8)), dim3(512), lds, stream, qblk,
                     static_cast<const bf16*>(pool), num_pages, page_table, max_pages, seq_lens,
                     sh.max_context, sh.units_per_seq, n_units, sh.npm, p.RK, p.page_elems, pw,
                     p.pass);
  return hipGetLastError();
}

template <int NT>
hipError_t launch_score(const dckv_plan& p, const DecodeShape& sh, const u32x4* qblk,
                        const void* pool, int64_t num_pages, const int32_t* page_table,
                        int32_t max_pages, const int32_t* seq_lens, uint32_t* pw,
                        hipStream_t stream) {
  switch (p.pass_ring) {
    case 16: return launch_score_r<NT, 16>(p, sh, qblk, pool, num_pages, page_table, max_pages, seq_lens, pw, stream);
  }
  return hipErrorInvalidValue;
}

size_t upproj_mfma_lds_bytes(const dckv_plan& p, int ct) {
  const size_t stride = size_t((p.rv + 31) / 32) * 32 + 8;
  return std::max<size_t>(size_t(ct) * stride * 2, size_t(kUpWavesMax) * (ct / 16) * 64 * 16);
}

size_t upproj_wide_lds_bytes(const dckv_plan& p, int rows, int rb) {
  return std::max<size_t>(size_t(rows) * p.rv, size_t(16) * rb * 64) * 4;
}

hipError_t launch_upproj(const dckv_plan& p, int32_t batch_rows, const float* amerged,
                         const void* R_value, float* out, hipStream_t stream) {
  const int rows = batch_rows * p.qpk;          // rows a KV head
  // one or two rows a KV head, with 64-column tiles that give the grid at
  // least 32 work-groups: the wide kernel (whole 128-byte pieces of R_v;
  // from three rows on its per-lane products cost more than the MFMA
  // kernel's R_v transpose)
  if (rows > 0 && rows <= 2 && p.dh % 64 == 0 && p.Hkv * (p.dh / 64) >= 32) {
    const int rb = rows <= 1 ? 1 : 2;
    const size_t lds = upproj_wide_lds_bytes(p, rows, rb);
    if (lds <= 160 * 1024) {
      auto kern = rb == 1 ? upproj_wide<1> : upproj_wide<2>;
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(kern, dim3(p.dh / 64, p.Hkv), dim3(1024), lds, stream, amerged,
                         static_cast<const bf16*>(R_value), out, rows, p.rv, p.tables);
      return hipGetLastError();
    }
  }
  // MFMA for at least 3 rows a KV head (fewer: R_v is read once either way
  // and the VALU kernels read it straight into registers): 32-column tiles
  // while the transposed R_v block fits LDS and the grid still fills the
  // chip, else 16
  const int groups = p.Hkv * ((rows + 63) / 64);
  const bool fit32 = p.dh % 32 == 0 && upproj_mfma_lds_bytes(p, 32) <= 160 * 1024;
  const bool fit16 = p.dh % 16 == 0 && upproj_mfma_lds_bytes(p, 16) <= 160 * 1024;
  const int ctm = rows < 3 ? 0
                  : (fit32 && (groups * (p.dh / 32) >= 256 || !fit16)) ? 32 : (fit16 ? 16 : 0);
  if (ctm) {
    const size_t lds = upproj_mfma_lds_bytes(p, ctm);
    // eight waves when four would each walk 32 rank steps or more
    const int tiles = rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
    const int W = ((p.rv + 31) / 32) * tiles / 4 >= 32 ? 8 : 4;
    auto kern = ctm == 32 ? (W == 8 ? upproj_mfma<32, 8> : upproj_mfma<32, 4>)
                          : (W == 8 ? upproj_mfma<16, 8> : upproj_mfma<16, 4>);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    const int ngr = p.Hkv * ((rows + 63) / 64);
    hipLaunchKernelGGL(kern, dim3(8 * ((ngr + 7) / 8) * (p.dh / ctm)), dim3(W * 64), lds, stream,
                       amerged, static_cast<const bf16*>(R_value), out, rows, p.rv, p.tables);
    return hipGetLastError();
  }
  // column tiles of 16 when tiles of 32 would leave most compute units idle
  const int rblocks = (rows + 7) / 8;
  const int ct = int64_t(rblocks) * p.Hkv * ((p.dh + 31) / 32) >= 256 ? 32 : 16;
  const size_t lds = upproj_lds_bytes(p, ct);
  if (ct == 32) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(upproj_rows<32>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(upproj_rows<32>, dim3(rblocks, p.Hkv, (p.dh + 31) / 32), dim3(256), lds,
                       stream, amerged, static_cast<const bf16*>(R_value), out, batch_rows, p.rv,
                       p.tables);
  } else {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(upproj_rows<16>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(upproj_rows<16>, dim3(rblocks, p.Hkv, (p.dh + 15) / 16), dim3(256), lds,
                       stream, amerged, static_cast<const bf16*>(R_value), out, batch_rows, p.rv,
                       p.tables);
  }
  return hipGetLastError();
}

hipError_t launch_decode_pass(const dckv_plan& p, const DecodeShape& sh, const float* q,
                              const void* pool, int64_t num_pages, const int32_t* page_table,
                              int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                              const void* R_value, float* out, void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  u32x4* qt = reinterpret_cast<u32x4*>(ws + sh.off_qt);
  uint32_t* pw = reinterpret_cast<uint32_t*>(ws + sh.off_p);
  float* vpart = reinterpret_cast<float*>(ws + sh.off_acc);
  float* vel = reinterpret_cast<float*>(ws + sh.off_ml);
  float* amerged = reinterpret_cast<float*>(ws + sh.off_opart);
  hipError_t e = launch_fold(p, p.pass, sh.batch, q, R_keys, qt, stream);
  if (e != hipSuccess) return e;
  e = p.pass.nt == 1 ? launch_score<1>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens,
                                       pw, stream)
                     : launch_score<2>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens,
                                       pw, stream);
  if (e != hipSuccess) return e;
  const u32x4* pw4 = reinterpret_cast<const u32x4*>(pw);
#define DCKV_VALUE(NT, RGT) \
  launch_value<NT, RGT>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, pw4, vpart, vel, stream)
  if (p.pass.n_slices > 1)
    e = launch_value_shared(p, sh, pool, num_pages, page_table, max_pages, seq_lens, pw4, vpart, vel,
                            stream);
  else if (p.pass.nt == 1)
    e = sh.rgt == 8 ? DCKV_VALUE(1, 8) : sh.rgt == 6 ? DCKV_VALUE(1, 6) : DCKV_VALUE(1, 4);
  else
    e = sh.rgt == 8 ? DCKV_VALUE(2, 8) : sh.rgt == 6 ? DCKV_VALUE(2, 6) : DCKV_VALUE(2, 4);
#undef DCKV_VALUE
  if (e != hipSuccess) return e;
  const int NS = 16 * p.pass.nt * p.pass.n_slices;       // row slots
  hipLaunchKernelGGL(merge_chunks, dim3(unsigned(sh.batch * NS), unsigned((p.rv + 255) / 256)),
                     dim3(256), 0, stream, vpart, vel, seq_lens, sh.max_context, sh.chunk_pages,
                     sh.n_chunks, p.rv, NS, amerged, p.pass);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_upproj(p, sh.batch * p.Q, amerged, R_value, out, stream);
}

}  // namespace dckv
