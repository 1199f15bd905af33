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
// upproj_rows: o_h = a_h R_v[:, kv(h) block] (Sec. III-A z R, Sec. III-D R_v).
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
// [ur * unit_pages, (ur + 1) * unit_pages) of it.  The eight waves serve
// PP = 2 / NT pages at a time: wave w takes head tile n = (w / 4) % NT and
// 16-token row block m = w % 4 of pages pl, pl + PP, ... (pl = w / (4 NT)),
// so the waves of a work-group stream the same pages side by side.  A
// wave's items are, page after page, the 1 KB operands of its 16 tokens in
// the key chunks of its tile's groups; a ring of RING loads runs ahead
// across page boundaries.  The weights of a row block are taken relative to
// its own integer exponent e = ceil(max over its 16 tokens), so no wave waits
// for another.
//
// With several queries a sequence the rows are cut into J slices (as for
// the single-pass kernel): work-group (unit, slice) loads the key chunks of
// its slice's groups, and a row of query i sees positions before
// T_b - Q + i + 1.
//
// Outputs per (sequence b, page pg of it, row tile t = slice * NT + n):
//   pbuf   2 KB: the weights as the value MFMA's B operand, 16 heads x 64
//          tokens: k-step ks (tokens 32ks..32ks+31) at ks * 1024 bytes, lane
//          L = 16 * (t%32 / 8) + head at L * 16, 8 tokens a lane
//   elbuf  512 B: e and l of row slot j and row block m at floats 8j + m and
//          8j + 4 + m, l the sum of the block's rounded weights
template <int NT, int RING>
__global__ __launch_bounds__(512, 1) void score_pages(
    const u32x4* __restrict__ qblk_ws, const bf16* __restrict__ pool, int64_t num_pages,
    const int32_t* __restrict__ page_table, int max_pages, const int32_t* __restrict__ seq_lens,
    int max_context, int unit_pages, int units_per_seq, int n_units, int npm, int RK,
    int64_t page_elems, uint32_t* __restrict__ pbuf, float* __restrict__ elbuf, MfmaTables mt) {
  constexpr int PP = 2 / NT;                   // pages side by side
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
  const int nmine = max(0, (p1 - p0 - pl + PP - 1) / PP);       // this wave's pages (<= 64)
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

  // the weights of this wave's 16 tokens of page k, from S
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
    // tokens 16m + 4lq .. +3: k-step m/2, operand lane 16 * (2(m%2) + lq/2) + lr
    const int64_t tile = (int64_t(b) * npm + pg) * RT + slice * NT + n;
    uint32_t* blk = pbuf + tile * 512;
    const int L = 16 * (2 * (m & 1) + (lq >> 1)) + lr;
    *reinterpret_cast<uint2*>(blk + (m >> 1) * 256 + L * 4 + 2 * (lq & 1)) = uint2{pk[0], pk[1]};
    psum = wave_sum16(psum);
    if (lq == 0) {
      elbuf[tile * 128 + 8 * lr + m] = e;
      elbuf[tile * 128 + 8 * lr + 4 + m] = psum;
    }
    S = floatx4{0.f, 0.f, 0.f, 0.f};
  };

  auto consume = [&](u32x4 a) {
    const int c = con_c < ln0 ? st0 + con_c : st1 + (con_c - ln0);
    if (c == kc_last) a = keep_first(a, kvalid_last);
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
    int64_t value_base, const u32x4* __restrict__ pbuf, const u32x4* __restrict__ elbuf,
    float* __restrict__ vpart, float* __restrict__ vel) {
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
    if (s < P0) return elbuf[((seq_page0 + ppg) * NT + (s >> 1)) * 32 + 2 * lr + (s & 1)];
    if (s < V0) {
      const int n = (s - P0) >> 1, ks = (s - P0) & 1;
      return pbuf[((seq_page0 + ppg) * NT + n) * 128 + ks * 64 + lane];
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
// (sequence b, chunk c, rank group g): the eight waves walk the chunk's pages
// together, wave w owning value tiles g * 8 * RGTW + w * RGTW .. + RGTW - 1
// against all RT row tiles, so each value latent byte is read once.  The
// weights of a page are staged in LDS already rescaled to the running
// exponents: thread i of the staging holds weight operand element i (row
// tile t, k-step, operand lane) of every page and keeps the running exponent
// E of that element's row slot (the same in every thread holding that slot:
// the same records in the same order), and the holder of k-step 0, lanes
// 0..15 also keeps the slot's running sum L and stages the factor 2^(E_old -
// E_new) by which the waves rescale their accumulators.  Two buffers, one
// barrier a page: the next page's weights load while the current one is
// used; a wave's value loads run DP pages ahead.
// Partials as value_pages, over NS = 16 RT row slots; no sums across waves.
template <int RTMAX, int RGTW, int DP>
__global__ __launch_bounds__(512, 1) void value_shared(
    const bf16* __restrict__ pool, int64_t num_pages, const int32_t* __restrict__ page_table,
    int max_pages, const int32_t* __restrict__ seq_lens, int max_context, int chunk_pages,
    int n_chunks, int n_rg, int batch, int npm, int rv, int mt_v, int64_t page_elems,
    int64_t value_base, int RT, const u32x4* __restrict__ pbuf, const u32x4* __restrict__ elbuf,
    float* __restrict__ vpart, float* __restrict__ vel) {
  constexpr int W = 8;
  constexpr int IP = 2 * RGTW;                      // value loads a page a wave
  constexpr int RING = DP * IP;
  constexpr int SV = (RTMAX * 128 + 511) / 512;     // weight elements a staging thread
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
  const int pid_tbl = (pt >= 0 && pt < num_pages) ? pt : -1;
  const int mt0 = rg * W * RGTW + w * RGTW;          // this wave's first value tile

  // LDS, two buffers: weights [RT][2][64] u32x4, then factors [NS] floats
  const int nw = RT * 128;
  u32x4* wbuf = reinterpret_cast<u32x4*>(smem);
  float* fbuf = reinterpret_cast<float*>(wbuf + 2 * nw);
  const u32x4* pb0 = pbuf + int64_t(b) * npm * RT * 128;
  const u32x4* eb0 = elbuf + int64_t(b) * npm * RT * 32;
  u32x4 sw[SV], se[SV], sl[SV];                     // raw weights, e and l records of the slot
  float Er[SV], Lr[SV];
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    Er[k] = -INFINITY;
    Lr[k] = 0.f;
  }
  auto stage_load = [&](int pg) {                   // pg < npm: loads at clamped indices
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      const int i = min(tid + 512 * k, nw - 1);
      const int slot = 16 * (i >> 7) + (i & 15);
      sw[k] = pb0[int64_t(pg) * RT * 128 + i];
      se[k] = eb0[int64_t(pg) * RT * 32 + 2 * slot];
      sl[k] = eb0[int64_t(pg) * RT * 32 + 2 * slot + 1];
    }
  };
  auto stage_store = [&](int buf) {
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      const int i = tid + 512 * k;
      if (i < nw) {
        const float4 ev = __builtin_bit_cast(float4, se[k]);
        const float En = fmaxf(Er[k], fmaxf(fmaxf(ev.x, ev.y), fmaxf(ev.z, ev.w)));
        const float f0 = pow2_rel(ev.x, En), f1 = pow2_rel(ev.y, En);
        const float f2 = pow2_rel(ev.z, En), f3 = pow2_rel(ev.w, En);
        // operand lane L holds tokens 32 ks + 8 (L / 16) ..: row block 2 ks + L / 32
        const int ks = (i >> 6) & 1, hi = (i >> 5) & 1;
        const float f = ks ? (hi ? f3 : f2) : (hi ? f1 : f0);
        wbuf[buf * nw + i] = scale8(sw[k], f);
        if ((i & 127) < 16) {                       // k-step 0, lanes 0..15: slot 16 t + i % 16
          const float4 lv = __builtin_bit_cast(float4, sl[k]);
          const float fa = Er[k] == -INFINITY ? 1.f : pow2_rel(Er[k], En);
          Lr[k] = Lr[k] * fa + (((lv.x * f0 + lv.y * f1) + lv.z * f2) + lv.w * f3);
          fbuf[buf * NS + 16 * (i >> 7) + (i & 15)] = fa;
        }
        Er[k] = En;
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

  u32x4 ring[RING];
  stage_load(g0);
#pragma unroll
  for (int d = 0; d < DP; ++d) {
    set_page(d);
#pragma unroll
    for (int s = 0; s < IP; ++s) ring[d * IP + s] = issue(s);
  }
  if (npg > 0) stage_store(0);
  __syncthreads();

  floatx4 acc[RGTW][RTMAX];
#pragma unroll
  for (int i = 0; i < RGTW; ++i)
#pragma unroll
    for (int t = 0; t < RTMAX; ++t) acc[i][t] = floatx4{0.f, 0.f, 0.f, 0.f};

  // page k of the chunk, its value loads in ring slots d * IP ..
  auto page = [&](int k, int d) {
    const int cur = k & 1;
    const bool more = k + 1 < npg;
    stage_load(g0 + (more ? k + 1 : k));            // the next page's weights, in flight
    const u32x4* lb = wbuf + cur * nw;
    float fa[RTMAX];
    bool resc = false;
#pragma unroll
    for (int t = 0; t < RTMAX; ++t) {
      fa[t] = t < RT ? fbuf[cur * NS + 16 * t + lr] : 1.f;
      resc = resc || fa[t] != 1.f;
    }
    if (__any(resc)) {
#pragma unroll
      for (int i = 0; i < RGTW; ++i)
#pragma unroll
        for (int t = 0; t < RTMAX; ++t) acc[i][t] *= fa[t];
    }
    const int nval = min(64, T_b - 64 * (g0 + k));
    const int keep0 = min(8, max(0, nval - 8 * lq));
    const int keep1 = min(8, max(0, nval - 32 - 8 * lq));
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      u32x4 a[RGTW];
#pragma unroll
      for (int i = 0; i < RGTW; ++i) {
        a[i] = ring[d * IP + 2 * i + ks];
        if (nval < 64) a[i] = keep_first(a[i], ks ? keep1 : keep0);
      }
#pragma unroll
      for (int t = 0; t < RTMAX; ++t) {
        if (t < RT) {
          const u32x4 B = lb[t * 128 + ks * 64 + lane];
#pragma unroll
          for (int i = 0; i < RGTW; ++i) acc[i][t] = mfma(a[i], B, acc[i][t]);
        }
      }
    }
    set_page(k + DP);                                // refill this page's slots
#pragma unroll
    for (int s = 0; s < IP; ++s) ring[d * IP + s] = issue(s);
    if (more) stage_store(cur ^ 1);
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
      const int i = tid + 512 * k;
      if (i < nw && (i & 127) < 16) {
        const int slot = 16 * (i >> 7) + (i & 15);
        vel[int64_t(cidx) * 2 * NS + slot] = Er[k];
        vel[int64_t(cidx) * 2 * NS + NS + slot] = Lr[k];
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

}  // namespace

size_t pass_score_lds_bytes(const dckv_plan& p) {
  return std::max<size_t>(size_t(p.pass.max_pairs) * 2048, kScoreMinLds);
}

size_t pass_value_lds_bytes(const dckv_plan& p, int rgt) {
  if (p.pass.n_slices > 1)   // two pages' weights and factors, 2 KB + 64 B a row tile
    return size_t(2) * p.pass.n_slices * p.pass.nt * (2048 + 64);
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
                        const int32_t* seq_lens, const u32x4* pbuf, const u32x4* elbuf, float* vpart,
                        float* vel, hipStream_t stream) {
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
                          sh.batch, sh.npm, p.rv, p.pass.mt_v, p.page_elems, p.value_base, pbuf,
                          elbuf, vpart, vel);
  else
    hipLaunchKernelGGL(kern, grid, dim3(512), lds, stream, static_cast<const bf16*>(pool),
                       num_pages, page_table, max_pages, seq_lens, sh.max_context, sh.chunk_pages,
                       sh.n_chunks, sh.n_rgroups, sh.batch, sh.npm, p.rv, p.pass.mt_v,
                       p.page_elems, p.value_base, pbuf, elbuf, vpart, vel);
  return hipGetLastError();
}

template <int RTMAX, int RGTW, int DP>
hipError_t launch_shared(const dckv_plan& p, const DecodeShape& sh, const void* pool,
                         int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                         const int32_t* seq_lens, const u32x4* pbuf, const u32x4* elbuf,
                         float* vpart, float* vel, hipStream_t stream) {
  auto kern = value_shared<RTMAX, RGTW, DP>;
  const size_t lds = pass_value_lds_bytes(p, RGTW);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  const int bc = sh.batch * sh.n_chunks;
  const dim3 grid(unsigned(8 * sh.n_rgroups * ((bc + 7) / 8)));
  const int RT = p.pass.n_slices * p.pass.nt;
  if (p.prof_before && p.prof_after)
    hipExtLaunchKernelGGL(kern, grid, dim3(512), uint32_t(lds), stream, p.prof_before, p.prof_after,
                          0u, static_cast<const bf16*>(pool), num_pages, page_table, max_pages,
                          seq_lens, sh.max_context, sh.chunk_pages, sh.n_chunks, sh.n_rgroups,
                          sh.batch, sh.npm, p.rv, p.pass.mt_v, p.page_elems, p.value_base, RT, pbuf,
                          elbuf, vpart, vel);
  else
    hipLaunchKernelGGL(kern, grid, dim3(512), lds, stream, static_cast<const bf16*>(pool), num_pages,
                       page_table, max_pages, seq_lens, sh.max_context, sh.chunk_pages, sh.n_chunks,
                       sh.n_rgroups, sh.batch, sh.npm, p.rv, p.pass.mt_v, p.page_elems, p.value_base,
                       RT, pbuf, elbuf, vpart, vel);
  return hipGetLastError();
}

// The shared-weights value pass for RT row tiles and RGTW value tiles a wave.
hipError_t launch_value_shared(const dckv_plan& p, const DecodeShape& sh, const void* pool,
                               int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                               const int32_t* seq_lens, const u32x4* pbuf, const u32x4* elbuf,
                               float* vpart, float* vel, hipStream_t stream) {
  const int RT = p.pass.n_slices * p.pass.nt;
#define DCKV_SHARED(RTMAX, RGTW, DP) \
  launch_shared<RTMAX, RGTW, DP>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, pbuf, elbuf, vpart, vel, stream)
  if (RT <= 4) return sh.rgt == 4 ? DCKV_SHARED(4, 4, 2) : DCKV_SHARED(4, 2, 4);
  if (RT <= 8) return sh.rgt == 2 ? DCKV_SHARED(8, 2, 3) : DCKV_SHARED(8, 1, 6);
#undef DCKV_SHARED
  return launch_shared<16, 1, 3>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, pbuf,
                                 elbuf, vpart, vel, stream);
}

template <int NT, int RING>
hipError_t launch_score_r(const dckv_plan& p, const DecodeShape& sh, const u32x4* qblk,
                          const void* pool, int64_t num_pages, const int32_t* page_table,
                          int32_t max_pages, const int32_t* seq_lens, uint32_t* pbuf, float* elbuf,
                          hipStream_t stream) {
  auto kern = score_pages<NT, RING>;
  const size_t lds = pass_score_lds_bytes(p);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  const int n_units = sh.batch * sh.units_per_seq;
  hipLaunchKernelGGL(kern, dim3(8 * p.pass.n_slices * ((n_units + 7) / 8)), dim3(512), lds, stream, qblk,
                     static_cast<const bf16*>(pool), num_pages, page_table, max_pages, seq_lens,
                     sh.max_context, sh.unit_pages, sh.units_per_seq, n_units, sh.npm, p.RK,
                     p.page_elems, pbuf, elbuf, p.pass);
  return hipGetLastError();
}

template <int NT>
hipError_t launch_score(const dckv_plan& p, const DecodeShape& sh, const u32x4* qblk,
                        const void* pool, int64_t num_pages, const int32_t* page_table,
                        int32_t max_pages, const int32_t* seq_lens, uint32_t* pbuf, float* elbuf,
                        hipStream_t stream) {
  switch (p.pass_ring) {
    case 16: return launch_score_r<NT, 16>(p, sh, qblk, pool, num_pages, page_table, max_pages, seq_lens, pbuf, elbuf, stream);
    case 32: return launch_score_r<NT, 32>(p, sh, qblk, pool, num_pages, page_table, max_pages, seq_lens, pbuf, elbuf, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_upproj(const dckv_plan& p, int32_t batch_rows, const float* amerged,
                         const void* R_value, float* out, hipStream_t stream) {
  // column tiles of 16 when tiles of 32 would leave most compute units idle
  const int rows = batch_rows * p.qpk;
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
  uint32_t* pbuf = reinterpret_cast<uint32_t*>(ws + sh.off_p);
  float* elbuf = reinterpret_cast<float*>(ws + sh.off_el);
  float* vpart = reinterpret_cast<float*>(ws + sh.off_acc);
  float* vel = reinterpret_cast<float*>(ws + sh.off_ml);
  float* amerged = reinterpret_cast<float*>(ws + sh.off_opart);
  hipError_t e = launch_fold(p, p.pass, sh.batch, q, R_keys, qt, stream);
  if (e != hipSuccess) return e;
  e = p.pass.nt == 1 ? launch_score<1>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens,
                                       pbuf, elbuf, stream)
                     : launch_score<2>(p, sh, qt, pool, num_pages, page_table, max_pages, seq_lens,
                                       pbuf, elbuf, stream);
  if (e != hipSuccess) return e;
  const u32x4* pb4 = reinterpret_cast<const u32x4*>(pbuf);
  const u32x4* el4 = reinterpret_cast<const u32x4*>(elbuf);
#define DCKV_VALUE(NT, RGT) \
  launch_value<NT, RGT>(p, sh, pool, num_pages, page_table, max_pages, seq_lens, pb4, el4, vpart, vel, stream)
  if (p.pass.n_slices > 1)
    e = launch_value_shared(p, sh, pool, num_pages, page_table, max_pages, seq_lens, pb4, el4, vpart,
                            vel, stream);
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
