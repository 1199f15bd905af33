// Rotary decode on MFMA (gfx950).
//
// With rotary position embedding a key is Rot(t)(z_t R_{g,h}): the rotation
// depends on the token's position, so the query can no longer be folded
// into the latent space once for all tokens (the fold of Sec. III-A,
// q (z R)^T = (q R^T) z^T, needs one R for every token).  The keys are
// rebuilt per token instead, turned, and dotted with the turned query.
//
// rope_factors: R_{g,h}^T of every KV head copied into 16 x 32 bf16 blocks in
//   MFMA A-operand order, one block per (32-column key chunk meeting the
//   group's columns, 16 rows of d_h), zero outside the group's columns.
// rope_scores_res (groups whose factor blocks fit LDS) and rope_scores (any
//   group): per (sequence, context splits, KV head) a work-group's waves
//   each take one 64-token page at a time and form K^T[dim][tok] +=
//   R^T[dim][k] Z[tok][k] over the group's key chunks on MFMA 16x16x32 bf16
//   (exact bf16 products, fp32 sums), the factor blocks read from LDS.  A
//   page done, each plane (i, i + d_h/2) is turned by the token's angle and
//   the key is dotted with the KV head's turned, scaled queries.  Per split
//   the work-group writes, per query head, the split maximum m, the weights
//   2^(s - m) rounded to bf16, and their sum l: the split's partial softmax,
//   in the form the value pass and the merge of the position-free decode
//   take.  rope_scores_res keeps the head's blocks resident for its whole
//   range of splits; rope_scores stages one chunk's blocks a step.
#include <cmath>

#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxQpk = 8;               // query heads a KV head
constexpr int kRopeMaxSplit = 1024;      // context tokens a split
constexpr int kDepth = 4;                // key chunks in flight ahead of the MFMAs
constexpr int kRsrcWord3 = 0x00020000;   // raw buffer descriptor word 3 (gfx9 family)
constexpr int kNonTemporal = 2;
constexpr int kOutOfRange = 0x40000000;   // byte offset beyond any page: the load reads zero
constexpr double kInv2Pi = 0.15915494309189533577;
constexpr int kResWaves = 8;              // waves of the resident-factor kernel
constexpr int kResFacElems = 57344;       // its LDS factor blocks: 112 KB of bf16
constexpr int kResMaxPages = 128;         // pages a work-group of it
constexpr int kResTargetGroups = 1024;    // work-groups it aims for (four a compute unit)
constexpr int kResScores = 8192;          // scores of a work-group's range in LDS
constexpr int kResDepth = 3;              // its key chunks in flight a wave

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

__device__ __forceinline__ floatx4 mfma(u32x4 a, u32x4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Keep the first n (0..8) bf16 of a 16-byte vector, zero the rest.
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

// cos and sin of the angle pos * theta, theta = 2 pi omega: the turns
// pos * omega are formed and reduced to [-1/2, 1/2] in fp64 (exact enough
// for any int32 position), then v_cos/v_sin take the fraction of a turn.
__device__ __forceinline__ void turn(int pos, double omega, float& c, float& s) {
  double x = double(pos) * omega;
  x -= rint(x);
  const float f = float(x);
  c = __builtin_amdgcn_cosf(f);
  s = __builtin_amdgcn_sinf(f);
}

// ---------------------------------------------------------------------------
// Grid (blocks of 256 threads over the head's transposed blocks, KV heads).
// Thread: one lane of one 16 x 32 block: row 16 it + l % 16 of R^T (a column
// of R_{g,h}), key columns 32 c + 8 (l / 16) .. + 7.
__global__ __launch_bounds__(256) void rope_factors(const bf16* __restrict__ Rk,
                                                    bf16* __restrict__ rt, RopeTables tb) {
  const int kv = blockIdx.y;
  const int e = blockIdx.x * 256 + threadIdx.x;
  const int dt = tb.head_dim / 16;
  const int koff = tb.koff[kv], rank = tb.rank[kv];
  const int c_lo = koff >> 5, nch = ((koff + rank - 1) >> 5) - c_lo + 1;
  const int blk = e >> 6, l = e & 63;
  if (blk >= nch * dt) return;
  const int ci = blk / dt, it = blk % dt;
  const int dim = 16 * it + (l & 15);
  const int col0 = 32 * (c_lo + ci) + 8 * (l >> 4);
  const bf16* src = Rk + tb.roff[kv] + tb.rcol[kv] + dim;
  uint32_t w[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t half[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int col = col0 + 2 * j + k;
      uint16_t bits = 0;
      if (col >= koff && col < koff + rank)
        bits = __builtin_bit_cast(uint16_t, src[int64_t(col - koff) * tb.rstride[kv]]);
      half[k] = bits;
    }
    w[j] = half[0] | (half[1] << 16);
  }
  *reinterpret_cast<u32x4*>(rt + tb.rt_off[kv] + int64_t(blk) * 512 + l * 8) = u32x4{w[0], w[1], w[2], w[3]};
}

// ---------------------------------------------------------------------------
// A wave's rebuilt page -> scores.  acc[it][n] holds K^T rows 16 it + 4 lq + v
// (v = 0..3) of tokens 16 n + lr.  Each plane (a, a + D/2) is turned by the
// token's angle, then the key is dotted with each query (qr: turned and
// scaled, rows of D floats); lane lq == 0 writes the score of token 16 n + lr
// to sc[hh * stride + off + 16 n + lr], or -inf past nval or on an empty
// page.  The angle of a plane is formed once a page (token pos0 + lr) and
// stepped to the lane's other tokens, 16 apart, by the turn through 16
// theta_a (cs16[a]: its cosine and sine).
template <int DT>
__device__ __forceinline__ void page_scores(floatx4 (&acc)[DT][4], int pos0, int nval, bool pvalid,
                                            const double* omega, const float2* cs16,
                                            const float* qr, int qpk, float* sc, int stride,
                                            int off, int lane) {
  constexpr int D = 16 * DT, HALF = DT / 2;
  const int lr = lane & 15, lq = lane >> 4;
#pragma unroll
  for (int it = 0; it < HALF; ++it)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int a = 16 * it + 4 * lq + v;
      float cs, sn;
      turn(pos0 + lr, omega[a], cs, sn);
      const float2 st = cs16[a];
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const float ka = acc[it][n][v], kb = acc[it + HALF][n][v];
        acc[it][n][v] = ka * cs - kb * sn;
        acc[it + HALF][n][v] = kb * cs + ka * sn;
        if (n < 3) {
          const float c2 = cs * st.x - sn * st.y;
          sn = sn * st.x + cs * st.y;
          cs = c2;
        }
      }
    }
  for (int hh = 0; hh < qpk; ++hh) {
    float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int it = 0; it < DT; ++it) {
      const floatx4 qa = *reinterpret_cast<const floatx4*>(qr + hh * D + 16 * it + 4 * lq);
#pragma unroll
      for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int v = 0; v < 4; ++v) part[n] = fmaf(qa[v], acc[it][n][v], part[n]);
    }
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      float x = part[n];
      x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      const int tok = 16 * n + lr;
      if (lq == 0) sc[hh * stride + off + tok] = (pvalid && tok < nval) ? x : -INFINITY;
    }
  }
}

// The split's partial softmax from its scores (sc, ntok tokens per query
// head): per query head the maximum m, the weights 2^(s - m) rounded to
// bf16 (written to the head's row of pbuf) and their sum l in a fixed order.
// NW waves; every thread of the work-group calls it.
template <int NW>
__device__ __forceinline__ void split_softmax(const float* sc, int ntok, int qpk, int kv, int b,
                                              int split, int n_split, int split_tokens,
                                              int n_slices, const RopeTables& tb, bf16* pbuf,
                                              float* part_ml, float* redm, float* redl) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nh = tb.nh;
  for (int hh = 0; hh < qpk; ++hh) {
    const int qs = tb.qslot[kv * qpk + hh];
    const int slice = qs >> 5, j = qs & 31;
    const int64_t prow = (int64_t(b) * n_slices + slice) * n_split + split;
    const float* srow = sc + hh * kRopeMaxSplit;
    float mx = -INFINITY;
    for (int t = tid; t < ntok; t += NW * 64) mx = fmaxf(mx, srow[t]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    if (lane == 0) redm[w] = mx;
    __syncthreads();
    float m = redm[0];
#pragma unroll
    for (int k = 1; k < NW; ++k) m = fmaxf(m, redm[k]);
    bf16* prow_p = pbuf + (prow * nh + j) * split_tokens;
    float ls = 0.f;
    for (int t = tid; t < ntok; t += NW * 64) {
      const float sv = srow[t];
      const float pv = (sv == -INFINITY) ? 0.f : exp2f(sv - m);
      const bf16 pb = static_cast<bf16>(pv);
      ls += static_cast<float>(pb);
      prow_p[t] = pb;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ls += __shfl_xor(ls, o);
    if (lane == 0) redl[w] = ls;
    __syncthreads();
    if (tid == 0) {
      float l = redl[0];
#pragma unroll
      for (int k = 1; k < NW; ++k) l += redl[k];
      float* pml = part_ml + prow * (2 * nh);
      pml[j] = m;
      pml[nh + j] = l;
    }
  }
}

// One wave's partial softmax of one split for one query head: srow holds
// the split's ntok scores; maximum, bf16 weights and their sum (lane sums
// in a fixed order, then a fixed butterfly), written as split_softmax does.
__device__ __forceinline__ void wave_split_softmax(const float* srow, int ntok, int qs, int b,
                                                   int split, int n_split, int split_tokens,
                                                   int n_slices, int nh, bf16* pbuf,
                                                   float* part_ml, int lane) {
  const int slice = qs >> 5, j = qs & 31;
  const int64_t prow = (int64_t(b) * n_slices + slice) * n_split + split;
  float m = -INFINITY;
  for (int t = lane; t < ntok; t += 64) m = fmaxf(m, srow[t]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  bf16* prow_p = pbuf + (prow * nh + j) * split_tokens;
  float ls = 0.f;
  for (int t = lane; t < ntok; t += 64) {
    const float sv = srow[t];
    const float pv = (sv == -INFINITY) ? 0.f : exp2f(sv - m);
    const bf16 pb = static_cast<bf16>(pv);
    ls += static_cast<float>(pb);
    prow_p[t] = pb;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ls += __shfl_xor(ls, o);
  if (lane == 0) {
    float* pml = part_ml + prow * (2 * nh);
    pml[j] = m;
    pml[nh + j] = ls;
  }
}

// ---------------------------------------------------------------------------
// The general kernel (any group width): the chunk's factor blocks staged per
// step.  DT: 16-row tiles of d_h (4 for d_h = 64, 8 for d_h = 128).
//
// Pipeline: the work-group's steps run over (page round, key chunk); step
// s stages the factor blocks of the next chunk into the LDS buffer the
// previous step freed, and multiplies the current chunk.  Each wave issues,
// per step, the factor loads for the chunk kDepth + 1 steps ahead and its
// own page's key loads for the chunk kDepth steps ahead, so the two streams
// come due in the order they were issued and one wait never holds back a
// younger load.
template <int DT>
__global__ __launch_bounds__(256, 1) void rope_scores(
    const float* __restrict__ q, const bf16* __restrict__ pool, int64_t num_pages,
    const int32_t* __restrict__ page_table, int max_pages, const int32_t* __restrict__ seq_lens,
    int max_context, int split_tokens, int n_split, int n_work, const bf16* __restrict__ rt,
    int RK, int64_t page_elems, double log2_base, float scale, int n_slices,
    bf16* __restrict__ pbuf, float* __restrict__ part_ml, RopeTables tb) {
  constexpr int D = 16 * DT, HALF = DT / 2;
  constexpr int FPT = DT / 4;                     // 16-byte factor loads a thread per chunk
  constexpr int P = kDepth;
  static_assert(P % 2 == 0, "the LDS buffer of a step is its parity");
  __shared__ __align__(16) bf16 fac[2][DT * 512];
  __shared__ __align__(16) float qr[kMaxQpk][D];
  __shared__ __align__(16) float sc[kMaxQpk][kRopeMaxSplit];
  __shared__ double omega[D / 2];
  __shared__ float2 cs16[D / 2];
  __shared__ int pids[kRopeMaxSplit / 64];
  __shared__ float redm[4], redl[4];

  // XCD-aware order: ids id, id + 8, ... (one XCD) take consecutive work
  // items, and consecutive items are the KV heads of one split, group by
  // group, so a group's key chunks are read from one L2
  const int id = blockIdx.x;
  const int xcd = id & 7, qq = id >> 3;
  const int per = n_work >> 3, extra = n_work & 7;
  const int wi = xcd * per + min(xcd, extra) + qq;
  const int Hkv = tb.n_kv_heads, qpk = tb.q_per_kv;
  const int kv = tb.work_kv[wi % Hkv];
  const int u = wi / Hkv;
  const int b = u / n_split, split = u % n_split;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lq = lane >> 4;

  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int t0 = split * split_tokens;
  const int t1 = min(t0 + split_tokens, T_b);
  if (t0 >= t1) return;                           // the merge reads only splits holding tokens
  const int np = (t1 - t0 + 63) >> 6;
  const int koff = tb.koff[kv], rank = tb.rank[kv];
  const int c_lo = koff >> 5, nch = ((koff + rank - 1) >> 5) - c_lo + 1;
  const bf16* rth = rt + tb.rt_off[kv];
  const int kc_last = (RK - 1) >> 5;
  const int kvalid_last = min(8, max(0, RK - (32 * kc_last + 8 * lq)));

  // ---- prologue: plane frequencies, the split's pages, turned queries
  if (tid < D / 2) {
    const double om = exp2(-(2.0 * tid / D) * log2_base) * kInv2Pi;
    omega[tid] = om;
    float c16, s16;
    turn(16, om, c16, s16);
    cs16[tid] = make_float2(c16, s16);
  }
  if (tid < np) {
    const int pg = page_table[int64_t(b) * max_pages + (t0 >> 6) + tid];
    pids[tid] = (pg >= 0 && pg < num_pages) ? pg : -1;
  }
  __syncthreads();
  {
    const int pq = T_b - 1;                       // the decode query: the newest position
    const int Hq = Hkv * qpk;
    for (int e = tid; e < qpk * (D / 2); e += 256) {
      const int hh = e / (D / 2), i = e % (D / 2);
      const float* qh = q + (int64_t(b) * Hq + kv * qpk + hh) * D;
      float c, s;
      turn(pq, omega[i], c, s);
      const float xa = qh[i], xb = qh[i + D / 2];
      qr[hh][i] = (xa * c - xb * s) * scale;
      qr[hh][i + D / 2] = (xb * c + xa * s) * scale;
    }
  }

  // ---- producer state: step index -> (round, chunk); a round is four pages
  const int rounds = (np + 3) >> 2;
  const int total = rounds * nch;
  const int page_bytes = int(page_elems * 2);
  const int lane_key = 2 * ((16 * 0 + lr) * 32 + 8 * lq);   // token tile 0 of the page
  auto page_rsrc = [&](int round) {
    const int pg = 4 * round + w;
    int pid = -1;
    if (pg < np) pid = __builtin_amdgcn_readfirstlane(pids[pg]);
    const bf16* base = pid >= 0 ? pool + int64_t(pid) * page_elems : pool;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(base), 0, pid >= 0 ? page_bytes : 0,
                                             kRsrcWord3);
  };
  // factor loads of chunk c (clamped: a step past the end reloads the last chunk)
  auto load_fac = [&](u32x4 (&f)[FPT], int c) {
    const bf16* src = rth + int64_t(min(c, nch - 1)) * (DT * 512);
#pragma unroll
    for (int k = 0; k < FPT; ++k) f[k] = *reinterpret_cast<const u32x4*>(src + (tid + 256 * k) * 8);
  };
  auto store_fac = [&](const u32x4 (&f)[FPT], int buf) {
#pragma unroll
    for (int k = 0; k < FPT; ++k) *reinterpret_cast<u32x4*>(&fac[buf][(tid + 256 * k) * 8]) = f[k];
  };
  // key loads of the wave's page for chunk c: four token tiles
  auto load_key = [&](u32x4 (&z)[4], __amdgpu_buffer_rsrc_t rs, int c) {
    const int o = 2 * 2048 * (c_lo + min(c, nch - 1)) + lane_key;
#pragma unroll
    for (int n = 0; n < 4; ++n)
      z[n] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, o + 2 * 512 * n, 0, kNonTemporal));
  };

  // ---- fill: chunk 0's factors straight to LDS, then kDepth steps of loads
  u32x4 fr[P][FPT];
  u32x4 zr[P][4];
  int is_c = 0, is_round = 0;                     // issue position (key stream)
  __amdgpu_buffer_rsrc_t is_rs = page_rsrc(0);
  {
    u32x4 f0[FPT];
    load_fac(f0, 0);
    store_fac(f0, 0);
  }
#pragma unroll
  for (int s = 0; s < P; ++s) {
    load_fac(fr[s], (s + 1) % nch);
    load_key(zr[s], is_rs, is_c);
    if (++is_c == nch) {
      is_c = 0;
      is_rs = page_rsrc(++is_round);
    }
  }

  floatx4 acc[DT][4];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};

  int c = 0, round = 0;                           // consume position
  for (int s0 = 0; s0 < total; s0 += P) {
#pragma unroll
    for (int s = 0; s < P; ++s) {
      if (s0 + s < total) {                       // uniform over the work-group
        // step s0 + s reads buffer s & 1 (P is even, so the step's parity is s's)
        __syncthreads();                          // fac[s & 1] complete; fac[(s + 1) & 1] free
        store_fac(fr[s], (s + 1) & 1);            // next step's factors (possibly the next round's chunk 0)
        load_fac(fr[s], (c + 1 + P) % nch);
        {
          u32x4 zn[4];
          load_key(zn, is_rs, is_c);
          u32x4 z[4];
#pragma unroll
          for (int n = 0; n < 4; ++n) {
            z[n] = zr[s][n];
            zr[s][n] = zn[n];
          }
          if (++is_c == nch) {
            is_c = 0;
            is_rs = page_rsrc(++is_round);
          }
          if (c_lo + c == kc_last) {
#pragma unroll
            for (int n = 0; n < 4; ++n) z[n] = keep_first(z[n], kvalid_last);
          }
          const bf16* A = fac[s & 1];
#pragma unroll
          for (int it = 0; it < DT; ++it) {
            const u32x4 a = *reinterpret_cast<const u32x4*>(A + it * 512 + lane * 8);
#pragma unroll
            for (int n = 0; n < 4; ++n) acc[it][n] = mfma(a, z[n], acc[it][n]);
          }
        }
        if (c == nch - 1) {                       // the round's pages are rebuilt
          const int pg = 4 * round + w;
          if (pg < np)
            page_scores<DT>(acc, t0 + 64 * pg, min(64, (t1 - t0) - 64 * pg), pids[pg] >= 0, omega,
                            cs16, &qr[0][0], qpk, &sc[0][0], kRopeMaxSplit, 64 * pg, lane);
#pragma unroll
          for (int i = 0; i < DT; ++i)
#pragma unroll
            for (int n = 0; n < 4; ++n) acc[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};
          c = 0;
          ++round;
        } else {
          ++c;
        }
      }
    }
  }
  __syncthreads();

  // ---- the split's partial softmax, one query head at a time
  split_softmax<4>(&sc[0][0], 64 * np, qpk, kv, b, split, n_split, split_tokens, n_slices, tb, pbuf,
                   part_ml, redm, redl);
}


// ---------------------------------------------------------------------------
// The resident-factor kernel, for groups whose transposed factor blocks fit
// LDS (at most kResFacElems elements: 14 key chunks at d_h = 128, 28 at 64).
// One 512-thread work-group (eight waves, two a SIMD, so one wave's turning
// and dot products overlap the other's MFMAs) per (sequence, range of spw
// context splits, KV head).  The head's blocks are staged in LDS once; the
// waves then run through the range's pages independently, eight pages a
// round, each wave with its own page and its own ring of key loads kResDepth
// chunks ahead.  Scores of the whole range stay in LDS (qpk * spw * L <=
// kResScores floats); at the end each wave takes whole splits for their
// softmax, so the waves meet only twice: after staging and before the tail.
template <int DT>
__global__ __launch_bounds__(512, 1) void rope_scores_res(
    const float* __restrict__ q, const bf16* __restrict__ pool, int64_t num_pages,
    const int32_t* __restrict__ page_table, int max_pages, const int32_t* __restrict__ seq_lens,
    int max_context, int split_tokens, int n_split, int spw, int n_ranges, int n_work,
    const bf16* __restrict__ rt, int RK, int64_t page_elems, double log2_base, float scale,
    int n_slices, bf16* __restrict__ pbuf, float* __restrict__ part_ml, RopeTables tb) {
  constexpr int W = kResWaves, D = 16 * DT, P = kResDepth;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16* fac = reinterpret_cast<bf16*>(smem);                                // [nch][DT][512]
  float* sc = reinterpret_cast<float*>(smem + size_t(kResFacElems) * 2);    // [qpk][spw * L]
  float* qr = sc + kResScores;                                              // [kMaxQpk][D]
  double* omega = reinterpret_cast<double*>(qr + kMaxQpk * D);              // [D/2]
  float2* cs16 = reinterpret_cast<float2*>(omega + D / 2);                  // [D/2]
  int* pids = reinterpret_cast<int*>(cs16 + D / 2);                         // [kResMaxPages]

  // XCD-aware order as in rope_scores: the KV heads of one (sequence, range)
  // are consecutive items on one XCD
  const int id = blockIdx.x;
  const int xcd = id & 7, qq = id >> 3;
  const int per = n_work >> 3, extra = n_work & 7;
  const int wi = xcd * per + min(xcd, extra) + qq;
  const int Hkv = tb.n_kv_heads, qpk = tb.q_per_kv;
  const int kv = tb.work_kv[wi % Hkv];
  const int u = wi / Hkv;
  const int b = u / n_ranges, rg = u % n_ranges;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lq = lane >> 4, lr = lane & 15;

  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int L = split_tokens;
  const int s_lo = rg * spw;
  const int t0w = s_lo * L;
  const int t1w = min(T_b, min(n_split, s_lo + spw) * L);
  if (t0w >= t1w) return;
  const int npw = (t1w - t0w + 63) >> 6;           // pages of the range (<= kResMaxPages)
  const int nsp = (t1w - t0w + L - 1) / L;         // splits holding tokens
  const int pps = L >> 6;                          // pages a split
  const int rps = (pps + W - 1) / W;               // rounds a split
  const int koff = tb.koff[kv], rank = tb.rank[kv];
  const int c_lo = koff >> 5, nch = ((koff + rank - 1) >> 5) - c_lo + 1;
  const bf16* rth = rt + tb.rt_off[kv];
  const int kc_last = (RK - 1) >> 5;
  const int kvalid_last = min(8, max(0, RK - (32 * kc_last + 8 * lq)));

  // ---- prologue: frequencies and pages; then the turned queries and the
  // head's factor blocks (eight 16-byte loads in flight a thread)
  if (tid < D / 2) {
    const double om = exp2(-(2.0 * tid / D) * log2_base) * kInv2Pi;
    omega[tid] = om;
    float c16, s16;
    turn(16, om, c16, s16);
    cs16[tid] = make_float2(c16, s16);
  }
  if (tid < npw) {
    const int pg = page_table[int64_t(b) * max_pages + (t0w >> 6) + tid];
    pids[tid] = (pg >= 0 && pg < num_pages) ? pg : -1;
  }
  __syncthreads();
  {
    const int pq = T_b - 1;
    const int Hq = Hkv * qpk;
    for (int e = tid; e < qpk * (D / 2); e += W * 64) {
      const int hh = e / (D / 2), i = e % (D / 2);
      const float* qh = q + (int64_t(b) * Hq + kv * qpk + hh) * D;
      float c, s;
      turn(pq, omega[i], c, s);
      const float xa = qh[i], xb = qh[i + D / 2];
      qr[hh * D + i] = (xa * c - xb * s) * scale;
      qr[hh * D + i + D / 2] = (xb * c + xa * s) * scale;
    }
    const int nvec = nch * DT * 64;
    for (int base = tid; base < nvec; base += 8 * W * 64) {
      u32x4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        v[k] = *reinterpret_cast<const u32x4*>(rth + 8 * min(base + k * W * 64, nvec - 1));
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (base + k * W * 64 < nvec) *reinterpret_cast<u32x4*>(fac + 8 * (base + k * W * 64)) = v[k];
    }
  }
  __syncthreads();

  // ---- steps: (split, round, chunk); this wave's page of a round is
  // round * W + w of the split.  A round is padded to nchp = a multiple of P
  // chunks, so a loop body is P chunks of one round and the page's scores
  // follow the body that ends the round: the loads of every step are issued
  // on every path (a padding chunk's load is out of range and reads zero)
  // and each wait is for its own ring slot only.
  const int nchp = (nch + P - 1) / P * P;
  const int total = nsp * rps * nchp;
  const int page_bytes = int(page_elems * 2);
  const int lane_key = 2 * (lr * 32 + 8 * lq);
  auto page_rsrc = [&](int sp, int r) {
    const int pgi = r * W + w;
    const int idx = sp * pps + pgi;
    int pid = -1;
    if (pgi < pps && idx < npw) pid = __builtin_amdgcn_readfirstlane(pids[idx]);
    const bf16* base = pid >= 0 ? pool + int64_t(pid) * page_elems : pool;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(base), 0, pid >= 0 ? page_bytes : 0,
                                             kRsrcWord3);
  };
  auto load_key = [&](u32x4 (&z)[4], __amdgpu_buffer_rsrc_t rs, int c) {
    const int o = c < nch ? 2 * 2048 * (c_lo + c) + lane_key : kOutOfRange;
#pragma unroll
    for (int n = 0; n < 4; ++n)
      z[n] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, o + 2 * 512 * n, 0, kNonTemporal));
  };
  u32x4 zr[P][4];
  int is_c = 0, is_r = 0, is_s = 0;
  __amdgpu_buffer_rsrc_t is_rs = page_rsrc(0, 0);
  auto advance_issue = [&]() {
    if (++is_c == nchp) {
      is_c = 0;
      if (++is_r == rps) {
        is_r = 0;
        ++is_s;
      }
      is_rs = page_rsrc(is_s, is_r);
    }
  };
#pragma unroll
  for (int s = 0; s < P; ++s) {
    load_key(zr[s], is_rs, is_c);
    advance_issue();
  }

  floatx4 acc[DT][4];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};

  int c0 = 0, r = 0, sp = 0;                       // consume position: first chunk of the body
  for (int s0 = 0; s0 < total; s0 += P) {
#pragma unroll
    for (int s = 0; s < P; ++s) {
      const int c = c0 + s;
      if (c < nch) {                               // a real chunk (uniform)
        if (c_lo + c == kc_last) {
#pragma unroll
          for (int n = 0; n < 4; ++n) zr[s][n] = keep_first(zr[s][n], kvalid_last);
        }
        const bf16* A = fac + c * (DT * 512) + lane * 8;
        u32x4 a[DT];                               // the step's factor fragments, all in flight
#pragma unroll
        for (int it = 0; it < DT; ++it) a[it] = *reinterpret_cast<const u32x4*>(A + it * 512);
#pragma unroll
        for (int it = 0; it < DT; ++it)
#pragma unroll
          for (int n = 0; n < 4; ++n) acc[it][n] = mfma(a[it], zr[s][n], acc[it][n]);
        __builtin_amdgcn_sched_group_barrier(0x100, DT, 0);      // the DT LDS reads first,
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * DT, 0);  // then the step's MFMAs
      }
      // the slot is used in place and reloaded after its MFMAs: no register
      // copy ties a wait to the loads just issued
      load_key(zr[s], is_rs, is_c);                // past the range: an empty page, reads zero
      advance_issue();
    }
    c0 += P;
    if (c0 == nchp) {                              // the wave's page of the round is rebuilt
      const int pgi = r * W + w;
      const int pos0 = t0w + sp * L + 64 * pgi;
      if (pgi < pps && pos0 < t1w)
        page_scores<DT>(acc, pos0, min(64, t1w - pos0), pids[sp * pps + pgi] >= 0, omega, cs16,
                        qr, qpk, sc, spw * L, sp * L + 64 * pgi, lane);
#pragma unroll
      for (int i = 0; i < DT; ++i)
#pragma unroll
        for (int n = 0; n < 4; ++n) acc[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};
      c0 = 0;
      if (++r == rps) {
        r = 0;
        ++sp;
      }
    }
  }

  // ---- the splits' partial softmaxes: wave w takes splits w, w + W, ...
  __syncthreads();
  for (int k = w; k < nsp * qpk; k += W) {
    const int spk = k / qpk, hh = k % qpk;
    const int ntok = min(L, t1w - (t0w + spk * L));
    wave_split_softmax(sc + hh * (spw * L) + spk * L, (ntok + 63) & ~63,
                       tb.qslot[kv * qpk + hh], b, s_lo + spk, n_split, L, n_slices, tb.nh, pbuf,
                       part_ml, lane);
  }
}

}  // namespace

DecodeShape rope_shape(const dckv_plan& p, int32_t batch, int32_t max_context) {
  DecodeShape s = decode_shape(p, batch, max_context);
  // the split's scores and weights live in LDS: at most kRopeMaxSplit tokens
  int64_t L = std::min<int64_t>(s.split_tokens, kRopeMaxSplit);
  s.split_tokens = int32_t(L);
  s.n_split = max_context > 0 ? int32_t((max_context + L - 1) / L) : 1;
  const int64_t units = int64_t(batch) * s.n_split;
  s.n_units = int32_t((units + 7) / 8 * 8);
  s.merge_ranks = mfma_merge_ranks(p, batch);
  s.n_rchunks = (p.rv + s.merge_ranks - 1) / s.merge_ranks;
  const size_t nh = 16 * size_t(p.mfma.nt);
  const size_t rows = size_t(batch) * p.mfma.n_slices * s.n_split;
  s.off_qt = 0;
  s.off_rt = 0;
  s.off_p = align_up(size_t(p.rope_rt_elems) * 2, 256);
  s.off_ml = s.off_p + align_up(rows * nh * size_t(L) * 2, 256);
  s.off_acc = s.off_ml + align_up(rows * 2 * nh * sizeof(float), 256);
  s.off_opart = s.off_acc + align_up(rows * nh * size_t(p.rv) * sizeof(float), 256);
  s.bytes = s.off_opart + align_up(size_t(batch) * p.Hq * p.rv * sizeof(float), 256);
  return s;
}

int rope_max_split_tokens() { return kRopeMaxSplit; }
int rope_max_q_per_kv() { return kMaxQpk; }

hipError_t launch_rope_factors(const dckv_plan& p, const void* R_keys, void* rt, hipStream_t stream) {
  int max_blocks = 0;
  for (int kv = 0; kv < p.Hkv; ++kv) {
    const int koff = p.rope.koff[kv], rank = p.rope.rank[kv];
    const int nch = ((koff + rank - 1) >> 5) - (koff >> 5) + 1;
    max_blocks = std::max(max_blocks, nch * (p.dh / 16));
  }
  hipLaunchKernelGGL(rope_factors, dim3((max_blocks * 64 + 255) / 256, p.Hkv), dim3(256), 0, stream,
                     static_cast<const bf16*>(R_keys), static_cast<bf16*>(rt), p.rope);
  return hipGetLastError();
}

size_t rope_res_lds_bytes(int dh) {
  return size_t(kResFacElems) * 2 + size_t(kResScores) * 4 + size_t(kMaxQpk) * dh * 4 +
         size_t(dh / 2) * 16 + kResMaxPages * 4;
}

hipError_t launch_rope_scores(const dckv_plan& p, const DecodeShape& sh, const float* q,
                              const void* pool, int64_t num_pages, const int32_t* page_table,
                              int32_t max_pages, const int32_t* seq_lens, const void* rt,
                              double rope_base, void* pbuf, float* part_ml, hipStream_t stream) {
  const double log2_base = std::log2(rope_base);
  const float scale = kLog2e / std::sqrt(float(p.dh));
  const bool events = p.prof_before && p.prof_after;   // stamped by the kernel's own dispatch
  int max_nch = 0;
  for (int kv = 0; kv < p.Hkv; ++kv) {
    const int koff = p.rope.koff[kv], rank = p.rope.rank[kv];
    max_nch = std::max(max_nch, ((koff + rank - 1) >> 5) - (koff >> 5) + 1);
  }
  const int L = sh.split_tokens, pps = L / 64;
  if (max_nch * (p.dh / 16) * 512 <= kResFacElems) {
    // several splits a work-group, about kResTargetGroups work-groups in all
    const int64_t units = int64_t(sh.batch) * p.Hkv * sh.n_split;
    int spw = int(std::max<int64_t>(1, units / kResTargetGroups));
    spw = std::min(spw, std::max(1, std::min(kResMaxPages / pps, 4096 / L)));
    spw = std::min(spw, kResScores / (p.qpk * L));   // the range's scores fit LDS (qpk * L <= 8192)
    const int n_ranges = (sh.n_split + spw - 1) / spw;
    const int n_work = sh.batch * n_ranges * p.Hkv;
    const size_t lds = rope_res_lds_bytes(p.dh);
    auto go = [&](auto kern) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
      if (e != hipSuccess) return e;
      if (events)
        hipExtLaunchKernelGGL(kern, dim3(n_work), dim3(kResWaves * 64), uint32_t(lds), stream,
                              p.prof_before, p.prof_after, 0u, q, static_cast<const bf16*>(pool),
                              num_pages, page_table, max_pages, seq_lens, sh.max_context, L,
                              sh.n_split, spw, n_ranges, n_work, static_cast<const bf16*>(rt), p.RK,
                              p.page_elems, log2_base, scale, p.mfma.n_slices,
                              static_cast<bf16*>(pbuf), part_ml, p.rope);
      else
        hipLaunchKernelGGL(kern, dim3(n_work), dim3(kResWaves * 64), lds, stream, q,
                           static_cast<const bf16*>(pool), num_pages, page_table, max_pages,
                           seq_lens, sh.max_context, L, sh.n_split, spw, n_ranges, n_work,
                           static_cast<const bf16*>(rt), p.RK, p.page_elems, log2_base, scale,
                           p.mfma.n_slices, static_cast<bf16*>(pbuf), part_ml, p.rope);
      return hipGetLastError();
    };
    if (p.dh == 128) return go(rope_scores_res<8>);
    if (p.dh == 64) return go(rope_scores_res<4>);
    return hipErrorInvalidValue;
  }
  const int n_work = sh.batch * sh.n_split * p.Hkv;
  auto go = [&](auto kern) {
    if (events)
      hipExtLaunchKernelGGL(kern, dim3(n_work), dim3(256), 0, stream, p.prof_before, p.prof_after,
                            0u, q, static_cast<const bf16*>(pool), num_pages, page_table, max_pages,
                            seq_lens, sh.max_context, sh.split_tokens, sh.n_split, n_work,
                            static_cast<const bf16*>(rt), p.RK, p.page_elems, log2_base, scale,
                            p.mfma.n_slices, static_cast<bf16*>(pbuf), part_ml, p.rope);
    else
      hipLaunchKernelGGL(kern, dim3(n_work), dim3(256), 0, stream, q,
                         static_cast<const bf16*>(pool), num_pages, page_table, max_pages, seq_lens,
                         sh.max_context, sh.split_tokens, sh.n_split, n_work,
                         static_cast<const bf16*>(rt), p.RK, p.page_elems, log2_base, scale,
                         p.mfma.n_slices, static_cast<bf16*>(pbuf), part_ml, p.rope);
    return hipGetLastError();
  };
  if (p.dh == 128) return go(rope_scores<8>);
  if (p.dh == 64) return go(rope_scores<4>);
  return hipErrorInvalidValue;
}

}  // namespace dckv
