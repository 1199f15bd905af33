// Decode attention over the compressed cache without rebuilding keys or
// values (read side of Sec. III-A, x W ~ z R):
//   fold   q~_h = q_h R_{g,h}^T * log2(e)/sqrt(d_h)   (Sec. III-C group factor)
//   split  per (sequence, head, context split): scores s_t = q~_h . z_{g,t},
//          online softmax in base 2, acc = sum_t p_t z_{v,t} in value-latent
//          space (Sec. III-D shared value latent)
//   merge  fixed ascending-split log-sum-exp merge, then o_h = (acc / l)
//          R_v[:, kv(h) block] (one up-projection per head)
#include <algorithm>
#include <vector>
#include <cmath>

#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

constexpr int kThreads = 256;
constexpr int kTargetWorkgroups = 256;    // MI355X compute units
constexpr int32_t kValuSplitTokens = 1024;
constexpr int kAccPerThread = DCKV_MAX_VALUE_RANK / kThreads;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ---------------------------------------------------------------- fold
template <typename T>
__global__ __launch_bounds__(kThreads) void fold_kernel(const float* __restrict__ q,
                                                        const T* __restrict__ Rk,
                                                        float* __restrict__ qt, HeadTables tb,
                                                        float scale) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int dh = tb.head_dim;
  __shared__ float qs[DCKV_MAX_HEAD_DIM];
  for (int d = threadIdx.x; d < dh; d += kThreads) qs[d] = q[(int64_t(b) * tb.n_q_heads + h) * dh + d];
  __syncthreads();
  const int r = tb.rank_of_q[h];
  const T* base = Rk + tb.roff_of_q[h] + tb.rcol_of_q[h];
  const int stride = tb.rstride_of_q[h];
  float* dst = qt + int64_t(b) * tb.qlen + tb.qoff[h];
  for (int j = threadIdx.x; j < r; j += kThreads) {
    const T* row = base + int64_t(j) * stride;
    float acc = 0.f;
    for (int d = 0; d < dh; ++d) acc = fmaf(qs[d], to_f32(row[d]), acc);
    dst[j] = acc * scale;
  }
}

// ------------------------------------------------- split (portable VALU)
// One 256-thread block per (split, query head, query row): query row
// bq = b * Q + i is query i of sequence b, which sees the first
// T_b - Q + i + 1 cache positions (causal inside the chunk of Q).  Scores:
// 4 threads per token, each summing a quarter of the group's rank.  Values:
// each thread owns value columns tid, tid+256, ...
template <typename T>
__global__ __launch_bounds__(kThreads) void split_valu(
    const float* __restrict__ qt, const T* __restrict__ pool, int64_t num_pages,
    const int32_t* __restrict__ page_table, int max_pages, const int32_t* __restrict__ seq_lens,
    int max_context, int split_tokens, int n_split, int rv, int64_t page_elems,
    int64_t value_base, float* __restrict__ part_ml, float* __restrict__ part_acc, HeadTables tb) {
  const int split = blockIdx.x, h = blockIdx.y, bq = blockIdx.z;
  const int b = bq / tb.n_queries, qi = bq % tb.n_queries;
  const int tid = threadIdx.x;
  __shared__ float qs[DCKV_MAX_GROUP_RANK];
  __shared__ float part[4][DCKV_PAGE_TOKENS];
  __shared__ float ps[DCKV_PAGE_TOKENS];

  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int T_q = max(0, T_b - tb.n_queries + qi + 1);   // positions this query sees
  const int t0 = split * split_tokens;
  const int t1 = min(t0 + split_tokens, T_q);
  const int r = tb.rank_of_q[h];
  const int koff = tb.koff_of_q[h];
  for (int j = tid; j < r; j += kThreads) qs[j] = qt[int64_t(bq) * tb.qlen + tb.qoff[h] + j];
  __syncthreads();

  float acc[kAccPerThread];
#pragma unroll
  for (int i = 0; i < kAccPerThread; ++i) acc[i] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const int slot = tid & (DCKV_PAGE_TOKENS - 1), quarter = tid >> 6;

  for (int tok = t0; tok < t1; tok += DCKV_PAGE_TOKENS) {
    const int n = min(DCKV_PAGE_TOKENS, t1 - tok);
    const int page = page_table[int64_t(b) * max_pages + tok / DCKV_PAGE_TOKENS];
    const bool valid = page >= 0 && page < num_pages;
    const T* pg = pool + (valid ? int64_t(page) * page_elems : 0);
    float sp = 0.f;
    if (valid && slot < n) {
      // chunk-major keys: column c of this slot at (c/32)*2048 + slot*32 + c%32
      const T* kslot = pg + slot * 32;
      for (int k = quarter; k < r; k += 4) {
        const int c = koff + k;
        sp = fmaf(qs[k], to_f32(kslot[(c >> 5) * 2048 + (c & 31)]), sp);
      }
    }
    part[quarter][slot] = sp;
    __syncthreads();
    if (tid < DCKV_PAGE_TOKENS)
      ps[tid] = (valid && tid < n) ? (part[0][tid] + part[1][tid]) + (part[2][tid] + part[3][tid])
                                   : -INFINITY;
    __syncthreads();
    float cmax = -INFINITY;
    for (int t = 0; t < n; ++t) cmax = fmaxf(cmax, ps[t]);
    const float m_new = fmaxf(m_run, cmax);
    __syncthreads();
    if (m_new == -INFINITY) continue;  // uniform: no valid token so far
    const float alpha = exp2f(m_run - m_new);
    if (tid < DCKV_PAGE_TOKENS) ps[tid] = tid < n ? exp2f(ps[tid] - m_new) : 0.f;
    __syncthreads();
    float csum = 0.f;
    for (int t = 0; t < n; ++t) csum += ps[t];
    l_run = l_run * alpha + csum;
#pragma unroll
    for (int i = 0; i < kAccPerThread; ++i) {
      const int j = tid + i * kThreads;
      if (j < rv) {
        float a = acc[i] * alpha;
        if (valid) {
          // tile-major values: column j of slot t at (j/16)*1024 + (t/32)*512 + (j%16)*32 + t%32
          const T* vcol = pg + value_base + int64_t(j >> 4) * 1024 + (j & 15) * 32;
          for (int t = 0; t < n; ++t) a = fmaf(ps[t], to_f32(vcol[(t >> 5) * 512 + (t & 31)]), a);
        }
        acc[i] = a;
      }
    }
    m_run = m_new;
    __syncthreads();
  }

  const int64_t row = (int64_t(bq) * tb.n_q_heads + h) * n_split + split;
  if (tid == 0) {
    part_ml[row * 2 + 0] = m_run;
    part_ml[row * 2 + 1] = l_run;
  }
#pragma unroll
  for (int i = 0; i < kAccPerThread; ++i) {
    const int j = tid + i * kThreads;
    if (j < rv) part_acc[row * rv + j] = acc[i];
  }
}

// ------------------------------------------------------ merge + up-project
template <typename T>
__global__ __launch_bounds__(kThreads) void merge_upproject(
    const float* __restrict__ part_ml, const float* __restrict__ part_acc,
    const T* __restrict__ Rv, float* __restrict__ out, int n_split, int rv, HeadTables tb) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x;
  const int dh = tb.head_dim;
  const int n = tb.n_kv_heads * dh;
  const int kv = h / tb.q_per_kv;
  __shared__ float ash[DCKV_MAX_VALUE_RANK];
  const int64_t row0 = (int64_t(b) * tb.n_q_heads + h) * n_split;
  float M = -INFINITY;
  for (int s = 0; s < n_split; ++s) M = fmaxf(M, part_ml[(row0 + s) * 2]);
  float* o = out + (int64_t(b) * tb.n_q_heads + h) * dh;
  if (M == -INFINITY) {
    for (int d = tid; d < dh; d += kThreads) o[d] = 0.f;
    return;
  }
  float L = 0.f;
  for (int s = 0; s < n_split; ++s) L += exp2f(part_ml[(row0 + s) * 2] - M) * part_ml[(row0 + s) * 2 + 1];
  const float inv = 1.f / L;
  for (int j = tid; j < rv; j += kThreads) {
    float a = 0.f;
    for (int s = 0; s < n_split; ++s) {
      const float w = exp2f(part_ml[(row0 + s) * 2] - M);
      a = fmaf(w, part_acc[(row0 + s) * rv + j], a);
    }
    ash[j] = a * inv;
  }
  __syncthreads();
  for (int d = tid; d < dh; d += kThreads) {
    float acc = 0.f;
    const T* col = Rv + int64_t(kv) * dh + d;
    for (int j = 0; j < rv; ++j) acc = fmaf(ash[j], to_f32(col[int64_t(j) * n]), acc);
    o[d] = acc;
  }
}

template <typename T>
hipError_t launch_decode_t(const dckv_plan& p, const DecodeShape& sh, const float* q,
                           const void* pool, int64_t num_pages, const int32_t* page_table,
                           int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                           const void* R_value, float* out, void* workspace, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  float* qt = reinterpret_cast<float*>(ws + sh.off_qt);
  float* ml = reinterpret_cast<float*>(ws + sh.off_ml);
  float* acc = reinterpret_cast<float*>(ws + sh.off_acc);
  const float scale = kLog2e / std::sqrt(float(p.dh));
  const int rows = sh.batch * p.Q;               // query rows (sequence, query)
  hipLaunchKernelGGL(fold_kernel<T>, dim3(p.Hq, rows), dim3(kThreads), 0, stream, q,
                     static_cast<const T*>(R_keys), qt, p.tables, scale);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.prof_before && p.prof_after)   // events stamped by the kernel's own dispatch
    hipExtLaunchKernelGGL(split_valu<T>, dim3(sh.n_split, p.Hq, rows), dim3(kThreads), 0u,
                          stream, p.prof_before, p.prof_after, 0u, qt, static_cast<const T*>(pool),
                          num_pages, page_table, max_pages, seq_lens, sh.max_context,
                          sh.split_tokens, sh.n_split, p.rv, p.page_elems, p.value_base, ml, acc,
                          p.tables);
  else
    hipLaunchKernelGGL(split_valu<T>, dim3(sh.n_split, p.Hq, rows), dim3(kThreads), 0, stream,
                       qt, static_cast<const T*>(pool), num_pages, page_table, max_pages, seq_lens,
                       sh.max_context, sh.split_tokens, sh.n_split, p.rv, p.page_elems,
                       p.value_base, ml, acc, p.tables);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_upproject<T>, dim3(p.Hq, rows), dim3(kThreads), 0, stream, ml, acc,
                     static_cast<const T*>(R_value), out, sh.n_split, p.rv, p.tables);
  return hipGetLastError();
}

}  // namespace

// Two-pass shape.  Score work-groups of eight pages, so that ragged batches
// balance over the compute units.  Value work-groups (sequence, chunk, rank
// group): the tiles a group and the chunk count are chosen so that the
// work-groups fill whole rounds of the compute units, with fewer chunks
// (fewer partials) on ties; split_tokens / 64, when given, is the chunk
// length.  One row slice: waves take pages of the chunk, a group of 4, 6 or
// 8 tiles; the estimate is rounds x (pages a wave x (tiles + head tiles, the
// weight loads counted at half a tile each) + a fixed cost of 4).  Several
// slices: the eight waves walk the chunk's pages together, 2 or 1 tiles a
// wave (1 only beyond 8 row tiles); the estimate, in sixteenths of a page
// of one tile a wave, is rounds x (pages x (16 tiles + 8 + row tiles) + 64):
// a page's weights staged and a barrier cost about half a tile, each row
// tile a sixteenth more.
static DecodeShape pass_shape(const dckv_plan& p, int32_t batch, int32_t max_context) {
  DecodeShape s{};
  s.batch = batch;
  s.max_context = max_context;
  s.pass = true;
  const int64_t npm = std::max<int64_t>(1, (int64_t(max_context) + DCKV_PAGE_TOKENS - 1) / DCKV_PAGE_TOKENS);
  s.npm = int32_t(npm);
  s.unit_pages = kUnitPages;
  s.units_per_seq = int32_t((npm + s.unit_pages - 1) / s.unit_pages);
  const int64_t cap = pass_max_chunk_pages(p);
  const int64_t B = std::max<int32_t>(batch, 1);
  const int32_t RT = p.pass.n_slices * p.pass.nt;
  const bool shared = p.pass.n_slices > 1;
  std::vector<int32_t> options;
  if (!shared) options = {8, 6, 4};
  else if (RT <= 8) options = {2, 1};
  else options = {1};
  int64_t best_cost = -1;
  for (int32_t rgt : options) {
    const int64_t tiles = shared ? int64_t(kSharedWaves) * rgt : rgt;   // value tiles a work-group
    const int64_t nrg = (p.pass.mt_v + tiles - 1) / tiles;
    auto consider = [&](int64_t cp) {
      const int64_t nc = (npm + cp - 1) / cp;
      const int64_t rounds = (B * nc * nrg + kTargetWorkgroups - 1) / kTargetWorkgroups;
      const int64_t cost = shared ? rounds * (cp * (16 * rgt + 8 + RT) + 64)
                                  : rounds * ((cp + 7) / 8 * (rgt + p.pass.nt) + 4);
      if (best_cost < 0 || cost < best_cost || (cost == best_cost && nc < s.n_chunks)) {
        best_cost = cost;
        s.rgt = rgt;
        s.n_rgroups = int32_t(nrg);
        s.chunk_pages = int32_t(cp);
        s.n_chunks = int32_t(nc);
      }
    };
    if (p.split_tokens > 0) {
      consider(std::min<int64_t>(cap, std::max<int64_t>(1, p.split_tokens / DCKV_PAGE_TOKENS)));
    } else {
      // from the fewest chunks the cap allows to about two work-groups a
      // compute unit (at least the first candidate)
      const int64_t lo = (npm + cap - 1) / cap;
      const int64_t hi = std::min(npm, std::max(lo, std::max<int64_t>(1, 2 * kTargetWorkgroups / (B * nrg)) + 1));
      for (int64_t nc = lo; nc <= hi; ++nc) consider((npm + nc - 1) / nc);
    }
  }
  s.split_tokens = s.chunk_pages * DCKV_PAGE_TOKENS;
  s.n_split = s.n_chunks;
  const size_t ns = 16 * size_t(RT);          // row slots
  s.off_qt = 0;
  s.off_p = align_up(size_t(batch) * p.pass.n_slices * p.pass.max_pairs * 2048, 256);
  s.off_ml = s.off_p + align_up(size_t(batch) * npm * RT * 2560, 256);   // weights and records
  const size_t rows = size_t(batch) * s.n_chunks;
  s.off_acc = s.off_ml + align_up(rows * 2 * ns * sizeof(float), 256);
  s.off_opart = s.off_acc + align_up(rows * ns * size_t(p.rv) * sizeof(float), 256);
  s.bytes = s.off_opart + align_up(size_t(batch) * p.Q * p.Hq * p.rv * sizeof(float), 256);
  return s;
}

DecodeShape decode_shape(const dckv_plan& p, int32_t batch, int32_t max_context) {
  // The two-pass kernels when asked for, when the single-pass kernel does not
  // apply, or when it would cut the rows into several slices (a value rank
  // beyond what one slice's accumulators hold), each slice reading the whole
  // value part again, and the batch holds enough pages to give every wave of
  // the chip one.  Otherwise the single-pass kernel: measured on the one-query
  // layers it is as fast or faster, the two passes each paying a work-group
  // prologue and a tail.
  if (p.pass_ok) {
    const int64_t npm = (int64_t(max_context) + DCKV_PAGE_TOKENS - 1) / DCKV_PAGE_TOKENS;
    const bool many_pages = int64_t(batch) * npm >= int64_t(8) * kTargetWorkgroups;
    if (p.decode_passes == 2 || !p.mfma_ok || (many_pages && p.mfma.n_slices > 1))
      return pass_shape(p, batch, max_context);
  }
  DecodeShape s{};
  s.batch = batch;
  s.max_context = max_context;
  s.mfma = p.mfma_ok;
  int64_t L = p.split_tokens;
  if (L == 0) {
    if (s.mfma) {
      // about one work-group per compute unit over the whole batch, at most
      // the split kernel's page-list capacity
      const int64_t tokens = int64_t(batch) * max_context * p.mfma.n_slices;
      L = (tokens + kTargetWorkgroups - 1) / kTargetWorkgroups;
      L = std::max<int64_t>(DCKV_PAGE_TOKENS, (L + DCKV_PAGE_TOKENS - 1) / DCKV_PAGE_TOKENS * DCKV_PAGE_TOKENS);
      L = std::min<int64_t>(L, mfma_max_split_tokens());
    } else {
      L = kValuSplitTokens;
    }
  }
  if (s.mfma && L > mfma_max_split_tokens()) s.mfma = false;   // an explicit split beyond the cap
  s.split_tokens = int32_t(L);
  s.n_split = max_context > 0 ? int32_t((max_context + L - 1) / L) : 1;
  s.off_qt = 0;
  s.off_ml = align_up(size_t(batch) * p.Q * p.qlen * sizeof(float), 256);
  if (s.mfma)   // the MFMA path keeps hi/lo query blocks of 2 KB per (sequence, slice, chunk)
    s.off_ml = align_up(size_t(batch) * p.mfma.n_slices * p.mfma.max_pairs * 2048, 256);
  if (s.mfma) {
    const int64_t units = int64_t(batch) * s.n_split;
    s.n_units = int32_t((units + 7) / 8 * 8);
    s.merge_ranks = mfma_merge_ranks(p, batch);
    s.n_rchunks = (p.rv + s.merge_ranks - 1) / s.merge_ranks;
    const size_t nh = 16 * size_t(p.mfma.nt);
    const size_t rows = size_t(batch) * p.mfma.n_slices * s.n_split;
    s.off_acc = s.off_ml + align_up(rows * 2 * nh * sizeof(float), 256);
    s.off_opart = s.off_acc + align_up(rows * nh * size_t(p.rv) * sizeof(float), 256);
    s.bytes = s.off_opart + align_up(size_t(batch) * p.Q * p.Hq * p.rv * sizeof(float), 256);
  } else {
    const size_t rows = size_t(batch) * p.Q * p.Hq * s.n_split;
    s.off_acc = s.off_ml + align_up(rows * 2 * sizeof(float), 256);
    s.off_opart = s.off_acc + align_up(rows * p.rv * sizeof(float), 256);
    s.bytes = s.off_opart;
  }
  return s;
}

hipError_t launch_decode(const dckv_plan& p, const DecodeShape& shape, const float* q,
                         const void* pool, int64_t num_pages, const int32_t* page_table,
                         int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                         const void* R_value, float* out, void* workspace, hipStream_t stream) {
  if (shape.pass)
    return launch_decode_pass(p, shape, q, pool, num_pages, page_table, max_pages, seq_lens, R_keys,
                              R_value, out, workspace, stream);
  if (shape.mfma)
    return launch_decode_mfma(p, shape, q, pool, num_pages, page_table, max_pages, seq_lens, R_keys,
                              R_value, out, workspace, stream);
  if (p.dtype == DCKV_F32)
    return launch_decode_t<float>(p, shape, q, pool, num_pages, page_table, max_pages, seq_lens,
                                  R_keys, R_value, out, workspace, stream);
  return launch_decode_t<bf16>(p, shape, q, pool, num_pages, page_table, max_pages, seq_lens, R_keys,
                               R_value, out, workspace, stream);
}

}  // namespace dckv
