// Uncompressed KV decode: the baseline the compressed cache is measured
// against (same harness, same head map, scale 1/sqrt(d_h), no mask).
// Paged cache: pages of 64 tokens; keys [H_kv][64][d_h] then values
// [H_kv][64][d_h], bf16, so one head's keys (or values) of a page are one
// contiguous run of 64 * d_h elements.
//
//   split  one 256-thread work-group per (context split, KV head, sequence):
//          scores of the head's qpk query heads over the page's 64 tokens
//          (4 lanes a token, a quarter of d_h each, summed by shuffles), a
//          base-2 online softmax (one wave a query head, its new maximum,
//          rescale factor and page sum published through LDS), then
//          o += p V with each lane owning 8 columns of d_h for its token
//          group.  The next page's keys and values are loaded while the
//          current page is processed.  Writes unnormalised o and (m, l).
//   merge  fixed ascending-split log-sum-exp merge.
#include <algorithm>
#include <cmath>

#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

constexpr int kDenseThreads = 256;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ float wave_max64(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum64(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// DH = d_h (64, 128 or 256); QP >= qpk query heads a KV head (1, 2, 4 or 8).
template <int DH, int QP>
__global__ __launch_bounds__(kDenseThreads) void dense_split(
    const float* __restrict__ q, const bf16* __restrict__ pool, int64_t num_pages,
    const int32_t* __restrict__ page_table, int max_pages, const int32_t* __restrict__ seq_lens,
    int max_context, int split_tokens, int n_split, int n_q_heads, int n_kv_heads, float scale,
    float* __restrict__ part_o, float* __restrict__ part_ml) {
  constexpr int KQ = DH / 4;                 // key columns a lane (a quarter of d_h)
  constexpr int NK = KQ / 8;                 // 16-byte key loads a lane a page
  constexpr int DG = DH / 8;                 // 8-column value groups
  constexpr int NTG = kDenseThreads / DG;    // token groups
  constexpr int NV = 64 / NTG;               // tokens a lane a page
  const int split = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int qpk = n_q_heads / n_kv_heads;
  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int t0 = split * split_tokens;
  const int t1 = min(t0 + split_tokens, T_b);
  if (t0 >= t1) return;                      // the merge reads only splits holding tokens

  __shared__ float qs[QP][DH];               // scaled queries of this KV head
  __shared__ float sp[QP][64];               // scores, then probabilities, of a page
  __shared__ float stat[QP][3];              // rescale factor, page sum, new maximum
  __shared__ float red[4][QP][DH];           // per-wave partial outputs
  for (int i = tid; i < QP * DH; i += kDenseThreads) {
    const int j = i / DH, d = i % DH;
    qs[j][d] = j < qpk ? q[(int64_t(b) * n_q_heads + kv * qpk + j) * DH + d] * scale : 0.f;
  }

  const int tok = tid >> 2, quarter = tid & 3;          // score role
  const int dg = tid % DG, tg = tid / DG;                // value role
  const int64_t page_elems = int64_t(2) * 64 * n_kv_heads * DH;
  const int64_t vbase = int64_t(64) * n_kv_heads * DH;
  const int64_t head_off = int64_t(kv) * 64 * DH;

  float acc[QP][8];
  float m_run[QP], l_run[QP];
#pragma unroll
  for (int j = 0; j < QP; ++j) {
    m_run[j] = -INFINITY;
    l_run[j] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = 0.f;
  }

  const int npages = (t1 - t0 + 63) / 64;
  u32x4_t kr[NK], vr[NV];
  auto load_page = [&](int pi, u32x4_t (&kk)[NK], u32x4_t (&vv)[NV]) {
    const int pos = t0 + 64 * pi;
    int pg = page_table[int64_t(b) * max_pages + pos / 64];
    pg = (pg >= 0 && pg < num_pages) ? pg : 0;           // invalid pages are masked below
    const bf16* base = pool + int64_t(pg) * page_elems + head_off;
#pragma unroll
    for (int i = 0; i < NK; ++i)
      kk[i] = *reinterpret_cast<const u32x4_t*>(base + tok * DH + quarter * KQ + 8 * i);
#pragma unroll
    for (int i = 0; i < NV; ++i)
      vv[i] = *reinterpret_cast<const u32x4_t*>(base + vbase + (tg + NTG * i) * DH + 8 * dg);
  };
  load_page(0, kr, vr);
  __syncthreads();                           // qs ready

  for (int pi = 0; pi < npages; ++pi) {
    const int pos = t0 + 64 * pi;
    const int n = min(64, t1 - pos);
    const int pgid = page_table[int64_t(b) * max_pages + pos / 64];
    const bool valid = pgid >= 0 && pgid < num_pages;
    u32x4_t kc[NK], vc[NV];
#pragma unroll
    for (int i = 0; i < NK; ++i) kc[i] = kr[i];
#pragma unroll
    for (int i = 0; i < NV; ++i) vc[i] = vr[i];
    if (pi + 1 < npages) load_page(pi + 1, kr, vr);      // next page in flight

    // ---- scores of this lane's token over its quarter of d_h
#pragma unroll
    for (int j = 0; j < QP; ++j) {
      if (j < qpk) {
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < NK; ++i) {
          const float* qq = &qs[j][quarter * KQ + 8 * i];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s = fmaf(qq[2 * e], bf_lo(kc[i][e]), s);
            s = fmaf(qq[2 * e + 1], bf_hi(kc[i][e]), s);
          }
        }
        s += __shfl_xor(s, 1);
        s += __shfl_xor(s, 2);
        if (quarter == 0) sp[j][tok] = (valid && tok < n) ? s : -INFINITY;
      }
    }
    __syncthreads();

    // ---- online softmax: wave w serves query heads w and w + 4
#pragma unroll
    for (int jj = 0; jj < (QP + 3) / 4; ++jj) {
      const int j = w + 4 * jj;
      if (j < qpk) {
        float m_prev = -INFINITY;
#pragma unroll
        for (int k = 0; k < QP; ++k)
          if (k == j) m_prev = m_run[k];   // compile-time register index
        const float s = sp[j][lane];
        const float m_new = fmaxf(m_prev, wave_max64(s));
        const float p = (s == -INFINITY) ? 0.f : exp2f(s - m_new);
        sp[j][lane] = p;
        const float psum = wave_sum64(p);
        if (lane == 0) {
          stat[j][0] = (m_new == -INFINITY) ? 1.f : exp2f(m_prev - m_new);
          stat[j][1] = psum;
          stat[j][2] = m_new;
        }
      }
    }
    __syncthreads();

    // ---- running state and o += p V (every lane keeps the same m, l)
#pragma unroll
    for (int j = 0; j < QP; ++j) {
      if (j < qpk) {
        const float alpha = stat[j][0];
        l_run[j] = l_run[j] * alpha + stat[j][1];
        m_run[j] = stat[j][2];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[j][e] *= alpha;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          const float p = sp[j][tg + NTG * i];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[j][2 * e] = fmaf(p, bf_lo(vc[i][e]), acc[j][2 * e]);
            acc[j][2 * e + 1] = fmaf(p, bf_hi(vc[i][e]), acc[j][2 * e + 1]);
          }
        }
      }
    }
    __syncthreads();                         // sp and stat are rewritten next page
  }

  // ---- token groups: the wave's groups by a fixed shuffle butterfly (lanes
  // that differ in the bits above the value group), then the 4 waves in order
#pragma unroll
  for (int j = 0; j < QP; ++j) {
    if (j < qpk) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x = acc[j][e];
#pragma unroll
        for (int o = DG; o < 64; o <<= 1) x += __shfl_xor(x, o);
        acc[j][e] = x;
      }
    }
  }
  if (lane < DG) {
#pragma unroll
    for (int j = 0; j < QP; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) red[w][j][8 * lane + e] = acc[j][e];
  }
  __syncthreads();
  const int64_t row0 = (int64_t(b) * n_split + split) * n_q_heads + kv * qpk;
  for (int i = tid; i < qpk * DH; i += kDenseThreads) {
    const int j = i / DH, d = i % DH;
    part_o[(row0 + j) * DH + d] = ((red[0][j][d] + red[1][j][d]) + red[2][j][d]) + red[3][j][d];
  }
  if (tid == 0) {
#pragma unroll
    for (int j = 0; j < QP; ++j)
      if (j < qpk) {
        part_ml[(row0 + j) * 2 + 0] = m_run[j];
        part_ml[(row0 + j) * 2 + 1] = l_run[j];
      }
  }
}

// One block of d_h threads per (query head, sequence): fixed ascending-split merge.
__global__ __launch_bounds__(256) void dense_merge(const float* __restrict__ part_o,
                                                   const float* __restrict__ part_ml,
                                                   const int32_t* __restrict__ seq_lens,
                                                   int max_context, int split_tokens, int n_split,
                                                   int n_q_heads, int dh, float* __restrict__ out) {
  const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  int T_b = seq_lens[b];
  T_b = T_b < 0 ? 0 : (T_b > max_context ? max_context : T_b);
  const int ns = (T_b + split_tokens - 1) / split_tokens;
  const int64_t r0 = int64_t(b) * n_split * n_q_heads + h;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, part_ml[(r0 + int64_t(s) * n_q_heads) * 2]);
  float L = 0.f, o = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < ns; ++s) {
      const int64_t r = r0 + int64_t(s) * n_q_heads;
      const float wgt = exp2f(part_ml[r * 2] - M);
      L = fmaf(wgt, part_ml[r * 2 + 1], L);
      if (d < dh) o = fmaf(wgt, part_o[r * dh + d], o);
    }
  }
  if (d < dh) out[(int64_t(b) * n_q_heads + h) * dh + d] = (M == -INFINITY || L <= 0.f) ? 0.f : o / L;
}

template <int DH, int QP>
hipError_t launch_dense_t(const DenseShape& sh, const float* q, const void* pool,
                          int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                          const int32_t* seq_lens, float* part_o, float* part_ml,
                          hipEvent_t before, hipEvent_t after, hipStream_t stream) {
  const float scale = kLog2e / std::sqrt(float(DH));
  const dim3 grid(sh.n_split, sh.n_kv_heads, sh.batch);
  auto kern = dense_split<DH, QP>;
  if (before && after)
    hipExtLaunchKernelGGL(kern, grid, dim3(kDenseThreads), 0u, stream, before, after,
                          0u, q, static_cast<const bf16*>(pool), num_pages, page_table, max_pages,
                          seq_lens, sh.max_context, sh.split_tokens, sh.n_split, sh.n_q_heads,
                          sh.n_kv_heads, scale, part_o, part_ml);
  else
    hipLaunchKernelGGL(kern, grid, dim3(kDenseThreads), 0, stream, q,
                       static_cast<const bf16*>(pool), num_pages, page_table, max_pages, seq_lens,
                       sh.max_context, sh.split_tokens, sh.n_split, sh.n_q_heads, sh.n_kv_heads,
                       scale, part_o, part_ml);
  return hipGetLastError();
}

template <int DH>
hipError_t launch_dense_d(const DenseShape& sh, const float* q, const void* pool,
                          int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                          const int32_t* seq_lens, float* part_o, float* part_ml,
                          hipEvent_t before, hipEvent_t after, hipStream_t stream) {
  const int qpk = sh.n_q_heads / sh.n_kv_heads;
#define DCKV_DENSE(QPV)                                                                       \
  return launch_dense_t<DH, QPV>(sh, q, pool, num_pages, page_table, max_pages, seq_lens, \
                                 part_o, part_ml, before, after, stream)
  if (qpk <= 1) DCKV_DENSE(1);
  if (qpk <= 2) DCKV_DENSE(2);
  if (qpk <= 4) DCKV_DENSE(4);
  DCKV_DENSE(8);
#undef DCKV_DENSE
}

size_t align_up_d(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

DenseShape dense_shape(int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int32_t batch,
                       int32_t max_context, int32_t split_tokens) {
  DenseShape s{};
  s.n_q_heads = n_q_heads;
  s.n_kv_heads = n_kv_heads;
  s.head_dim = head_dim;
  s.batch = batch;
  s.max_context = max_context;
  int64_t L = split_tokens;
  if (L == 0) {   // about four work-groups a compute unit over (splits, KV heads, batch)
    const int64_t work = int64_t(batch) * max_context * n_kv_heads;
    L = (work + 1023) / 1024;
    L = std::max<int64_t>(64, (L + 63) / 64 * 64);
  }
  s.split_tokens = int32_t(L);
  s.n_split = max_context > 0 ? int32_t((max_context + L - 1) / L) : 1;
  const size_t rows = size_t(batch) * s.n_split * n_q_heads;
  s.off_o = 0;
  s.off_ml = align_up_d(rows * head_dim * sizeof(float), 256);
  s.bytes = s.off_ml + align_up_d(rows * 2 * sizeof(float), 256);
  return s;
}

hipError_t launch_dense_decode(const DenseShape& sh, const float* q, const void* pool,
                               int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                               const int32_t* seq_lens, float* out, void* workspace,
                               hipEvent_t before, hipEvent_t after, hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  float* part_o = reinterpret_cast<float*>(ws + sh.off_o);
  float* part_ml = reinterpret_cast<float*>(ws + sh.off_ml);
  hipError_t e;
  switch (sh.head_dim) {
    case 64:
      e = launch_dense_d<64>(sh, q, pool, num_pages, page_table, max_pages, seq_lens, part_o,
                             part_ml, before, after, stream);
      break;
    case 128:
      e = launch_dense_d<128>(sh, q, pool, num_pages, page_table, max_pages, seq_lens, part_o,
                              part_ml, before, after, stream);
      break;
    case 256:
      e = launch_dense_d<256>(sh, q, pool, num_pages, page_table, max_pages, seq_lens, part_o,
                              part_ml, before, after, stream);
      break;
    default:
      return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(dense_merge, dim3(sh.n_q_heads, sh.batch), dim3(std::max(64, int(sh.head_dim))),
                     0, stream, part_o, part_ml, seq_lens, sh.max_context, sh.split_tokens,
                     sh.n_split, sh.n_q_heads, int(sh.head_dim), out);
  return hipGetLastError();
}

}  // namespace dckv
