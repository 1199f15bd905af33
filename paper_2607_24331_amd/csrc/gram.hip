// Offline contractions of the compression pipeline.
//
// gram: G = A~^T A~ for A [rows, cols] (row-major, one sample a row), with
// A~ = A - 1 mu^T (column means) when centring is asked for.  It feeds the
// CKA head similarity (Sec. III-A: CKA compares centred representations;
// Sec. III-C: S[i][j] between the heads' activations) and the calibration
// Gram X^T X of the value refinement (Sec. III-D).  fp32 throughout: the
// products run on v_mfma_f32_16x16x4_f32 with fp32 inputs and accumulators.
//
// head_similarity: S[i][j] = ||G_ij||_F^2 / (||G_ii||_F ||G_jj||_F) over the
// d_h x d_h blocks of a centred Gram, which is linear CKA (Sec. III-A).
#include <cmath>

#include "device.h"
#include "internal.h"

namespace dckv {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kGK = 32;                   // samples a staging step
constexpr int kMeanRows = 256;            // rows a column-sum work-group

// Column sums of rows [rb*kMeanRows, ...) for 256 columns a work-group.
template <typename T>
__global__ __launch_bounds__(256) void colsum_partial(const T* __restrict__ A, int64_t rows,
                                                      int cols, float* __restrict__ part) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int64_t r0 = int64_t(blockIdx.y) * kMeanRows;
  const int64_t r1 = rows < r0 + kMeanRows ? rows : r0 + kMeanRows;
  if (c >= cols) return;
  float s = 0.f;
  int64_t r = r0;
  for (; r + 8 <= r1; r += 8) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = to_f32(A[(r + k) * cols + c]);
#pragma unroll
    for (int k = 0; k < 8; ++k) s += v[k];
  }
  for (; r < r1; ++r) s += to_f32(A[r * cols + c]);
  part[int64_t(blockIdx.y) * cols + c] = s;
}

// mu[c] = (sum of the partial sums in row-block order) / rows.
__global__ __launch_bounds__(256) void colmean_finish(const float* __restrict__ part, int nblk,
                                                      int64_t rows, int cols,
                                                      float* __restrict__ mu) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  float s = 0.f;
  for (int b = 0; b < nblk; ++b) s += part[int64_t(b) * cols + c];
  mu[c] = s / float(rows);
}

// Staging of 8 consecutive columns of one sample: raw 16-byte loads first
// (consumed a staging step later, so they stay in flight during the
// products), then conversion to fp32, centring and masking outside A.
struct Raw8 {
  uint4 q[2];
};

template <typename T>
__device__ __forceinline__ Raw8 load_raw(const T* __restrict__ A, int64_t rows, int cols,
                                         int64_t r, int c) {
  Raw8 x;
  const int64_t rr = r < rows ? r : rows - 1;          // clamped: every load is in bounds
  const int cc = c < cols ? c : 0;
  const uint4* p = reinterpret_cast<const uint4*>(A + rr * cols + cc);
  x.q[0] = p[0];
  x.q[1] = sizeof(T) == 4 ? p[1] : uint4{0u, 0u, 0u, 0u};
  return x;
}

template <typename T>
__device__ __forceinline__ void finish8(const Raw8& x, int64_t rows, int cols, int64_t r, int c,
                                        const float* mu8, float (&v)[8]) {
  if constexpr (sizeof(T) == 4) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      v[4 * k + 0] = __uint_as_float(x.q[k].x);
      v[4 * k + 1] = __uint_as_float(x.q[k].y);
      v[4 * k + 2] = __uint_as_float(x.q[k].z);
      v[4 * k + 3] = __uint_as_float(x.q[k].w);
    }
  } else {
    const uint32_t w[4] = {x.q[0].x, x.q[0].y, x.q[0].z, x.q[0].w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = __uint_as_float(w[j] << 16);
      v[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = (r < rows && c + k < cols) ? v[k] - mu8[k] : 0.f;
}

// One TS x TS tile (ti <= tj) of G per work-group of WR x WC waves, each
// wave a (TS/WR) x (TS/WC) block of 16 x 16 products.  Staging: kGK
// samples x TS columns of the tile's row block and column block in LDS
// (double-buffered; row stride TS + 16 floats, which keeps the operand
// reads free of bank conflicts), in 8-column chunks, the next step's loads
// in flight during the current step's products.  Products: lane l feeds
// A[i = l % 16][k = l / 16] and B[k = l / 16][j = l % 16]; the accumulator
// holds D[4 (l / 16) + v][l % 16].  An off-diagonal tile is written twice:
// as is, and transposed through LDS into the mirror tile.
template <typename T, int TS, int WR, int WC>
__global__ __launch_bounds__(WR * WC * 64) void gram_tiles(const T* __restrict__ A, int64_t rows,
                                                           int cols, const float* __restrict__ mu,
                                                           float* __restrict__ G, int n_tiles) {
  constexpr int NT = WR * WC * 64;                     // threads
  constexpr int PAD = TS + 16;
  constexpr int RW = TS / WR, CW = TS / WC;            // wave block
  constexpr int MX = RW / 16, MY = CW / 16;
  constexpr int CHUNKS = kGK * TS / 8;                 // 8-column chunks a slab
  constexpr int CPT = (CHUNKS + NT - 1) / NT;          // chunks a thread
  static_assert(RW % 16 == 0 && CW % 16 == 0, "wave blocks of whole 16 x 16 products");
  extern __shared__ __align__(16) float smem[];        // [2][2][kGK][PAD]
  int lin = blockIdx.x, ti = 0;
  while (lin >= n_tiles - ti) {
    lin -= n_tiles - ti;
    ++ti;
  }
  const int tj = ti + lin;
  const bool diag = ti == tj;
  const int i0 = ti * TS, j0 = tj * TS;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wi = w / WC, wj = w % WC;
  int crow[CPT], ccol[CPT];
  float muI[CPT][8], muJ[CPT][8];
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    const int c = tid + q * NT;
    crow[q] = c < CHUNKS ? c / (TS / 8) : kGK;         // kGK: no chunk for this thread
    ccol[q] = (c % (TS / 8)) * 8;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int ci = i0 + ccol[q] + k, cj = j0 + ccol[q] + k;
      muI[q][k] = (mu && ci < cols) ? mu[ci] : 0.f;
      muJ[q][k] = (mu && cj < cols) ? mu[cj] : 0.f;
    }
  }
  floatx4 acc[MX][MY];
#pragma unroll
  for (int x = 0; x < MX; ++x)
#pragma unroll
    for (int y = 0; y < MY; ++y) acc[x][y] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nsteps = int((rows + kGK - 1) / kGK);
  Raw8 rI[CPT], rJ[CPT];
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    rI[q] = load_raw<T>(A, rows, cols, crow[q], i0 + ccol[q]);
    rJ[q] = diag ? rI[q] : load_raw<T>(A, rows, cols, crow[q], j0 + ccol[q]);
  }
  for (int st = 0; st < nsteps; ++st) {
    float* sI = smem + (st & 1) * 2 * kGK * PAD;
    float* sJ = diag ? sI : sI + kGK * PAD;
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
      if (crow[q] >= kGK) continue;
      const int64_t r = int64_t(st) * kGK + crow[q];
      float v[8];
      finish8<T>(rI[q], rows, cols, r, i0 + ccol[q], muI[q], v);
      *reinterpret_cast<float4*>(sI + crow[q] * PAD + ccol[q]) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<float4*>(sI + crow[q] * PAD + ccol[q] + 4) = make_float4(v[4], v[5], v[6], v[7]);
      if (!diag) {
        finish8<T>(rJ[q], rows, cols, r, j0 + ccol[q], muJ[q], v);
        *reinterpret_cast<float4*>(sJ + crow[q] * PAD + ccol[q]) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4*>(sJ + crow[q] * PAD + ccol[q] + 4) = make_float4(v[4], v[5], v[6], v[7]);
      }
    }
    __syncthreads();
    if (st + 1 < nsteps) {                      // next step's raw loads, consumed after the products
#pragma unroll
      for (int q = 0; q < CPT; ++q) {
        const int64_t r = int64_t(st + 1) * kGK + crow[q];
        rI[q] = load_raw<T>(A, rows, cols, r, i0 + ccol[q]);
        if (!diag) rJ[q] = load_raw<T>(A, rows, cols, r, j0 + ccol[q]);
      }
    }
    // every operand of the step is read first, so the LDS latency is paid
    // once a step rather than once a k-step
    float a[kGK / 4][MX], b[kGK / 4][MY];
#pragma unroll
    for (int s = 0; s < kGK / 4; ++s) {
      const int kr = 4 * s + (lane >> 4);
#pragma unroll
      for (int x = 0; x < MX; ++x) a[s][x] = sI[kr * PAD + RW * wi + 16 * x + (lane & 15)];
#pragma unroll
      for (int y = 0; y < MY; ++y) b[s][y] = sJ[kr * PAD + CW * wj + 16 * y + (lane & 15)];
    }
    __builtin_amdgcn_sched_barrier(0);          // keep the reads ahead of the products
#pragma unroll
    for (int s = 0; s < kGK / 4; ++s)
#pragma unroll
      for (int x = 0; x < MX; ++x)
#pragma unroll
        for (int y = 0; y < MY; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s][x], b[s][y], acc[x][y], 0, 0, 0);
  }

  // the tile as is
#pragma unroll
  for (int x = 0; x < MX; ++x)
#pragma unroll
    for (int y = 0; y < MY; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = i0 + RW * wi + 16 * x + 4 * (lane >> 4) + v;
        const int j = j0 + CW * wj + 16 * y + (lane & 15);
        if (i < cols && j < cols) G[int64_t(i) * cols + j] = acc[x][y][v];
      }
  if (diag) return;
  // the mirror tile: waves transpose their blocks through LDS, as many at a
  // time as the staging memory holds
  constexpr int TWS = CW * (RW + 1);                   // floats a wave's transposed block
  constexpr int WAVES_AT_ONCE = (2 * 2 * kGK * PAD) / TWS;
  static_assert(WAVES_AT_ONCE >= 1, "staging memory holds one transposed block");
  for (int w0 = 0; w0 < WR * WC; w0 += WAVES_AT_ONCE) {
    __syncthreads();                                    // staging / previous round no longer read
    if (w >= w0 && w < w0 + WAVES_AT_ONCE) {
      float* tw = smem + (w - w0) * TWS;
#pragma unroll
      for (int x = 0; x < MX; ++x)
#pragma unroll
        for (int y = 0; y < MY; ++y)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            tw[(16 * y + (lane & 15)) * (RW + 1) + 16 * x + 4 * (lane >> 4) + v] = acc[x][y][v];
    }
    __syncthreads();
    if (w >= w0 && w < w0 + WAVES_AT_ONCE) {
      const float* tw = smem + (w - w0) * TWS;
      for (int rr = 0; rr < CW; ++rr)
        for (int cc = lane; cc < RW; cc += 64) {
          const int j = j0 + CW * wj + rr, i = i0 + RW * wi + cc;
          if (j < cols && i < cols) G[int64_t(j) * cols + i] = tw[rr * (RW + 1) + cc];
        }
    }
  }
}

// F[i][j] = ||G_ij||_F^2, one work-group a block, fixed-order sums; F is
// written into S's memory and turned into S by head_sim_finish.  Both
// (i, j) and (j, i) sum the block above the diagonal in the same order, so
// F, and with it S, is exactly symmetric as linear CKA is.
__global__ __launch_bounds__(256) void head_sim_blocks(const float* __restrict__ G, int h, int d,
                                                       float* __restrict__ F) {
  const int bx = blockIdx.x, by = blockIdx.y;
  const int i = min(bx, by), j = max(bx, by);
  const int n = h * d, tid = threadIdx.x;
  __shared__ float red[256];
  float f = 0.f;
  for (int e = tid; e < d * d; e += 256) {
    const float g = G[int64_t(i * d + e / d) * n + j * d + e % d];
    f = fmaf(g, g, f);
  }
  red[tid] = f;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) red[tid] += red[tid + s];
    __syncthreads();
  }
  if (tid == 0) F[bx * h + by] = red[0];
}

// S[i][j] = F[i][j] / (sqrt(F[i][i]) sqrt(F[j][j])) in place: one work-group
// reads every F it needs before any thread writes.
__global__ __launch_bounds__(1024) void head_sim_finish(float* __restrict__ S, int h) {
  const int tid = threadIdx.x, nn = h * h;
  float v[4], di[4], dj[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e = tid + 1024 * k;
    v[k] = di[k] = dj[k] = 0.f;
    if (e < nn) {
      v[k] = S[e];
      di[k] = S[(e / h) * h + e / h];
      dj[k] = S[(e % h) * h + e % h];
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e = tid + 1024 * k;
    if (e < nn) {
      const float den = sqrtf(di[k]) * sqrtf(dj[k]);
      S[e] = den > 0.f ? v[k] / den : 0.f;
    }
  }
}

constexpr int kComputeUnits = 256;        // MI355X

template <int TS, int WR, int WC>
hipError_t launch_tiles(const void* A, int32_t dtype, int64_t rows, int32_t cols, const float* mu,
                        float* G, int nt, hipStream_t stream) {
  const size_t lds = size_t(2) * 2 * kGK * (TS + 16) * sizeof(float);
  const dim3 grid(unsigned(int64_t(nt) * (nt + 1) / 2)), block(WR * WC * 64);
  hipError_t e;
  if (dtype == DCKV_BF16) {
    auto k = gram_tiles<bf16, TS, WR, WC>;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, int(lds))) != hipSuccess)
      return e;
    hipLaunchKernelGGL(k, grid, block, lds, stream, static_cast<const bf16*>(A), rows, cols, mu, G, nt);
  } else {
    auto k = gram_tiles<float, TS, WR, WC>;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, int(lds))) != hipSuccess)
      return e;
    hipLaunchKernelGGL(k, grid, block, lds, stream, static_cast<const float*>(A), rows, cols, mu, G, nt);
  }
  return hipGetLastError();
}

}  // namespace

size_t gram_workspace_bytes(int64_t rows, int32_t cols) {
  const int64_t nblk = (rows + kMeanRows - 1) / kMeanRows;
  return size_t((nblk + 1) * cols) * sizeof(float);
}

hipError_t launch_gram(const void* A, int32_t dtype, int64_t rows, int32_t cols, bool center,
                       float* G, void* workspace, hipStream_t stream) {
  const float* mu = nullptr;
  if (center) {
    float* part = static_cast<float*>(workspace);
    const int nblk = int((rows + kMeanRows - 1) / kMeanRows);
    float* m = part + int64_t(nblk) * cols;
    const dim3 g1((cols + 255) / 256, nblk);
    if (dtype == DCKV_BF16)
      hipLaunchKernelGGL(colsum_partial<bf16>, g1, dim3(256), 0, stream,
                         static_cast<const bf16*>(A), rows, cols, part);
    else
      hipLaunchKernelGGL(colsum_partial<float>, g1, dim3(256), 0, stream,
                         static_cast<const float*>(A), rows, cols, part);
    hipLaunchKernelGGL(colmean_finish, dim3((cols + 255) / 256), dim3(256), 0, stream, part, nblk,
                       rows, cols, m);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    mu = m;
  }
  // Tile size: the whole grid should fit the chip at once, since a second
  // round that is mostly empty costs as much as a full one.  With 128-column
  // tiles two work-groups share a compute unit; 192-column tiles take one
  // each.  Pick the size whose most loaded compute unit has the least work.
  const int nt128 = (cols + 127) / 128, nt192 = (cols + 191) / 192;
  const int64_t tiles128 = int64_t(nt128) * (nt128 + 1) / 2, tiles192 = int64_t(nt192) * (nt192 + 1) / 2;
  const int64_t cost128 = (tiles128 + kComputeUnits - 1) / kComputeUnits * 128 * 128;
  const int64_t cost192 = (tiles192 + kComputeUnits - 1) / kComputeUnits * 192 * 192;
  hipError_t e;
  if (cost192 < cost128)
    e = launch_tiles<192, 2, 4>(A, dtype, rows, cols, mu, G, nt192, stream);
  else
    e = launch_tiles<128, 2, 2>(A, dtype, rows, cols, mu, G, nt128, stream);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

hipError_t launch_head_similarity(const float* G, int32_t h, int32_t d, float* S,
                                  hipStream_t stream) {
  hipLaunchKernelGGL(head_sim_blocks, dim3(h, h), dim3(256), 0, stream, G, h, d, S);
  hipLaunchKernelGGL(head_sim_finish, dim3(1), dim3(1024), 0, stream, S, h);
  return hipGetLastError();
}

}  // namespace dckv
