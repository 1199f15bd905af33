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

constexpr int kGT = 128;                  // output tile (rows and columns)
constexpr int kGK = 32;                   // samples a staging step
constexpr int kGPad = 144;                // LDS row stride in floats (bank-conflict-free reads)
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

// 16 consecutive columns of one sample as fp32, centred; zero outside A.
template <typename T>
__device__ __forceinline__ void load16(const T* __restrict__ A, int64_t rows, int cols,
                                       int64_t r, int c, const float* mu16, float (&v)[16]);

template <>
__device__ __forceinline__ void load16<float>(const float* __restrict__ A, int64_t rows, int cols,
                                              int64_t r, int c, const float* mu16, float (&v)[16]) {
  const int64_t rr = r < rows ? r : rows - 1;          // clamped: every load is in bounds
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int cc = c + 4 * k < cols ? c + 4 * k : 0;
    const float4 x = *reinterpret_cast<const float4*>(A + rr * cols + cc);
    v[4 * k + 0] = x.x;
    v[4 * k + 1] = x.y;
    v[4 * k + 2] = x.z;
    v[4 * k + 3] = x.w;
  }
#pragma unroll
  for (int k = 0; k < 16; ++k) v[k] = (r < rows && c + k < cols) ? v[k] - mu16[k] : 0.f;
}

template <>
__device__ __forceinline__ void load16<bf16>(const bf16* __restrict__ A, int64_t rows, int cols,
                                             int64_t r, int c, const float* mu16, float (&v)[16]) {
  const int64_t rr = r < rows ? r : rows - 1;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int cc = c + 8 * k < cols ? c + 8 * k : 0;
    const uint4 x = *reinterpret_cast<const uint4*>(A + rr * cols + cc);
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[8 * k + 2 * j] = __uint_as_float(w[j] << 16);
      v[8 * k + 2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
#pragma unroll
  for (int k = 0; k < 16; ++k) v[k] = (r < rows && c + k < cols) ? v[k] - mu16[k] : 0.f;
}

// One 128 x 128 tile (ti <= tj) of G per work-group; 4 waves of 64 x 64.
// Staging: 32 samples x 128 columns of the tile's row block and column block
// in LDS (double-buffered), each thread 16 columns of one sample, the next
// step's loads in flight during the current step's products.  Products:
// lane l feeds A[i = l % 16][k = l / 16] and B[k = l / 16][j = l % 16];
// the accumulator holds D[4 (l / 16) + v][l % 16].  An off-diagonal tile is
// written twice: as is, and transposed through LDS into the mirror tile.
template <typename T>
__global__ __launch_bounds__(256) void gram_tiles(const T* __restrict__ A, int64_t rows, int cols,
                                                  const float* __restrict__ mu,
                                                  float* __restrict__ G, int n_tiles) {
  __shared__ __align__(16) float smem[2 * 2 * kGK * kGPad];
  int lin = blockIdx.x, ti = 0;
  while (lin >= n_tiles - ti) {
    lin -= n_tiles - ti;
    ++ti;
  }
  const int tj = ti + lin;
  const bool diag = ti == tj;
  const int i0 = ti * kGT, j0 = tj * kGT;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wi = w >> 1, wj = w & 1;
  const int srow = tid >> 3, scol = (tid & 7) * 16;    // staging: sample, first column
  float muI[16], muJ[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int ci = i0 + scol + k, cj = j0 + scol + k;
    muI[k] = (mu && ci < cols) ? mu[ci] : 0.f;
    muJ[k] = (mu && cj < cols) ? mu[cj] : 0.f;
  }
  floatx4 acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nsteps = int((rows + kGK - 1) / kGK);
  float vI[16], vJ[16];
  load16<T>(A, rows, cols, srow, i0 + scol, muI, vI);
  if (!diag) load16<T>(A, rows, cols, srow, j0 + scol, muJ, vJ);
  for (int st = 0; st < nsteps; ++st) {
    float* sI = smem + (st & 1) * 2 * kGK * kGPad;
    float* sJ = diag ? sI : sI + kGK * kGPad;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      *reinterpret_cast<float4*>(sI + srow * kGPad + scol + 4 * k) =
          make_float4(vI[4 * k], vI[4 * k + 1], vI[4 * k + 2], vI[4 * k + 3]);
    if (!diag) {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        *reinterpret_cast<float4*>(sJ + srow * kGPad + scol + 4 * k) =
            make_float4(vJ[4 * k], vJ[4 * k + 1], vJ[4 * k + 2], vJ[4 * k + 3]);
    }
    __syncthreads();
    if (st + 1 < nsteps) {
      const int64_t r = int64_t(st + 1) * kGK + srow;
      load16<T>(A, rows, cols, r, i0 + scol, muI, vI);
      if (!diag) load16<T>(A, rows, cols, r, j0 + scol, muJ, vJ);
    }
#pragma unroll
    for (int s = 0; s < kGK / 4; ++s) {
      const int kr = 4 * s + (lane >> 4);
      float a[4], b[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) a[x] = sI[kr * kGPad + 64 * wi + 16 * x + (lane & 15)];
#pragma unroll
      for (int y = 0; y < 4; ++y) b[y] = sJ[kr * kGPad + 64 * wj + 16 * y + (lane & 15)];
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[x], b[y], acc[x][y], 0, 0, 0);
    }
  }

  // the tile as is
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = i0 + 64 * wi + 16 * x + 4 * (lane >> 4) + v;
        const int j = j0 + 64 * wj + 16 * y + (lane & 15);
        if (i < cols && j < cols) G[int64_t(i) * cols + j] = acc[x][y][v];
      }
  if (diag) return;
  // the mirror tile: each wave transposes its 64 x 64 block through LDS
  __syncthreads();                                      // staging buffers no longer read
  float* tw = smem + w * 64 * 65;
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        tw[(16 * y + (lane & 15)) * 65 + 16 * x + 4 * (lane >> 4) + v] = acc[x][y][v];
  __syncthreads();
  for (int rr = 0; rr < 64; ++rr) {
    const int j = j0 + 64 * wj + rr, i = i0 + 64 * wi + lane;
    if (j < cols && i < cols) G[int64_t(j) * cols + i] = tw[rr * 65 + lane];
  }
}

// S[i][j] from the Gram blocks; one work-group a (i, j), fixed-order sums.
__global__ __launch_bounds__(256) void head_sim(const float* __restrict__ G, int h, int d,
                                                float* __restrict__ S) {
  const int i = blockIdx.x, j = blockIdx.y;
  const int n = h * d, tid = threadIdx.x;
  __shared__ float red[3][256];
  float f[3] = {0.f, 0.f, 0.f};
  const int bi[3] = {i, i, j}, bj[3] = {j, i, j};
#pragma unroll
  for (int q = 0; q < 3; ++q)
    for (int e = tid; e < d * d; e += 256) {
      const float g = G[int64_t(bi[q] * d + e / d) * n + bj[q] * d + e % d];
      f[q] = fmaf(g, g, f[q]);
    }
#pragma unroll
  for (int q = 0; q < 3; ++q) red[q][tid] = f[q];
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s)
#pragma unroll
      for (int q = 0; q < 3; ++q) red[q][tid] += red[q][tid + s];
    __syncthreads();
  }
  if (tid == 0) {
    const float den = sqrtf(red[1][0]) * sqrtf(red[2][0]);
    S[i * h + j] = den > 0.f ? red[0][0] / den : 0.f;
  }
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
  const int nt = (cols + kGT - 1) / kGT;
  const dim3 grid(unsigned(nt * (nt + 1) / 2));
  if (dtype == DCKV_BF16)
    hipLaunchKernelGGL(gram_tiles<bf16>, grid, dim3(256), 0, stream, static_cast<const bf16*>(A),
                       rows, cols, mu, G, nt);
  else
    hipLaunchKernelGGL(gram_tiles<float>, grid, dim3(256), 0, stream, static_cast<const float*>(A),
                       rows, cols, mu, G, nt);
  return hipGetLastError();
}

hipError_t launch_head_similarity(const float* G, int32_t h, int32_t d, float* S,
                                  hipStream_t stream) {
  hipLaunchKernelGGL(head_sim, dim3(h, h), dim3(256), 0, stream, G, h, d, S);
  return hipGetLastError();
}

}  // namespace dckv
