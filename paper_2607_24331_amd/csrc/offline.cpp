// Host side of the offline compression calls: argument checks before the
// Gram and head-similarity kernels are enqueued, and the two host steps of
// Algorithm 1 (head clustering; rank allocation), Sec. III-C.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "internal.h"

using dckv::aligned;
using dckv::fail;

extern "C" {

int dckv_gram_workspace_bytes(int64_t rows, int32_t cols, int32_t center, size_t* bytes) {
  if (!bytes) return fail(DCKV_EINVAL, "gram_workspace_bytes: null output pointer");
  if (rows < 1 || cols < 1) return fail(DCKV_EINVAL, "gram_workspace_bytes: rows %lld, cols %d", (long long)rows, cols);
  *bytes = center ? dckv::gram_workspace_bytes(rows, cols) : 0;
  return DCKV_OK;
}

int dckv_gram(const void* A, int32_t dtype, int64_t rows, int32_t cols, int32_t center, float* G,
              void* workspace, size_t workspace_bytes, void* stream) {
  if (!A || !G) return fail(DCKV_EINVAL, "gram: null A or G");
  if (dtype != DCKV_F32 && dtype != DCKV_BF16)
    return fail(DCKV_EDTYPE, "gram: dtype %d is neither DCKV_F32 nor DCKV_BF16", dtype);
  if (rows < 1 || rows > int64_t(65535) * 256)
    return fail(DCKV_EINVAL, "gram: rows %lld outside [1, 65535*256]", (long long)rows);
  if (cols < 8 || cols % 8 != 0 || cols > 32768)
    return fail(DCKV_EINVAL, "gram: cols %d is not a multiple of 8 in [8, 32768]", cols);
  if (!aligned(A, 16) || !aligned(G, 16)) return fail(DCKV_EALIGN, "gram: A and G must be 16-byte aligned");
  const size_t need = center ? dckv::gram_workspace_bytes(rows, cols) : 0;
  if (need > 0) {
    if (!workspace || workspace_bytes < need)
      return fail(DCKV_EWORKSPACE, "gram: workspace %zu bytes < %zu", workspace_bytes, need);
    if (!aligned(workspace, 256)) return fail(DCKV_EALIGN, "gram: workspace must be 256-byte aligned");
  }
  const hipError_t e = dckv::launch_gram(A, dtype, rows, cols, center != 0, G, workspace,
                                         static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(DCKV_EHIP, "gram: %s", hipGetErrorString(e));
  return DCKV_OK;
}

int dckv_head_similarity(const float* G, int32_t num_heads, int32_t head_dim, float* S,
                         void* stream) {
  if (!G || !S) return fail(DCKV_EINVAL, "head_similarity: null G or S");
  if (num_heads < 1 || num_heads > DCKV_MAX_HEADS)
    return fail(DCKV_EINVAL, "head_similarity: num_heads %d outside [1,%d]", num_heads, DCKV_MAX_HEADS);
  if (head_dim < 1 || head_dim > DCKV_MAX_HEAD_DIM)
    return fail(DCKV_EINVAL, "head_similarity: head_dim %d outside [1,%d]", head_dim, DCKV_MAX_HEAD_DIM);
  if (!aligned(G, 4) || !aligned(S, 4)) return fail(DCKV_EALIGN, "head_similarity: misaligned G or S");
  const hipError_t e = dckv::launch_head_similarity(G, num_heads, head_dim, S,
                                                    static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(DCKV_EHIP, "head_similarity: %s", hipGetErrorString(e));
  return DCKV_OK;
}

int dckv_cluster_heads(const double* S, int32_t num_heads, int32_t K, int32_t* group_of_head) {
  if (!S || !group_of_head) return fail(DCKV_EINVAL, "cluster_heads: null S or output");
  const int h = num_heads;
  if (h < 1 || h > DCKV_MAX_HEADS) return fail(DCKV_EINVAL, "cluster_heads: num_heads %d outside [1,%d]", h, DCKV_MAX_HEADS);
  if (K < 1 || K > h) return fail(DCKV_EINVAL, "cluster_heads: K %d outside [1,%d]", K, h);
  // clusters as sorted member lists; the distance between clusters is the
  // mean over member pairs of 1 - S[i][j], summed in member order
  std::vector<std::vector<int>> cl(h);
  for (int i = 0; i < h; ++i) cl[i] = {i};
  while (int(cl.size()) > K) {
    int ba = -1, bb = -1;
    double bd = 0.0;
    for (int a = 0; a < int(cl.size()); ++a)
      for (int b = a + 1; b < int(cl.size()); ++b) {
        double s = 0.0;
        for (int i : cl[a])
          for (int j : cl[b]) s += 1.0 - S[i * h + j];
        const double d = s / double(cl[a].size() * cl[b].size());
        // clusters are kept ordered by smallest member, so (a, b) order is the
        // lexicographic order of (min a, min b)
        if (ba < 0 || d < bd) {
          bd = d;
          ba = a;
          bb = b;
        }
      }
    std::vector<int> merged = cl[ba];
    merged.insert(merged.end(), cl[bb].begin(), cl[bb].end());
    std::sort(merged.begin(), merged.end());
    cl.erase(cl.begin() + bb);
    cl.erase(cl.begin() + ba);
    cl.push_back(merged);
    std::sort(cl.begin(), cl.end(), [](const std::vector<int>& x, const std::vector<int>& y) { return x[0] < y[0]; });
  }
  for (int g = 0; g < int(cl.size()); ++g)
    for (int i : cl[g]) group_of_head[i] = g;
  return DCKV_OK;
}

int dckv_allocate_ranks(int32_t K, const int32_t* heads, const double* energy,
                        double energy_total, const double* sigma, int32_t sigma_stride,
                        const int32_t* rank_cap, int32_t r, int32_t* init_ranks, int32_t* ranks) {
  if (!heads || !energy || !sigma || !rank_cap || !init_ranks || !ranks)
    return fail(DCKV_EINVAL, "allocate_ranks: null pointer");
  if (K < 1 || K > DCKV_MAX_HEADS) return fail(DCKV_EINVAL, "allocate_ranks: K %d outside [1,%d]", K, DCKV_MAX_HEADS);
  if (r < 1) return fail(DCKV_EINVAL, "allocate_ranks: budget %d < 1", r);
  if (!(energy_total > 0.0)) return fail(DCKV_EINVAL, "allocate_ranks: total energy must be positive");
  int64_t h = 0;
  for (int i = 0; i < K; ++i) {
    if (heads[i] < 1) return fail(DCKV_EINVAL, "allocate_ranks: group %d has %d heads", i, heads[i]);
    if (rank_cap[i] < 1 || rank_cap[i] > sigma_stride)
      return fail(DCKV_EINVAL, "allocate_ranks: rank cap %d of group %d outside [1, sigma_stride %d]", rank_cap[i], i, sigma_stride);
    h += heads[i];
  }
  for (int i = 0; i < K; ++i) {
    const int ri = int(std::floor(double(r) * energy[i] / energy_total + 0.5));
    init_ranks[i] = std::max(1, std::min(ri, rank_cap[i]));
    ranks[i] = init_ranks[i];
  }
  auto holds = [&]() {
    int64_t weighted = 0, total = 0;
    for (int i = 0; i < K; ++i) {
      weighted += int64_t(ranks[i]) * heads[i];
      total += ranks[i];
    }
    return weighted <= 4 * int64_t(r) && total <= r;
  };
  while (!holds()) {
    int best = -1;
    double bc = 0.0;
    for (int i = 0; i < K; ++i) {
      if (ranks[i] <= 1) continue;
      const double s = sigma[int64_t(i) * sigma_stride + ranks[i] - 1];
      const double c = s * s * double(h) / double(heads[i]);
      if (best < 0 || c < bc) {
        bc = c;
        best = i;
      }
    }
    if (best < 0) break;                         // every group at rank 1
    --ranks[best];
  }
  return DCKV_OK;
}

}  // extern "C"
