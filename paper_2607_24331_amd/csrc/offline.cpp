// Host side of the offline compression calls: argument checks before the
// Gram and head-similarity kernels are enqueued, and the two host steps of
// Algorithm 1 (head clustering; rank allocation), Sec. III-C.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <utility>
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

int dckv_cluster_merges(const double* S, int32_t num_heads, int32_t* merge_a, int32_t* merge_b,
                        double* height) {
  if (!S || (num_heads > 1 && (!merge_a || !merge_b)))
    return fail(DCKV_EINVAL, "cluster_merges: null S or output");
  const int h = num_heads;
  if (h < 1 || h > DCKV_MAX_HEADS)
    return fail(DCKV_EINVAL, "cluster_merges: num_heads %d outside [1,%d]", h, DCKV_MAX_HEADS);
  // A cluster is named by its smallest head.  d[a][b] is the average of
  // 1 - S over the member pairs of clusters a and b; after a and b merge
  // into a (a < b), the merged cluster's distance to any other cluster c is
  // the size-weighted mean (n_a d[a][c] + n_b d[b][c]) / (n_a + n_b), which
  // is that average over the merged member pairs again.
  double d[DCKV_MAX_HEADS][DCKV_MAX_HEADS];
  int size[DCKV_MAX_HEADS];
  bool live[DCKV_MAX_HEADS];
  for (int i = 0; i < h; ++i) {
    size[i] = 1;
    live[i] = true;
    for (int j = 0; j < h; ++j) d[i][j] = 1.0 - S[i * h + j];
  }
  for (int step = 0; step + 1 < h; ++step) {
    // the closest pair; scanning (a, b) in ascending order of the clusters'
    // smallest heads makes the first of equal distances the lexicographically
    // smallest pair
    int ba = -1, bb = -1;
    for (int a = 0; a < h; ++a) {
      if (!live[a]) continue;
      for (int b = a + 1; b < h; ++b)
        if (live[b] && (ba < 0 || d[a][b] < d[ba][bb])) {
          ba = a;
          bb = b;
        }
    }
    merge_a[step] = ba;
    merge_b[step] = bb;
    if (height) height[step] = d[ba][bb];
    const double wa = size[ba], wb = size[bb], w = wa + wb;
    for (int c = 0; c < h; ++c) {
      if (!live[c] || c == ba || c == bb) continue;
      const double v = (wa * d[ba][c] + wb * d[bb][c]) / w;
      d[ba][c] = v;
      d[c][ba] = v;
    }
    size[ba] += size[bb];
    live[bb] = false;
  }
  return DCKV_OK;
}

int dckv_cluster_heads(const double* S, int32_t num_heads, int32_t K, int32_t* group_of_head) {
  if (!S || !group_of_head) return fail(DCKV_EINVAL, "cluster_heads: null S or output");
  const int h = num_heads;
  if (h < 1 || h > DCKV_MAX_HEADS) return fail(DCKV_EINVAL, "cluster_heads: num_heads %d outside [1,%d]", h, DCKV_MAX_HEADS);
  if (K < 1 || K > h) return fail(DCKV_EINVAL, "cluster_heads: K %d outside [1,%d]", K, h);
  int32_t ma[DCKV_MAX_HEADS], mb[DCKV_MAX_HEADS];
  const int st = dckv_cluster_merges(S, h, ma, mb, nullptr);
  if (st != DCKV_OK) return st;
  // the first h - K merges of the sequence leave K clusters; each head
  // follows its cluster's name (smallest head) through the merges
  int root[DCKV_MAX_HEADS];
  for (int i = 0; i < h; ++i) root[i] = i;
  for (int s = 0; s < h - K; ++s)
    for (int i = 0; i < h; ++i)
      if (root[i] == mb[s]) root[i] = ma[s];
  // groups numbered in ascending order of their smallest head
  int label[DCKV_MAX_HEADS];
  int next = 0;
  for (int i = 0; i < h; ++i) label[i] = (root[i] == i) ? next++ : -1;
  for (int i = 0; i < h; ++i) group_of_head[i] = label[root[i]];
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
  int64_t weighted = 0, total = 0;          // sum r_i h_i and sum r_i
  for (int i = 0; i < K; ++i) {
    const int ri = int(std::floor(double(r) * energy[i] / energy_total + 0.5));
    init_ranks[i] = std::max(1, std::min(ri, rank_cap[i]));
    ranks[i] = init_ranks[i];
    weighted += int64_t(ranks[i]) * heads[i];
    total += ranks[i];
  }
  // Lowering group i from rank k to k - 1 costs sigma_{i,k}^2 * h / h_i, and
  // a group's costs only grow as its rank falls (singular values descend).
  // So the greedy rule -- always the cheapest single step, the lower group
  // id on equal costs -- takes the steps of all groups in ascending
  // (cost, group) order: a min-heap holding each group's next step.
  auto cost = [&](int i) {
    const double s = sigma[int64_t(i) * sigma_stride + ranks[i] - 1];
    return s * s * double(h) / double(heads[i]);
  };
  std::vector<std::pair<double, int>> heap;
  heap.reserve(K);
  auto later = [](const std::pair<double, int>& x, const std::pair<double, int>& y) { return x > y; };
  for (int i = 0; i < K; ++i)
    if (ranks[i] > 1) heap.emplace_back(cost(i), i);
  std::make_heap(heap.begin(), heap.end(), later);
  while ((weighted > 4 * int64_t(r) || total > r) && !heap.empty()) {
    std::pop_heap(heap.begin(), heap.end(), later);
    const int i = heap.back().second;
    heap.pop_back();
    --ranks[i];
    weighted -= heads[i];
    --total;
    if (ranks[i] > 1) {
      heap.emplace_back(cost(i), i);
      std::push_heap(heap.begin(), heap.end(), later);
    }
  }
  return DCKV_OK;
}

}  // extern "C"
