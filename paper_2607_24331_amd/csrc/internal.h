// Internal declarations shared by the host plan code and the HIP kernels.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <string>
#include <vector>

#include "dckv.h"

namespace dckv {

// Per-query-head facts, passed by value as a kernel argument.
struct HeadTables {
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t q_per_kv;
  int32_t n_groups;
  int32_t qlen;                              // sum over heads of r_{g(h)}
  int32_t qoff[DCKV_MAX_HEADS + 1];          // folded-query offset of head h
  int32_t rank_of_q[DCKV_MAX_HEADS];         // r_{g(h)}
  int32_t koff_of_q[DCKV_MAX_HEADS];         // first key-latent column of g(h)
  int32_t rcol_of_q[DCKV_MAX_HEADS];         // first column of head h inside R_g
  int32_t rstride_of_q[DCKV_MAX_HEADS];      // row length of R_g: h_g * d_h
  int64_t roff_of_q[DCKV_MAX_HEADS];         // element offset of R_g
};

// Launch shape of one decode call, fixed by the plan and (batch, max_context).
struct DecodeShape {
  int32_t batch;
  int32_t max_context;
  int32_t split_tokens;
  int32_t n_split;          // ceil(max_context / split_tokens), at least 1
  size_t off_qt;            // workspace byte offsets
  size_t off_ml;
  size_t off_acc;
  size_t bytes;
};

}  // namespace dckv

struct dckv_plan {
  int32_t m, Hq, Hkv, dh, G, rv, dtype, split_tokens;
  int32_t RK, RKp, qpk, qlen;
  int64_t page_elems, value_base, key_factor_elems;
  std::vector<int32_t> group_of_kv, ranks, hg, pos_in_group, koff, qoff;
  std::vector<int64_t> roff;
  dckv::HeadTables tables;
  hipEvent_t prof_before = nullptr;  // benchmark instrumentation of the split kernel
  hipEvent_t prof_after = nullptr;
};

namespace dckv {

// Defined in the kernel sources.
DecodeShape decode_shape(const dckv_plan& p, int32_t batch, int32_t max_context);
hipError_t launch_append(const dckv_plan& p, const void* x, int32_t n_tok, const void* L_keys,
                         const void* L_value, const int64_t* slot, void* pool, int64_t num_pages,
                         hipStream_t stream);
hipError_t launch_decode(const dckv_plan& p, const DecodeShape& shape, const float* q,
                         const void* pool, int64_t num_pages, const int32_t* page_table,
                         int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                         const void* R_value, float* out, void* workspace, hipStream_t stream);

}  // namespace dckv
