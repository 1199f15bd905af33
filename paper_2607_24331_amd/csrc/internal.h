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
  int32_t n_queries;                         // Q: queries a sequence
  int32_t qlen;                              // sum over heads of r_{g(h)}
  int32_t qoff[DCKV_MAX_HEADS + 1];          // folded-query offset of head h
  int32_t rank_of_q[DCKV_MAX_HEADS];         // r_{g(h)}
  int32_t koff_of_q[DCKV_MAX_HEADS];         // first key-latent column of g(h)
  int32_t rcol_of_q[DCKV_MAX_HEADS];         // first column of head h inside R_g
  int32_t rstride_of_q[DCKV_MAX_HEADS];      // row length of R_g: h_g * d_h
  int64_t roff_of_q[DCKV_MAX_HEADS];         // element offset of R_g
};

constexpr int kMaxSlices = 8;     // (query, head) row slices of the MFMA decode path
constexpr int kSliceHeads = 32;   // at most two 16-head MFMA tiles per slice
constexpr int kUnitPages = 8;     // pages of a two-pass score work-group (one softmax exponent)
constexpr int kSharedWaves = 8;   // waves of a value work-group walking pages together (several slices)

// Schedule of the MFMA decode path (bf16 latents), fixed by the plan.  Rows
// (query, head) are ordered by (group, head, query), with the groups taken
// in the order the plan finds cheapest, and cut into J slices of at most
// 32; a work-group serves one slice of one context split.  The key columns
// a 16-row tile needs are the union of its groups' columns: at most two
// ranges of 32-column chunks, (kst[.][.][0], kln[.][.][0]) then
// (kst[.][.][1], kln[.][.][1]).
struct MfmaTables {
  int32_t n_slices;                        // J
  int32_t q_heads;                         // H_q
  int32_t queries;                         // Q: queries a sequence
  int32_t nt;                              // 16-head MFMA tiles per slice (1 or 2)
  int32_t mt_v;                            // value M-tiles: ceil(r_v / 16)
  int32_t waves;                           // waves a work-group: 4 or 8
  int32_t mtw;                             // value M-tiles per wave: ceil(mt_v / waves)
  int32_t mtw_t;                           // compiled tile capacity: 6, 8, 12, 16 or 32 >= mtw
  int32_t ring;                            // key block: loads in flight a wave (12, 14 or 16)
  int32_t max_pairs;                       // most LDS query blocks of any slice
  int32_t slice_heads[kMaxSlices];         // real rows in slice s
  int32_t hord[kMaxSlices][kSliceHeads];   // slot -> row i * H_q + h (query i, head h), -1 padding
  int32_t kst[kMaxSlices][2][2];           // first key chunk of each range of (slice, tile)
  int32_t kln[kMaxSlices][2][2];           // chunks in each range (0 for an unused range)
};

// Per-head facts of the rotary decode (rope.hip), built with the plan.  The
// key-rebuild kernel reads, for each KV head, the transposed factor blocks
// of its group: for every 32-column key chunk that meets the group's
// columns and every 16-row tile of the head's d_h rows, one 16 x 32 bf16
// block in MFMA A-operand order (zero outside the group's columns).
struct RopeTables {
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t q_per_kv;
  int32_t nh;                               // head slots a slice (16 * nt)
  int32_t koff[DCKV_MAX_HEADS];             // per KV head: first key column of its group
  int32_t rank[DCKV_MAX_HEADS];             // r_g of its group
  int32_t rcol[DCKV_MAX_HEADS];             // first column of the head inside R_g
  int32_t rstride[DCKV_MAX_HEADS];          // row length of R_g: h_g * d_h
  int32_t rt_off[DCKV_MAX_HEADS];           // element offset of the head's transposed blocks
  int32_t work_kv[DCKV_MAX_HEADS];          // KV heads in work order (group by group)
  int32_t qslot[DCKV_MAX_HEADS];            // query head -> slice * 32 + slot
  int64_t roff[DCKV_MAX_HEADS];             // per KV head: element offset of R_g
};

// Launch shape of one decode call, fixed by the plan and (batch, max_context).
struct DecodeShape {
  int32_t batch;
  int32_t max_context;
  int32_t split_tokens;
  int32_t n_split;          // ceil(max_context / split_tokens), at least 1
  bool mfma;                // bf16 single-pass MFMA path (split_mfma)
  bool pass;                // bf16 two-pass MFMA path (score_pages, value_pages)
  int32_t n_units;          // batch * n_split rounded up to a multiple of 8: grid units (MFMA path)
  int32_t n_rchunks;        // value-rank chunks of the merge (MFMA path)
  int32_t merge_ranks = 8;  // value ranks a merge work-group (8 or 16)
  // two-pass path
  int32_t npm;              // pages of the longest sequence: ceil(max_context / 64), at least 1
  int32_t unit_pages;       // pages a score work-group
  int32_t units_per_seq;    // score work-groups a sequence
  int32_t chunk_pages;      // pages a value chunk
  int32_t n_chunks;         // value chunks a sequence
  int32_t rgt;              // 16-rank value tiles a value work-group (4, 6 or 8), or with
                            // several row slices a wave (kSharedWaves waves a work-group)
  int32_t n_rgroups;        // value rank groups: ceil(r_v / (16 rgt)), with slices
                            // ceil(r_v / (16 kSharedWaves rgt))
  size_t off_qt;            // workspace byte offsets
  size_t off_ml;            // (m, l) of splits; two-pass: (E, L) of chunks
  size_t off_acc;           // split accumulators; two-pass: chunk accumulators
  size_t off_opart;         // merged value-latent rows
  size_t off_rt;            // rotary decode: transposed key factors
  size_t off_p;             // softmax weights (bf16): rotary splits; two-pass pages (with
                            // their (e, l) records)
  size_t bytes;
};

// Launch shape of one uncompressed decode call (dense.hip).
struct DenseShape {
  int32_t n_q_heads, n_kv_heads, head_dim, batch, max_context;
  int32_t split_tokens;     // context tokens a work-group
  int32_t n_split;          // ceil(max_context / split_tokens), at least 1
  size_t off_o, off_ml;     // workspace: unnormalised outputs, then (m, l)
  size_t bytes;
};

}  // namespace dckv

struct dckv_plan {
  int32_t m, Hq, Hkv, dh, G, rv, dtype, split_tokens, head_slices, decode_waves, Q;
  int32_t decode_passes;             // 0 per call, 1 single-pass, 2 two-pass
  int32_t RK, RKp, rvp, qpk, qlen;
  int64_t page_elems, value_base, key_factor_elems;
  std::vector<int32_t> group_of_kv, ranks, hg, pos_in_group, koff, qoff;
  std::vector<int64_t> roff;
  dckv::HeadTables tables;
  bool mfma_ok = false;              // bf16 single-pass MFMA decode path applies
  dckv::MfmaTables mfma{};
  bool pass_ok = false;              // bf16 two-pass decode applies (<= 256 (query, head) rows)
  dckv::MfmaTables pass{};           // its tables: slices of <= 32 rows, fewest chunk loads
  int32_t pass_ring = 0;             // score-pass loads in flight a wave (16; 32 measured slower)
  int32_t key_chunk_loads = 0;       // key chunks the MFMA tiles load a page
  dckv::RopeTables rope{};           // rotary decode tables (valid with mfma_ok)
  int64_t rope_rt_elems = 0;         // elements of the transposed key factors
  hipEvent_t prof_before = nullptr;  // benchmark instrumentation of the split kernel
  hipEvent_t prof_after = nullptr;
};

namespace dckv {

// Records a formatted message for dckv_last_error() and returns status.
int fail(int status, const char* fmt, ...);
bool aligned(const void* p, uintptr_t a);

// Offline contractions (gram.hip).
size_t gram_workspace_bytes(int64_t rows, int32_t cols);
hipError_t launch_gram(const void* A, int32_t dtype, int64_t rows, int32_t cols, bool center,
                       float* G, void* workspace, hipStream_t stream);
hipError_t launch_head_similarity(const float* G, int32_t h, int32_t d, float* S,
                                  hipStream_t stream);

// Host checks of a decode call (all but the workspace) and its launch shape.
int check_decode(const char* where, const dckv_plan* p, const float* q, int32_t batch,
                 const void* pool, int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                 const int32_t* seq_lens, int32_t max_context, const void* R_keys,
                 const void* R_value, const float* out, DecodeShape* shape);

// Builds plan.mfma and sets plan.mfma_ok (host only, no HIP call).
void build_mfma_tables(dckv_plan& p);

// Builds plan.pass and sets plan.pass_ok (host only, no HIP call).
void build_pass_tables(dckv_plan& p);

// Two-pass decode (decode_pass.hip).
size_t pass_score_lds_bytes(const dckv_plan& p);
size_t pass_value_lds_bytes(const dckv_plan& p, int rgt);
int pass_max_chunk_pages(const dckv_plan& p);
hipError_t launch_decode_pass(const dckv_plan& p, const DecodeShape& sh, const float* q,
                              const void* pool, int64_t num_pages, const int32_t* page_table,
                              int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                              const void* R_value, float* out, void* workspace, hipStream_t stream);
// o = a R_v for batch_rows (sequence, query) rows of merged value-latent rows.
hipError_t launch_upproj(const dckv_plan& p, int32_t batch_rows, const float* amerged,
                         const void* R_value, float* out, hipStream_t stream);
// Folded-query MFMA operand blocks (decode_mfma.hip) for the tables `mt`.
hipError_t launch_fold(const dckv_plan& p, const MfmaTables& mt, int32_t batch, const float* q,
                       const void* R_keys, void* qblk, hipStream_t stream);

// MFMA decode path (decode_mfma.hip).
size_t mfma_split_lds_bytes(const dckv_plan& p);
int mfma_merge_ranks(const dckv_plan& p, int32_t batch);   // value ranks a merge work-group
int mfma_max_split_tokens();
hipError_t launch_decode_mfma(const dckv_plan& p, const DecodeShape& sh, const float* q,
                              const void* pool, int64_t num_pages, const int32_t* page_table,
                              int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                              const void* R_value, float* out, void* workspace, hipStream_t stream);

// Rotary decode (rope.hip, decode_mfma.hip).
void build_rope_tables(dckv_plan& p);
DecodeShape rope_shape(const dckv_plan& p, int32_t batch, int32_t max_context);
int rope_max_q_per_kv();
size_t rope_value_lds_bytes(const dckv_plan& p, int32_t split_tokens);
hipError_t launch_rope_factors(const dckv_plan& p, const void* R_keys, void* rt, hipStream_t stream);
hipError_t launch_rope_scores(const dckv_plan& p, const DecodeShape& sh, const float* q,
                              const void* pool, int64_t num_pages, const int32_t* page_table,
                              int32_t max_pages, const int32_t* seq_lens, const void* rt,
                              double rope_base, void* pbuf, float* part_ml, hipStream_t stream);
hipError_t launch_decode_rope(const dckv_plan& p, const DecodeShape& sh, const float* q,
                              const void* pool, int64_t num_pages, const int32_t* page_table,
                              int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                              const void* R_value, double rope_base, float* out, void* workspace,
                              hipStream_t stream);

// Defined in the kernel sources.
DecodeShape decode_shape(const dckv_plan& p, int32_t batch, int32_t max_context);
DenseShape dense_shape(int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int32_t batch,
                       int32_t max_context, int32_t split_tokens);
hipError_t launch_dense_decode(const DenseShape& sh, const float* q, const void* pool,
                               int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                               const int32_t* seq_lens, float* out, void* workspace,
                               hipEvent_t before, hipEvent_t after, hipStream_t stream);
hipError_t launch_append(const dckv_plan& p, const void* x, int32_t n_tok, const void* L_keys,
                         const void* L_value, const int64_t* slot, void* pool, int64_t num_pages,
                         hipStream_t stream);
hipError_t launch_decode(const dckv_plan& p, const DecodeShape& shape, const float* q,
                         const void* pool, int64_t num_pages, const int32_t* page_table,
                         int32_t max_pages, const int32_t* seq_lens, const void* R_keys,
                         const void* R_value, float* out, void* workspace, hipStream_t stream);

}  // namespace dckv
