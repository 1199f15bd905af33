/*
 * dckv.h -- compressed-KV decode attention (DynaCalKV) on MI355X (gfx950).
 *
 * The method (Sec. III of the paper) caches, per token, low-rank latents
 * instead of keys and values:
 *   keys    the key projection W^(k) is split column-wise into groups of
 *           heads; group g is factored W_g ~ L_g R_g with its own rank r_g
 *           (Sec. III-C), so each token stores one r_g-wide latent per group;
 *   values  the whole value projection is factored W^(v) ~ L_v R_v with one
 *           rank r_v (Sec. III-D), so each token stores one r_v-wide latent
 *           shared by every head;
 *   write   z = x L (Sec. III-A) for new tokens;
 *   read    x W ~ z R (Sec. III-A), used here without rebuilding keys or
 *           values: each query head is folded into its group's latent space
 *           (q_h R_{g,h}^T), scores are taken against the key latents, the
 *           softmax-weighted sum is accumulated in value-latent space and
 *           multiplied once by the head's slice of R_v.
 *
 * Conventions of this library (readings where the paper is silent):
 *   - softmax scale 1/sqrt(d_h); no positional transform (dckv_decode_rope
 *     below is the rotary variant); no mask (a decode query attends to
 *     every cached token of its sequence);
 *   - query head h reads KV head floor(h / (H_q / H_kv));
 *   - the heads of group g are ordered by ascending KV-head index: the j-th
 *     of them owns columns [j*d_h, (j+1)*d_h) of R_g;
 *   - group g's latent occupies key-latent columns [koff_g, koff_g + r_g),
 *     koff_g = r_0 + ... + r_{g-1}.
 *
 * Paged cache layout (64 tokens per page; R_K = sum_g r_g; R_Kp = R_K
 * rounded up to a multiple of 32; r_vp = r_v rounded up to a multiple of 16;
 * page_elems = 64*R_Kp + 64*r_vp elements of the latent dtype):
 *   key part    chunk-major: key columns in chunks of 32, each chunk holding
 *               the 64 slots one after another: (slot s, key column k) at
 *               (k/32)*2048 + s*32 + k%32; columns R_K..R_Kp-1 are written
 *               as zero by dckv_latent_append
 *   value part  tile-major: value columns in tiles of 16, each tile holding
 *               the slot halves 0-31 and 32-63 in turn as 16 columns x 32
 *               slots: (slot s, value column j) at 64*R_Kp + (j/16)*1024 +
 *               (s/32)*512 + (j%16)*32 + s%32; columns r_v..r_vp-1 are
 *               never written and never read
 *   Either way one 16 x 32 MFMA operand tile (16 tokens x 32 key columns, or
 *   16 value columns x 32 tokens) is one contiguous run of 512 elements.
 *   Position pos of sequence b lives in page page_table[b*max_pages + pos/64],
 *   slot pos%64.  Page p starts at element p*page_elems of the pool.
 *
 * Threading and ownership: the caller owns every device buffer (inputs,
 * outputs, pool, workspace).  The library owns only the host-side plan.
 * dckv_latent_append and dckv_decode enqueue kernels on the given HIP stream
 * and return without synchronising; they allocate no device memory, copy
 * nothing between host and device and never block.  All arguments are
 * validated on the host before any launch: on failure the call returns a
 * negative status, records a message for dckv_last_error and enqueues
 * nothing.  Faults inside kernels surface at the caller's next
 * synchronisation.  A plan may be shared by threads; the error message is
 * per thread.
 */
#ifndef DCKV_H
#define DCKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DCKV_PAGE_TOKENS 64
#define DCKV_MAX_HEADS 64      /* H_q limit */
#define DCKV_MAX_GROUPS 64     /* G limit */
#define DCKV_MAX_HEAD_DIM 256  /* d_h limit */
#define DCKV_MAX_VALUE_RANK 4096
#define DCKV_MAX_GROUP_RANK 4096
#define DCKV_MAX_QUERIES 64     /* queries a sequence in one decode call */

typedef enum {
  DCKV_OK = 0,
  DCKV_EINVAL = -1,      /* bad shape, partition, rank, pointer or size */
  DCKV_EDTYPE = -2,      /* unsupported latent dtype */
  DCKV_EALIGN = -3,      /* a device pointer is not 16-byte aligned */
  DCKV_EWORKSPACE = -4,  /* workspace smaller than dckv_decode_workspace_bytes */
  DCKV_EHIP = -5,        /* a HIP launch or query failed */
  DCKV_ENOMEM = -6       /* host allocation for the plan failed */
} dckv_status;

typedef enum { DCKV_F32 = 0, DCKV_BF16 = 1 } dckv_dtype;

/* One attention layer's compressed-KV description (host memory; copied by
 * dckv_plan_create, so the arrays may be freed afterwards). */
typedef struct dckv_layer_desc {
  int32_t hidden;                  /* m: width of x (input of the K/V projections) */
  int32_t num_q_heads;             /* H_q, 1..DCKV_MAX_HEADS, multiple of num_kv_heads */
  int32_t num_kv_heads;            /* H_kv: the key/value heads the groups partition */
  int32_t head_dim;                /* d_h, 1..DCKV_MAX_HEAD_DIM */
  int32_t num_groups;              /* G, 1..DCKV_MAX_GROUPS */
  const int32_t* group_of_kv_head; /* [H_kv] group id of each KV head; every group
                                      must receive at least one head (Sec. III-C:
                                      the group sizes sum to the head count) */
  const int32_t* group_rank;       /* [G] r_g with 1 <= r_g <= min(m, h_g*d_h) */
  int32_t value_rank;              /* r_v with 1 <= r_v <= min(m, H_kv*d_h) */
  int32_t latent_dtype;            /* dckv_dtype of latents, x and the L/R factors */
  int32_t split_tokens;            /* context tokens per decode work split; a
                                      multiple of 64, or 0 to choose per call from
                                      (batch, max_context) */
  int32_t head_slices;             /* slices of the (query, head) rows served by
                                      separate decode work-groups (bf16 path); 0 for
                                      the default (one slice per 32 rows) */
  int32_t queries_per_seq;         /* Q: queries a sequence in one decode call (0 or 1:
                                      plain decode; more: speculative verification or
                                      chunked prefill), at most DCKV_MAX_QUERIES */
  int32_t decode_waves;            /* waves of a bf16 decode work-group: 4 or 8,
                                      or 0 for the default (eight when every wave
                                      gets at least one 16-rank value tile, i.e.
                                      r_v > 112, else four) */
  int32_t decode_passes;           /* bf16 decode kernels: 0 chooses per call (the
                                      single-pass split kernel, except for one query a
                                      sequence and at most 32 query heads when it would
                                      need several row slices -- value ranks above what
                                      one slice's accumulators hold -- and the call holds
                                      at least 2048 page slots, or when it does not
                                      apply: then the two-pass kernels); 1 never the
                                      two-pass kernels; 2 always the two-pass kernels
                                      (DCKV_EINVAL if the layer does not fit them) */
} dckv_layer_desc;

/* Derived layout facts of a plan. */
typedef struct dckv_plan_geometry {
  int32_t key_rank_total;          /* R_K = sum of r_g */
  int32_t key_width_padded;        /* R_Kp: R_K rounded up to a multiple of 32 */
  int32_t value_width_padded;      /* r_vp: r_v rounded up to a multiple of 16 */
  int32_t value_rank;              /* r_v */
  int32_t q_per_kv;                /* H_q / H_kv */
  int32_t folded_query_len;        /* sum over query heads h of r_{g(h)} */
  int32_t split_tokens;            /* tokens per decode split as described (0: per call) */
  int32_t mfma_path;               /* 1 if decode uses the bf16 MFMA kernels */
  int32_t head_slices;             /* query-head slices of the MFMA path (0 otherwise) */
  int32_t queries_per_seq;         /* Q of the plan (at least 1) */
  int32_t decode_waves;            /* waves a decode work-group on the MFMA path (0 otherwise) */
  int32_t decode_ring;             /* key-phase block of the MFMA path: 16-byte loads in
                                      flight a wave while keys stream (12, 14 or 16: the
                                      size that pads the slowest wave's key loads least;
                                      value loads go in blocks of 12 or 16 fixed by the
                                      value tiles a wave; 0 otherwise) */
  int32_t value_tiles_per_wave;    /* 16-rank value tiles a wave on the MFMA path (0 otherwise) */
  int32_t key_chunk_loads;         /* 32-column key chunks the MFMA path loads a 64-token page,
                                      summed over its 16-row tiles: a tile loads the chunks of
                                      its rows' groups, so a group cut by a tile boundary is
                                      loaded twice (0 otherwise) */
  int32_t two_pass;                /* 1 if one-query decodes of this plan may take the
                                      two-pass MFMA kernels (a score pass writing each
                                      page's softmax weights, then a value pass over
                                      value-rank groups), as decode_passes chooses */
  int32_t reserved0;
  int64_t page_elems;              /* elements per page: 64*R_Kp + 64*r_vp */
  int64_t value_base;              /* element offset of the value part in a page: 64*R_Kp */
  int64_t key_factor_elems;        /* elements of the concatenated R_g blocks */
} dckv_plan_geometry;

typedef struct dckv_plan dckv_plan;  /* opaque, host memory only */

/* Validate a layer description and build its plan (bookkeeping of Sec.
 * III-C: the partition, head ratios, per-group column offsets).  Returns
 * DCKV_EINVAL / DCKV_EDTYPE for invalid descriptions (*out untouched),
 * DCKV_ENOMEM if the host allocation fails.  Makes no HIP call. */
int dckv_plan_create(const dckv_layer_desc* desc, dckv_plan** out);

/* Free a plan (NULL is accepted). */
void dckv_plan_destroy(dckv_plan* plan);

/* Copy the plan's bookkeeping out (host memory; any pointer may be NULL to
 * skip that array):
 *   geo           layout facts above
 *   koff          [G]      koff_g, first key-latent column of group g
 *   pos_in_group  [H_kv]   position of each KV head inside its group
 *   qoff          [H_q+1]  offset of query head h's folded query
 *                          (r_{g(h)} values) within one sequence's block
 *   roff          [G+1]    element offset of R_g in the concatenated blocks
 * Makes no HIP call. */
int dckv_plan_info(const dckv_plan* plan, dckv_plan_geometry* geo, int32_t* koff,
                   int32_t* pos_in_group, int32_t* qoff, int64_t* roff);

/* Bytes of device workspace dckv_decode needs for `batch` sequences of at
 * most `max_context` tokens.  Makes no HIP call. */
int dckv_decode_workspace_bytes(const dckv_plan* plan, int32_t batch, int32_t max_context,
                                size_t* bytes);

/* The launch a dckv_decode call of `batch` sequences of at most
 * `max_context` tokens takes: which kernels, and how the context is cut
 * (it depends on the plan and these two numbers only). */
typedef struct dckv_launch_info {
  int32_t kernels;       /* 0 portable VALU kernels, 1 single-pass MFMA split kernel,
                            2 two-pass MFMA kernels */
  int32_t split_tokens;  /* context tokens a split (a value chunk on the two-pass path) */
  int32_t n_split;       /* splits (chunks) of the longest sequence */
  int32_t head_slices;   /* row slices of the MFMA kernels (each slice's score work
                            reads its groups' key chunks; on the single-pass kernel
                            each also reads the value part), 1 on the portable path */
  int32_t value_tiles;   /* two-pass path: 16-rank value tiles a value work-group
                            (0 otherwise) */
} dckv_launch_info;
int dckv_decode_launch_info(const dckv_plan* plan, int32_t batch, int32_t max_context,
                            dckv_launch_info* info);

/* Latent write for new tokens (Sec. III-A z = x L, per group L_g of Sec.
 * III-C and whole-projection L_v of Sec. III-D), computed with fp32
 * accumulation and rounded to nearest-even into the pool.
 *   x        device [n_tok, m] row-major, latent dtype
 *   L_keys   device [R_K, m] row-major: the transpose of [L_0 | L_1 | ... |
 *            L_{G-1}] (m x R_K), i.e. the [out, in] layout of a linear
 *            layer's weight; row koff_g + j holds column j of L_g
 *   L_value  device [r_v, m] row-major: the transpose of L_v (m x r_v)
 *   slot     device int64 [n_tok]: page*64 + slot-in-page of each token;
 *            a negative slot, or one at or beyond num_pages*64, skips the token
 *   pool     device, num_pages * page_elems elements of the latent dtype
 *   stream   hipStream_t (NULL: the null stream)
 * n_tok == 0 is a no-op.  Pointers must be 16-byte aligned.  Two tokens
 * with the same slot race (the last write is unspecified). */
int dckv_latent_append(const dckv_plan* plan, const void* x, int32_t n_tok,
                       const void* L_keys, const void* L_value, const int64_t* slot,
                       void* pool, int64_t num_pages, void* stream);

/* Decode attention over the compressed cache for Q = queries_per_seq
 * queries per sequence (Q = 1: plain decode).  The Q new tokens already
 * occupy the last Q cache positions of their sequence: query i sits at
 * position seq_len - Q + i and attends to every position up to and including
 * its own (a causal mask inside the chunk); a query that sees no position
 * gets zeros.
 *   q           device fp32 [batch, Q, H_q, d_h]
 *   pool        device, laid out as above (num_pages pages)
 *   page_table  device int32 [batch, max_pages]; entries outside
 *               [0, num_pages) are treated as empty pages (no fault, their
 *               tokens contribute nothing)
 *   seq_lens    device int32 [batch]; each is clamped to [0, max_context]
 *   max_context host bound on every seq_len, at most max_pages*64
 *   R_keys      device, the R_g blocks back to back, each [r_g, h_g*d_h]
 *               row-major, group 0 first (key_factor_elems in total)
 *   R_value     device [r_v, H_kv*d_h] row-major
 *   out         device fp32 [batch, Q, H_q, d_h]; a sequence of length 0 gets zeros
 *   workspace   device scratch of at least dckv_decode_workspace_bytes(batch,
 *               max_context) bytes, 256-byte aligned; its contents on entry
 *               do not matter and are overwritten
 * Results are bitwise reproducible for a fixed plan and inputs: the work
 * split depends only on split_tokens and every reduction runs in a fixed
 * order.  batch == 0 is a no-op; batch * Q is at most 65535. */
int dckv_decode(const dckv_plan* plan, const float* q, int32_t batch, const void* pool,
                int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                const int32_t* seq_lens, int32_t max_context, const void* R_keys,
                const void* R_value, float* out, void* workspace, size_t workspace_bytes,
                void* stream);

/* Decode that allocates nothing, for callers that cannot allocate device
 * memory or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same computation, kernels,
 * arguments, validation and bitwise results as dckv_decode, without the
 * workspace: the scratch lives in a fixed device array of
 * DCKV_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds until
 * the process ends.  A call whose dckv_decode_workspace_bytes exceeds that
 * size returns DCKV_EWORKSPACE and enqueues nothing.  The call itself never
 * calls hipMalloc or hipFree; the first call on a device looks the array's
 * address up once (hipGetSymbolAddress).  Every call on one GPU shares that
 * GPU's array: calls that may overlap on one GPU (different streams, several
 * threads) race and must be ordered by the caller.  The array needs no
 * clearing: every byte a call reads was written earlier in that call. */
#define DCKV_NOALLOC_SCRATCH_BYTES (64u << 20)
int dckv_decode_noalloc(const dckv_plan* plan, const float* q, int32_t batch, const void* pool,
                        int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                        const int32_t* seq_lens, int32_t max_context, const void* R_keys,
                        const void* R_value, float* out, void* stream);

/* Benchmark instrumentation (not part of the method).  With two non-NULL
 * hipEvent_t handles, every later dckv_decode on this plan launches its
 * split-K attention kernel (the dominant kernel of a decode; for
 * dckv_decode_rope the key-rebuild kernel) with `before`
 * and `after` as the dispatch's own start and stop events
 * (hipExtLaunchKernel), so their interval is that kernel's execution alone;
 * NULL handles switch this off.  The
 * events stay owned by the caller.  A plan being instrumented must not be
 * used by several threads at once.  Makes no HIP call itself. */
int dckv_plan_set_profile_events(dckv_plan* plan, void* before, void* after);

/* ------------------------------------------------------------------------
 * Decode with rotary position embedding on the keys.  The paper never
 * mentions positional encodings; this is the reading for models that rotate
 * keys per position.  The factorisation of Sec. III-C is taken to be of the
 * key projection before the rotation, so the cache layout, the append and
 * the factors are those above.  The key of cache position t for query
 * head h is K_h[t] = Rot(t)(z_t R_{g,h}), and the query q_h is rotated to the
 * newest position, Rot(T_b - 1) q_h.  Rot(pos) turns each plane of
 * coordinates (i, i + d_h/2), i < d_h/2, by the angle
 * pos * rope_base^(-2i/d_h) (RoFormer's rotary embedding, rotate-half
 * pairing):
 *   x'_i = x_i cos - x_{i+d_h/2} sin,   x'_{i+d_h/2} = x_{i+d_h/2} cos + x_i sin.
 * Values are not rotated.  Softmax scale, head map and the rest are as for
 * dckv_decode.  A rotation that depends on t cannot be folded into the query
 * once, so each key is rebuilt per token (r_g * d_h MACs a token and KV head,
 * on MFMA), turned and dotted with the turned query.  Angles are reduced in
 * fp64 before the fp32 sine and cosine.
 *
 * Requirements: a bf16 plan on the MFMA path (geometry mfma_path == 1),
 * queries_per_seq 1, d_h 64 or 128, at most 8 query heads a KV head,
 * rope_base a finite number above 1.  Context splits are those of
 * dckv_decode capped at 1024 tokens.  Arguments, ownership, validation
 * (DCKV_EINVAL, DCKV_EALIGN, DCKV_EWORKSPACE, DCKV_EHIP; nothing enqueued on
 * error) and reproducibility as for dckv_decode (q and out [batch, H_q, d_h]
 * fp32), with a workspace of dckv_rope_workspace_bytes.  The workspace
 * also receives the factors R_g transposed into MFMA operand blocks, rebuilt
 * on every call.  With profile events set on the plan, the key-rebuild
 * kernel is the one stamped. */
int dckv_rope_workspace_bytes(const dckv_plan* plan, int32_t batch, int32_t max_context,
                              size_t* bytes);
int dckv_decode_rope(const dckv_plan* plan, const float* q, int32_t batch, const void* pool,
                     int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                     const int32_t* seq_lens, int32_t max_context, const void* R_keys,
                     const void* R_value, double rope_base, float* out, void* workspace,
                     size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Uncompressed baseline (no compression): decode over a paged bf16 K/V
 * cache with the same head map, scale and split-K scheme, so the compressed
 * path can be compared with the cache it replaces on the same harness.
 * Page of 64 tokens: keys [H_kv][64][d_h] then values [H_kv][64][d_h]; key
 * (slot s, KV head kv, column d) at (kv*64 + s)*d_h + d, the value at
 * 64*H_kv*d_h + (kv*64 + s)*d_h + d.  Supported: d_h in {64, 128, 256}, at
 * most 8 query heads a KV head.  split_tokens: a multiple of 64, or 0 to
 * choose from (batch, max_context). */
int dckv_dense_page_elems(int32_t num_kv_heads, int32_t head_dim, int64_t* elems);
int dckv_dense_workspace_bytes(int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                               int32_t split_tokens, int32_t batch, int32_t max_context,
                               size_t* bytes);
/* Arguments as for dckv_decode (q and out [batch, H_q, d_h] fp32, page_table,
 * seq_lens, max_context, workspace), plus: kv_pool, num_pages pages of the
 * layout above.  With two non-NULL hipEvent_t handles the split kernel is
 * launched with them as its dispatch's start and stop events (benchmark
 * instrumentation).  Validation, ownership and error behaviour as for
 * dckv_decode. */
int dckv_dense_decode(int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                      int32_t split_tokens, const float* q, int32_t batch, const void* kv_pool,
                      int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                      const int32_t* seq_lens, int32_t max_context, float* out, void* workspace,
                      size_t workspace_bytes, void* before_event, void* after_event,
                      void* stream);

/* ------------------------------------------------------------------------
 * Offline compression: run once per layer before serving, never on the
 * decode path.
 *
 * Gram matrix of samples (Sec. III-A: linear CKA compares centred
 * representations; Sec. III-D: the calibration Gram X^T X):
 *   G = A~^T A~, with A~ = A - 1 mu^T (mu: the column means) when center is
 *   nonzero, else A~ = A.
 *   A          device [rows, cols] row-major, dtype DCKV_F32 or DCKV_BF16,
 *              16-byte aligned; 1 <= rows <= 65535*256, cols a multiple of 8
 *              in [8, 32768]
 *   G          device [cols, cols] fp32, written in full (both triangles)
 *   workspace  device, at least dckv_gram_workspace_bytes (may be NULL
 *              when that is 0), 256-byte aligned
 * Products and sums are fp32 (MFMA f32) in a fixed order: bitwise
 * reproducible.  Errors: DCKV_EINVAL (shape, null pointer), DCKV_EDTYPE,
 * DCKV_EALIGN, DCKV_EWORKSPACE, DCKV_EHIP; nothing is launched on error. */
int dckv_gram_workspace_bytes(int64_t rows, int32_t cols, int32_t center, size_t* bytes);
int dckv_gram(const void* A, int32_t dtype, int64_t rows, int32_t cols, int32_t center, float* G,
              void* workspace, size_t workspace_bytes, void* stream);

/* Head similarity (Sec. III-C) from a centred Gram of the heads'
 * activations (columns h*d_h .. h*d_h + d_h - 1 belong to head h):
 *   S[i][j] = ||G_ij||_F^2 / (||G_ii||_F ||G_jj||_F), G_ij the d_h x d_h block
 *   of heads i and j -- the linear CKA of Sec. III-A; 0 where a head's block
 *   is zero.
 *   G device [h*d_h, h*d_h] fp32; S device [h, h] fp32 (out).
 * 1 <= h <= DCKV_MAX_HEADS, 1 <= d_h <= DCKV_MAX_HEAD_DIM.  Fixed-order sums. */
int dckv_head_similarity(const float* G, int32_t num_heads, int32_t head_dim, float* S,
                         void* stream);

/* Host: the whole merge sequence of Algorithm 1's head clustering
 * (ClusterHeads, Sec. III-C; the paper names agglomerative clustering):
 * average linkage on the distance 1 - S[i][j], h - 1 merges from h singleton
 * clusters down to one.  A cluster is named by its smallest head.  Merge s
 * joins clusters merge_a[s] < merge_b[s] (the merged cluster keeps the name
 * merge_a[s]) at linkage distance height[s]; on equal distances the pair
 * whose names are lexicographically smallest merges first.  Cutting the
 * sequence after h - K merges gives the K-group clustering of
 * dckv_cluster_heads, so one call serves every candidate K.
 *   S host [h][h] double (symmetric); merge_a, merge_b host [h - 1] (out);
 *   height host [h - 1] (out, may be NULL).
 * 1 <= h <= DCKV_MAX_HEADS.  Makes no HIP call. */
int dckv_cluster_merges(const double* S, int32_t num_heads, int32_t* merge_a, int32_t* merge_b,
                        double* height);

/* Host: Algorithm 1's head clustering (ClusterHeads, Sec. III-C):
 * agglomerative clustering into K groups with average linkage on the
 * distance 1 - S[i][j]; on equal distances the pair of clusters whose
 * smallest head ids are lexicographically smallest merges first.  Groups
 * are numbered in order of their smallest head.
 *   S host [h][h] double (symmetric); group_of_head host [h] (out).
 * 1 <= K <= h <= DCKV_MAX_HEADS.  Makes no HIP call. */
int dckv_cluster_heads(const double* S, int32_t num_heads, int32_t K, int32_t* group_of_head);

/* Host: Algorithm 1's rank allocation (InitRanksByEnergy then GreedyAdjust,
 * Sec. III-C) for K groups of a key projection with rank budget r:
 *   init_ranks[i] = floor(r * energy[i] / energy_total + 1/2), clipped to
 *   [1, rank_cap[i]]; then, while sum_i ranks[i]*heads[i] > 4 r (the budget
 *   sum_i r_i alpha_i <= 4 r / h) or sum_i ranks[i] > r, lower by one the
 *   rank with the smallest sigma_i[r_i - 1]^2 * h / heads[i] among ranks
 *   above 1 (equal costs: the lower group id); h = sum of heads.
 *   Since a group's costs grow as its rank falls, the lowering steps are
 *   taken in ascending (cost, group id) order across the groups.
 *   heads [K], energy [K] (||W_i||_F^2), rank_cap [K] (min(m, h_i d_h)),
 *   sigma [K][sigma_stride] (singular values of W_i, descending, at least
 *   rank_cap[i] of them) -- all host; init_ranks, ranks [K] host (out).
 * Makes no HIP call. */
int dckv_allocate_ranks(int32_t K, const int32_t* heads, const double* energy,
                        double energy_total, const double* sigma, int32_t sigma_stride,
                        const int32_t* rank_cap, int32_t r, int32_t* init_ranks, int32_t* ranks);

/* Message of the last failing call on this thread ("" if none). */
const char* dckv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DCKV_H */
