// Host side of the C ABI: validation, the plan's bookkeeping (Sec. III-C
// column-wise head groups with per-group ranks; Sec. III-D one value rank)
// and argument checks before any kernel is enqueued.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <new>
#include <string>

#include "internal.h"

namespace {

thread_local std::string g_last_error;

}  // namespace

namespace dckv {

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

}  // namespace dckv

using dckv::aligned;
using dckv::fail;

namespace dckv {

namespace {

// Places the rows of the groups, taken in the order `gorder`, into the J
// slices of `t` and records the key-chunk ranges of every 16-row tile.
// Returns false when some tile's chunks do not fit in two ranges.
bool place_rows(const dckv_plan& p, const std::vector<std::vector<int32_t>>& rows_of,
                const std::vector<int32_t>& gorder, int32_t J, int32_t per, MfmaTables& t,
                int32_t* total_chunks) {
  std::vector<int32_t> order;
  order.reserve(size_t(p.Q) * p.Hq);
  for (int32_t g : gorder) order.insert(order.end(), rows_of[g].begin(), rows_of[g].end());
  const int32_t nrows = int32_t(order.size());
  const int32_t nchunks = (p.RK + 31) / 32;
  int32_t max_pairs = 0, total = 0;
  std::vector<char> used(nchunks);
  for (int32_t s = 0; s < J; ++s) {
    const int32_t h0 = std::min(nrows, s * per), h1 = std::min(nrows, (s + 1) * per);
    t.slice_heads[s] = h1 - h0;
    for (int32_t i = 0; i < kSliceHeads; ++i) t.hord[s][i] = (h0 + i < h1) ? order[h0 + i] : -1;
    int32_t pairs = 0;
    for (int32_t n = 0; n < 2; ++n) {
      t.kst[s][n][0] = t.kst[s][n][1] = 0;
      t.kln[s][n][0] = t.kln[s][n][1] = 0;
      if (n >= t.nt) continue;
      std::fill(used.begin(), used.end(), 0);
      for (int32_t i = 16 * n; i < 16 * n + 16; ++i) {
        const int32_t row = t.hord[s][i];
        if (row < 0) continue;
        const int32_t g = p.group_of_kv[(row % p.Hq) / p.qpk];
        for (int32_t c = p.koff[g] / 32; c < (p.koff[g] + p.ranks[g] + 31) / 32; ++c) used[c] = 1;
      }
      int32_t nr = 0;
      for (int32_t c = 0; c < nchunks; ++c) {
        if (!used[c] || (c > 0 && used[c - 1])) continue;
        if (nr == 2) return false;
        int32_t e = c;
        while (e < nchunks && used[e]) ++e;
        t.kst[s][n][nr] = c;
        t.kln[s][n][nr] = e - c;
        ++nr;
      }
      pairs += t.kln[s][n][0] + t.kln[s][n][1];
    }
    max_pairs = std::max(max_pairs, pairs);
    total += pairs;
  }
  t.max_pairs = max_pairs;
  *total_chunks = total;
  return true;
}

// Items the slowest wave loads a page: key items padded to whole key blocks
// of `ring` loads (at least one block), then the value items padded to whole
// value blocks (12 or 16 loads, fixed by the value-tile capacity).
int32_t padded_items(const MfmaTables& t, int32_t ring) {
  const int32_t sw = std::min(4 * t.nt, t.waves), mpw = 4 * t.nt / sw;
  const int32_t vr = (2 * t.mtw_t) % 16 == 0 ? 16 : 12;
  int32_t nk_max = ring == vr ? 0 : ring;
  for (int32_t s = 0; s < t.n_slices; ++s)
    for (int32_t n = 0; n < t.nt; ++n) {
      const int32_t nk = (t.kln[s][n][0] + t.kln[s][n][1]) * mpw;
      nk_max = std::max(nk_max, (nk + ring - 1) / ring * ring);
    }
  return nk_max + (2 * t.mtw_t + vr - 1) / vr * vr;
}

}  // namespace

void build_mfma_tables(dckv_plan& p) {
  p.mfma_ok = false;
  p.mfma = MfmaTables{};
  if (p.dtype != DCKV_BF16) return;
  if (p.dh % 8 != 0) return;                   // the up-projection reads 8 columns at a time
  MfmaTables& t = p.mfma;
  const int32_t nrows = p.Q * p.Hq;
  int32_t J = p.head_slices > 0 ? p.head_slices : (nrows + kSliceHeads - 1) / kSliceHeads;
  t.mt_v = (p.rv + 15) / 16;
  // Eight waves (two a SIMD, so one wave's loads overlap the other's MFMAs)
  // whenever every wave gets at least one 16-rank value tile; four waves
  // for very small value ranks.  Accumulators take nt * mtw * 4 registers:
  // beyond 128 a lane, a default slicing takes twice the slices (16 rows a
  // slice), each slice then reading the value part on its own.
  t.waves = p.decode_waves ? p.decode_waves : (t.mt_v >= 8 ? 8 : 4);
  t.mtw = (t.mt_v + t.waves - 1) / t.waves;
  if (p.head_slices == 0) {
    while (J < kMaxSlices && J < nrows && ((nrows + J - 1) / J + 15) / 16 * t.mtw > 32) J *= 2;
    J = std::min(J, kMaxSlices);
  }
  if (J > kMaxSlices || J > nrows) return;
  const int32_t per = (nrows + J - 1) / J;
  if (per > kSliceHeads) return;
  t.n_slices = J;
  t.q_heads = p.Hq;
  t.queries = p.Q;
  t.nt = (per + 15) / 16;
  if (t.nt * t.mtw > 32) return;               // beyond 128 accumulator registers a lane
  t.mtw_t = 0;
  for (int32_t c : {6, 8, 12, 16, 32})
    if (t.mtw <= c && t.nt * c <= 32) {
      t.mtw_t = c;
      break;
    }
  if (t.mtw_t == 0) return;

  // Rows of each group in (head, query) order: row i * H_q + h.
  std::vector<std::vector<int32_t>> rows_of(p.G);
  for (int32_t h = 0; h < p.Hq; ++h)
    for (int32_t i = 0; i < p.Q; ++i) rows_of[p.group_of_kv[h / p.qpk]].push_back(i * p.Hq + h);

  // Group order and key block size: the slowest wave's padded items a page
  // first, then the key chunks loaded by all tiles (a group cut by a tile
  // boundary is loaded by both tiles); ties keep the earlier candidate, so
  // the group-id order and the longer block win.  Every order is tried for
  // up to seven groups; beyond that the group-id order alone.
  std::vector<int32_t> gorder(p.G);
  for (int32_t g = 0; g < p.G; ++g) gorder[g] = g;
  const bool search = p.G <= 7;
  MfmaTables cand = t, best = t;
  int32_t best_cost = -1, best_total = 0;
  do {
    int32_t total = 0;
    if (!place_rows(p, rows_of, gorder, J, per, cand, &total)) continue;
    for (int32_t ring : {16, 14, 12}) {
      // a key block longer or shorter than the value block costs registers:
      // only value-tile capacities up to 12 leave room for it
      if (t.mtw_t >= 16 && ring != 16) continue;
      const int32_t cost = padded_items(cand, ring);
      if (best_cost < 0 || cost < best_cost || (cost == best_cost && total < best_total)) {
        best = cand;
        best.ring = ring;
        best_cost = cost;
        best_total = total;
      }
    }
  } while (search && std::next_permutation(gorder.begin(), gorder.end()));
  if (best_cost < 0) return;                    // unreachable: the group-id order has one range a tile
  t = best;
  p.key_chunk_loads = best_total;
  const int64_t lds = int64_t(t.max_pairs) * 2048 + 32 * 72 * 2 + 2 * 8 * 32 * 4 + 256 * 4;
  if (lds > 160 * 1024) return;
  p.mfma_ok = true;
}

// Tables of the two-pass decode: the (query, head) rows in J = ceil(rows / 32)
// slices of one or two 16-row tiles (at most 8 slices), rows of a group
// together.  The score pass loads, a page, the key chunks of each tile's
// groups, so the group order is the one with the fewest chunk loads (every
// order for up to seven groups, else the group-id order; ties keep the
// earlier order).  Any value rank: the value pass takes 16-rank tiles in
// groups chosen per call.
void build_pass_tables(dckv_plan& p) {
  p.pass_ok = false;
  p.pass = MfmaTables{};
  p.pass_ring = 0;
  if (p.dtype != DCKV_BF16 || p.dh % 8 != 0) return;
  if (p.head_slices > 1 || p.decode_waves == 4) return;   // explicit single-pass shapes
  const int32_t nrows = p.Q * p.Hq;
  const int32_t J = (nrows + kSliceHeads - 1) / kSliceHeads;
  if (J > kMaxSlices) return;
  const int32_t per = (nrows + J - 1) / J;
  MfmaTables& t = p.pass;
  t.n_slices = J;
  t.q_heads = p.Hq;
  t.queries = p.Q;
  t.nt = (per + 15) / 16;
  t.mt_v = (p.rv + 15) / 16;
  t.waves = 8;
  std::vector<std::vector<int32_t>> rows_of(p.G);
  for (int32_t h = 0; h < p.Hq; ++h)
    for (int32_t i = 0; i < p.Q; ++i) rows_of[p.group_of_kv[h / p.qpk]].push_back(i * p.Hq + h);
  std::vector<int32_t> gorder(p.G);
  for (int32_t g = 0; g < p.G; ++g) gorder[g] = g;
  const bool search = p.G <= 7;
  MfmaTables cand = t, best = t;
  int32_t best_total = -1;
  do {
    int32_t total = 0;
    if (!place_rows(p, rows_of, gorder, J, per, cand, &total)) continue;
    if (best_total < 0 || total < best_total) {
      best = cand;
      best_total = total;
    }
  } while (search && std::next_permutation(gorder.begin(), gorder.end()));
  if (best_total < 0) return;
  t = best;
  p.pass_ring = 16;                            // score-pass loads in flight a wave
  if (pass_score_lds_bytes(p) > 160 * 1024 || pass_value_lds_bytes(p, 8) > 160 * 1024) return;
  p.pass_ok = true;
}

// Tables of the rotary decode: per KV head its group's key columns and
// factor block, the offset of its transposed factor blocks (one 16 x 32
// block per key chunk meeting the group's columns and per 16 rows of d_h),
// the heads in group order, and each query head's slot in the MFMA slices.
void build_rope_tables(dckv_plan& p) {
  p.rope = RopeTables{};
  p.rope_rt_elems = 0;
  if (!p.mfma_ok) return;
  RopeTables& r = p.rope;
  r.n_kv_heads = p.Hkv;
  r.head_dim = p.dh;
  r.q_per_kv = p.qpk;
  r.nh = 16 * p.mfma.nt;
  int32_t n = 0;
  for (int32_t g = 0; g < p.G; ++g)
    for (int32_t kv = 0; kv < p.Hkv; ++kv)
      if (p.group_of_kv[kv] == g) r.work_kv[n++] = kv;
  int64_t off = 0;
  for (int32_t kv = 0; kv < p.Hkv; ++kv) {
    const int32_t g = p.group_of_kv[kv];
    r.koff[kv] = p.koff[g];
    r.rank[kv] = p.ranks[g];
    r.rcol[kv] = p.pos_in_group[kv] * p.dh;
    r.rstride[kv] = p.hg[g] * p.dh;
    r.roff[kv] = p.roff[g];
    r.rt_off[kv] = int32_t(off);
    const int32_t nch = (p.koff[g] + p.ranks[g] - 1) / 32 - p.koff[g] / 32 + 1;
    off += int64_t(nch) * p.dh * 32;
  }
  p.rope_rt_elems = off;
  for (int32_t h = 0; h < DCKV_MAX_HEADS; ++h) r.qslot[h] = -1;
  for (int32_t sl = 0; sl < p.mfma.n_slices; ++sl)
    for (int32_t j2 = 0; j2 < kSliceHeads; ++j2) {
      const int32_t row = p.mfma.hord[sl][j2];
      if (row >= 0 && row < p.Hq) r.qslot[row] = sl * 32 + j2;   // query 0's rows
    }
}

// Host checks shared by the decode entry points: every argument except the
// workspace, then the launch shape.  Returns DCKV_OK with *shape set (for
// batch == 0 nothing else is checked), or a failure status.
int check_decode(const char* where, const dckv_plan* p, const float* q, int32_t batch,
                 const void* pool, int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                 const int32_t* seq_lens, int32_t max_context, const void* R_keys,
                 const void* R_value, const float* out, DecodeShape* shape) {
  if (!p) return fail(DCKV_EINVAL, "%s: null plan", where);
  if (batch < 0) return fail(DCKV_EINVAL, "%s: batch %d < 0", where, batch);
  if (batch == 0) return DCKV_OK;
  if (!q || !pool || !page_table || !seq_lens || !R_keys || !R_value || !out)
    return fail(DCKV_EINVAL, "%s: null device pointer", where);
  if (int64_t(batch) * p->Q > 65535)
    return fail(DCKV_EINVAL, "%s: batch %d x queries %d above 65535", where, batch, p->Q);
  if (num_pages < 1) return fail(DCKV_EINVAL, "%s: num_pages %lld < 1", where, (long long)num_pages);
  if (max_pages < 1) return fail(DCKV_EINVAL, "%s: max_pages %d < 1", where, max_pages);
  if (max_context < 0 || int64_t(max_context) > int64_t(max_pages) * DCKV_PAGE_TOKENS)
    return fail(DCKV_EINVAL, "%s: max_context %d outside [0, max_pages*64 = %lld]", where,
                max_context, (long long)max_pages * DCKV_PAGE_TOKENS);
  if (!aligned(q, 16) || !aligned(pool, 16) || !aligned(R_keys, 16) || !aligned(R_value, 16) ||
      !aligned(out, 16) || !aligned(page_table, 4) || !aligned(seq_lens, 4))
    return fail(DCKV_EALIGN, "%s: q, pool, R_keys, R_value and out must be 16-byte aligned", where);
  *shape = decode_shape(*p, batch, max_context);
  return DCKV_OK;
}

}  // namespace dckv

extern "C" {

const char* dckv_last_error(void) { return g_last_error.c_str(); }

int dckv_plan_create(const dckv_layer_desc* d, dckv_plan** out) {
  if (!d || !out) return fail(DCKV_EINVAL, "plan_create: null desc or out pointer");
  if (d->latent_dtype != DCKV_F32 && d->latent_dtype != DCKV_BF16)
    return fail(DCKV_EDTYPE, "plan_create: latent_dtype %d is neither DCKV_F32 nor DCKV_BF16",
                d->latent_dtype);
  if (d->hidden < 1) return fail(DCKV_EINVAL, "plan_create: hidden %d < 1", d->hidden);
  if (d->num_q_heads < 1 || d->num_q_heads > DCKV_MAX_HEADS)
    return fail(DCKV_EINVAL, "plan_create: num_q_heads %d outside [1,%d]", d->num_q_heads,
                DCKV_MAX_HEADS);
  if (d->num_kv_heads < 1 || d->num_q_heads % d->num_kv_heads != 0)
    return fail(DCKV_EINVAL, "plan_create: num_q_heads %d is not a multiple of num_kv_heads %d",
                d->num_q_heads, d->num_kv_heads);
  if (d->head_dim < 1 || d->head_dim > DCKV_MAX_HEAD_DIM)
    return fail(DCKV_EINVAL, "plan_create: head_dim %d outside [1,%d]", d->head_dim,
                DCKV_MAX_HEAD_DIM);
  if (d->num_groups < 1 || d->num_groups > DCKV_MAX_GROUPS || d->num_groups > d->num_kv_heads)
    return fail(DCKV_EINVAL, "plan_create: num_groups %d outside [1,min(%d,num_kv_heads)]",
                d->num_groups, DCKV_MAX_GROUPS);
  if (!d->group_of_kv_head || !d->group_rank)
    return fail(DCKV_EINVAL, "plan_create: null group_of_kv_head or group_rank");
  if (d->split_tokens < 0 || d->split_tokens % DCKV_PAGE_TOKENS != 0 || d->split_tokens > (1 << 24))
    return fail(DCKV_EINVAL, "plan_create: split_tokens %d is not 0 or a positive multiple of %d",
                d->split_tokens, DCKV_PAGE_TOKENS);
  if (d->decode_waves != 0 && d->decode_waves != 4 && d->decode_waves != 8)
    return fail(DCKV_EINVAL, "plan_create: decode_waves %d is not 0, 4 or 8", d->decode_waves);
  if (d->decode_passes < 0 || d->decode_passes > 2)
    return fail(DCKV_EINVAL, "plan_create: decode_passes %d is not 0, 1 or 2", d->decode_passes);
  if (d->head_slices < 0 || d->head_slices > DCKV_MAX_HEADS)
    return fail(DCKV_EINVAL, "plan_create: head_slices %d outside [0,%d]", d->head_slices,
                DCKV_MAX_HEADS);
  if (d->queries_per_seq < 0 || d->queries_per_seq > DCKV_MAX_QUERIES)
    return fail(DCKV_EINVAL, "plan_create: queries_per_seq %d outside [0,%d]",
                d->queries_per_seq, DCKV_MAX_QUERIES);

  const int32_t Hkv = d->num_kv_heads, G = d->num_groups, dh = d->head_dim;
  std::vector<int32_t> hg(G, 0), pos(Hkv, 0);
  for (int32_t kv = 0; kv < Hkv; ++kv) {
    const int32_t g = d->group_of_kv_head[kv];
    if (g < 0 || g >= G)
      return fail(DCKV_EINVAL, "plan_create: KV head %d assigned to group %d outside [0,%d)", kv, g, G);
    pos[kv] = hg[g]++;  // ascending head order inside the group
  }
  for (int32_t g = 0; g < G; ++g) {
    if (hg[g] == 0) return fail(DCKV_EINVAL, "plan_create: group %d has no heads", g);
    const int64_t cap = std::min<int64_t>(d->hidden, int64_t(hg[g]) * dh);
    const int32_t r = d->group_rank[g];
    if (r < 1 || r > cap || r > DCKV_MAX_GROUP_RANK)
      return fail(DCKV_EINVAL, "plan_create: rank %d of group %d outside [1,%lld] (limit %d)", r, g,
                  (long long)cap, DCKV_MAX_GROUP_RANK);
  }
  const int64_t vcap = std::min<int64_t>(d->hidden, int64_t(Hkv) * dh);
  if (d->value_rank < 1 || d->value_rank > vcap || d->value_rank > DCKV_MAX_VALUE_RANK)
    return fail(DCKV_EINVAL, "plan_create: value_rank %d outside [1,%lld] (limit %d)", d->value_rank,
                (long long)vcap, DCKV_MAX_VALUE_RANK);

  dckv_plan* p = new (std::nothrow) dckv_plan();
  if (!p) return fail(DCKV_ENOMEM, "plan_create: host allocation failed");
  try {
    p->m = d->hidden;
    p->Hq = d->num_q_heads;
    p->Hkv = Hkv;
    p->dh = dh;
    p->G = G;
    p->rv = d->value_rank;
    p->dtype = d->latent_dtype;
    p->split_tokens = d->split_tokens;
    p->head_slices = d->head_slices;
    p->decode_waves = d->decode_waves;
    p->decode_passes = d->decode_passes;
    p->Q = d->queries_per_seq > 0 ? d->queries_per_seq : 1;
    p->group_of_kv.assign(d->group_of_kv_head, d->group_of_kv_head + Hkv);
    p->ranks.assign(d->group_rank, d->group_rank + G);
    p->hg = hg;
    p->pos_in_group = pos;
    p->koff.resize(G);
    p->roff.resize(G + 1);
    int32_t acc = 0;
    int64_t racc = 0;
    for (int32_t g = 0; g < G; ++g) {
      p->koff[g] = acc;
      acc += p->ranks[g];
      p->roff[g] = racc;
      racc += int64_t(p->ranks[g]) * hg[g] * dh;
    }
    p->roff[G] = racc;
    p->RK = acc;
    p->RKp = (acc + 31) / 32 * 32;              // whole 32-column key chunks
    p->key_factor_elems = racc;
    p->rvp = (p->rv + 15) / 16 * 16;            // whole 16-column value tiles
    p->page_elems = int64_t(DCKV_PAGE_TOKENS) * p->RKp + int64_t(DCKV_PAGE_TOKENS) * p->rvp;
    p->value_base = int64_t(DCKV_PAGE_TOKENS) * p->RKp;
    p->qpk = p->Hq / Hkv;
    p->qoff.resize(p->Hq + 1);
    int32_t qacc = 0;
    dckv::HeadTables& t = p->tables;
    t = dckv::HeadTables{};
    t.n_q_heads = p->Hq;
    t.n_kv_heads = Hkv;
    t.head_dim = dh;
    t.q_per_kv = p->qpk;
    t.n_groups = G;
    t.n_queries = p->Q;
    for (int32_t h = 0; h < p->Hq; ++h) {
      const int32_t kv = h / p->qpk, g = p->group_of_kv[kv];
      p->qoff[h] = qacc;
      t.qoff[h] = qacc;
      t.rank_of_q[h] = p->ranks[g];
      t.koff_of_q[h] = p->koff[g];
      t.rcol_of_q[h] = pos[kv] * dh;
      t.rstride_of_q[h] = hg[g] * dh;
      t.roff_of_q[h] = p->roff[g];
      qacc += p->ranks[g];
    }
    p->qoff[p->Hq] = qacc;
    t.qoff[p->Hq] = qacc;
    t.qlen = qacc;
    p->qlen = qacc;
  } catch (...) {
    delete p;
    return fail(DCKV_ENOMEM, "plan_create: host allocation failed");
  }
  dckv::build_mfma_tables(*p);
  dckv::build_pass_tables(*p);
  dckv::build_rope_tables(*p);
  if (p->decode_passes == 2 && !p->pass_ok) {
    delete p;
    return fail(DCKV_EINVAL, "plan_create: decode_passes 2 needs bf16 latents, at most 256 (query, "
                "head) rows, d_h a multiple of 8 and no explicit head_slices or decode_waves 4");
  }
  if (p->decode_passes == 1) p->pass_ok = false;
  *out = p;
  return DCKV_OK;
}

void dckv_plan_destroy(dckv_plan* p) { delete p; }

int dckv_plan_set_profile_events(dckv_plan* p, void* before, void* after) {
  if (!p) return fail(DCKV_EINVAL, "plan_set_profile_events: null plan");
  if ((before == nullptr) != (after == nullptr))
    return fail(DCKV_EINVAL, "plan_set_profile_events: give both events or neither");
  p->prof_before = static_cast<hipEvent_t>(before);
  p->prof_after = static_cast<hipEvent_t>(after);
  return DCKV_OK;
}

int dckv_plan_info(const dckv_plan* p, dckv_plan_geometry* geo, int32_t* koff,
                   int32_t* pos_in_group, int32_t* qoff, int64_t* roff) {
  if (!p) return fail(DCKV_EINVAL, "plan_info: null plan");
  if (geo) {
    geo->key_rank_total = p->RK;
    geo->key_width_padded = p->RKp;
    geo->value_width_padded = p->rvp;
    geo->value_rank = p->rv;
    geo->q_per_kv = p->qpk;
    geo->folded_query_len = p->qlen;
    geo->split_tokens = p->split_tokens;
    geo->mfma_path = (p->mfma_ok || p->pass_ok) ? 1 : 0;
    geo->two_pass = p->pass_ok ? 1 : 0;
    geo->head_slices = p->mfma_ok ? p->mfma.n_slices : 0;
    geo->queries_per_seq = p->Q;
    geo->decode_waves = p->mfma_ok ? p->mfma.waves : 0;
    geo->decode_ring = p->mfma_ok ? p->mfma.ring : 0;
    geo->value_tiles_per_wave = p->mfma_ok ? p->mfma.mtw : 0;
    geo->key_chunk_loads = p->mfma_ok ? p->key_chunk_loads : 0;
    geo->page_elems = p->page_elems;
    geo->value_base = p->value_base;
    geo->key_factor_elems = p->key_factor_elems;
  }
  if (koff) std::copy(p->koff.begin(), p->koff.end(), koff);
  if (pos_in_group) std::copy(p->pos_in_group.begin(), p->pos_in_group.end(), pos_in_group);
  if (qoff) std::copy(p->qoff.begin(), p->qoff.end(), qoff);
  if (roff) std::copy(p->roff.begin(), p->roff.end(), roff);
  return DCKV_OK;
}

int dckv_decode_workspace_bytes(const dckv_plan* p, int32_t batch, int32_t max_context,
                                size_t* bytes) {
  if (!p || !bytes) return fail(DCKV_EINVAL, "decode_workspace_bytes: null plan or bytes pointer");
  if (batch < 0 || max_context < 0)
    return fail(DCKV_EINVAL, "decode_workspace_bytes: negative batch %d or max_context %d", batch,
                max_context);
  *bytes = dckv::decode_shape(*p, batch, max_context).bytes;
  return DCKV_OK;
}

int dckv_decode_launch_info(const dckv_plan* p, int32_t batch, int32_t max_context,
                            dckv_launch_info* info) {
  if (!p || !info) return fail(DCKV_EINVAL, "decode_launch_info: null plan or info pointer");
  if (batch < 0 || max_context < 0)
    return fail(DCKV_EINVAL, "decode_launch_info: negative batch %d or max_context %d", batch,
                max_context);
  const dckv::DecodeShape sh = dckv::decode_shape(*p, batch, max_context);
  info->kernels = sh.pass ? 2 : (sh.mfma ? 1 : 0);
  info->split_tokens = sh.split_tokens;
  info->n_split = sh.n_split;
  info->head_slices = sh.pass ? p->pass.n_slices : (sh.mfma ? p->mfma.n_slices : 1);
  info->value_tiles = sh.pass ? (p->pass.n_slices > 1 ? dckv::kSharedWaves * sh.rgt : sh.rgt) : 0;
  return DCKV_OK;
}

int dckv_latent_append(const dckv_plan* p, const void* x, int32_t n_tok, const void* L_keys,
                       const void* L_value, const int64_t* slot, void* pool, int64_t num_pages,
                       void* stream) {
  if (!p) return fail(DCKV_EINVAL, "latent_append: null plan");
  if (n_tok < 0) return fail(DCKV_EINVAL, "latent_append: n_tok %d < 0", n_tok);
  if (n_tok == 0) return DCKV_OK;
  if (!x || !L_keys || !L_value || !slot || !pool)
    return fail(DCKV_EINVAL, "latent_append: null device pointer");
  if (num_pages < 1) return fail(DCKV_EINVAL, "latent_append: num_pages %lld < 1", (long long)num_pages);
  if (n_tok > 64 * 65535) return fail(DCKV_EINVAL, "latent_append: n_tok %d above %d", n_tok, 64 * 65535);
  if (!aligned(x, 16) || !aligned(L_keys, 16) || !aligned(L_value, 16) || !aligned(pool, 16) ||
      !aligned(slot, 8))
    return fail(DCKV_EALIGN, "latent_append: x, L_keys, L_value and pool must be 16-byte aligned, slot 8-byte");
  hipError_t e = dckv::launch_append(*p, x, n_tok, L_keys, L_value, slot, pool, num_pages,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(DCKV_EHIP, "latent_append: %s", hipGetErrorString(e));
  return DCKV_OK;
}

int dckv_decode(const dckv_plan* p, const float* q, int32_t batch, const void* pool,
                int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                const int32_t* seq_lens, int32_t max_context, const void* R_keys,
                const void* R_value, float* out, void* workspace, size_t workspace_bytes,
                void* stream) {
  dckv::DecodeShape shape;
  int st = dckv::check_decode("decode", p, q, batch, pool, num_pages, page_table, max_pages,
                              seq_lens, max_context, R_keys, R_value, out, &shape);
  if (st != DCKV_OK || batch == 0) return st;
  if (!workspace) return fail(DCKV_EINVAL, "decode: null device pointer");
  if (!aligned(workspace, 256)) return fail(DCKV_EALIGN, "decode: workspace must be 256-byte aligned");
  if (workspace_bytes < shape.bytes)
    return fail(DCKV_EWORKSPACE, "decode: workspace of %zu bytes, %zu needed", workspace_bytes,
                shape.bytes);
  hipError_t e = dckv::launch_decode(*p, shape, q, pool, num_pages, page_table, max_pages, seq_lens,
                                     R_keys, R_value, out, workspace, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(DCKV_EHIP, "decode: %s", hipGetErrorString(e));
  return DCKV_OK;
}

// ------------------------------------------------ rotary decode
static int rope_check(const char* where, const dckv_plan* p) {
  if (!p) return fail(DCKV_EINVAL, "%s: null plan", where);
  if (!p->mfma_ok)
    return fail(DCKV_EINVAL, "%s: the rotary decode runs on the bf16 MFMA path, which this plan does not take", where);
  if (p->Q != 1) return fail(DCKV_EINVAL, "%s: one query a sequence (the plan has %d)", where, p->Q);
  if (p->dh != 64 && p->dh != 128) return fail(DCKV_EINVAL, "%s: head_dim %d is not 64 or 128", where, p->dh);
  if (p->qpk > dckv::rope_max_q_per_kv())
    return fail(DCKV_EINVAL, "%s: %d query heads a KV head (at most %d)", where, p->qpk, dckv::rope_max_q_per_kv());
  for (int32_t h = 0; h < p->Hq; ++h)   // every head owns a slot of the MFMA slices
    if (p->rope.qslot[h] < 0) return fail(DCKV_EINVAL, "%s: query head %d has no MFMA slot", where, h);
  return DCKV_OK;
}

int dckv_rope_workspace_bytes(const dckv_plan* p, int32_t batch, int32_t max_context, size_t* bytes) {
  int st = rope_check("rope_workspace_bytes", p);
  if (st != DCKV_OK) return st;
  if (!bytes) return fail(DCKV_EINVAL, "rope_workspace_bytes: null bytes pointer");
  if (batch < 0 || max_context < 0)
    return fail(DCKV_EINVAL, "rope_workspace_bytes: negative batch %d or max_context %d", batch, max_context);
  *bytes = dckv::rope_shape(*p, batch, max_context).bytes;
  return DCKV_OK;
}

int dckv_decode_rope(const dckv_plan* p, const float* q, int32_t batch, const void* pool,
                     int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                     const int32_t* seq_lens, int32_t max_context, const void* R_keys,
                     const void* R_value, double rope_base, float* out, void* workspace,
                     size_t workspace_bytes, void* stream) {
  int st = rope_check("decode_rope", p);
  if (st != DCKV_OK) return st;
  if (!(rope_base > 1.0) || !std::isfinite(rope_base))
    return fail(DCKV_EINVAL, "decode_rope: rope_base %g is not a finite number above 1", rope_base);
  if (batch < 0) return fail(DCKV_EINVAL, "decode_rope: batch %d < 0", batch);
  if (batch == 0) return DCKV_OK;
  if (!q || !pool || !page_table || !seq_lens || !R_keys || !R_value || !out || !workspace)
    return fail(DCKV_EINVAL, "decode_rope: null device pointer");
  if (batch > 65535) return fail(DCKV_EINVAL, "decode_rope: batch %d above 65535", batch);
  if (num_pages < 1) return fail(DCKV_EINVAL, "decode_rope: num_pages %lld < 1", (long long)num_pages);
  if (max_pages < 1) return fail(DCKV_EINVAL, "decode_rope: max_pages %d < 1", max_pages);
  if (max_context < 0 || int64_t(max_context) > int64_t(max_pages) * DCKV_PAGE_TOKENS)
    return fail(DCKV_EINVAL, "decode_rope: max_context %d outside [0, max_pages*64 = %lld]", max_context,
                (long long)max_pages * DCKV_PAGE_TOKENS);
  if (!aligned(q, 16) || !aligned(pool, 16) || !aligned(R_keys, 16) || !aligned(R_value, 16) ||
      !aligned(out, 16) || !aligned(page_table, 4) || !aligned(seq_lens, 4))
    return fail(DCKV_EALIGN, "decode_rope: q, pool, R_keys, R_value and out must be 16-byte aligned");
  if (!aligned(workspace, 256)) return fail(DCKV_EALIGN, "decode_rope: workspace must be 256-byte aligned");
  const dckv::DecodeShape shape = dckv::rope_shape(*p, batch, max_context);
  if (workspace_bytes < shape.bytes)
    return fail(DCKV_EWORKSPACE, "decode_rope: workspace of %zu bytes, %zu needed", workspace_bytes,
                shape.bytes);
  hipError_t e = dckv::launch_decode_rope(*p, shape, q, pool, num_pages, page_table, max_pages,
                                          seq_lens, R_keys, R_value, rope_base, out, workspace,
                                          static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(DCKV_EHIP, "decode_rope: %s", hipGetErrorString(e));
  return DCKV_OK;
}

// ------------------------------------------------ uncompressed baseline
static int dense_check(const char* where, int32_t Hq, int32_t Hkv, int32_t dh, int32_t split) {
  if (Hq < 1 || Hq > DCKV_MAX_HEADS || Hkv < 1 || Hq % Hkv != 0 || Hq / Hkv > 8)
    return fail(DCKV_EINVAL, "%s: %d query heads over %d KV heads (need a multiple, at most 8 a KV head, %d heads in all)",
                where, Hq, Hkv, DCKV_MAX_HEADS);
  if (dh != 64 && dh != 128 && dh != 256)
    return fail(DCKV_EINVAL, "%s: head_dim %d is not 64, 128 or 256", where, dh);
  if (split < 0 || split % DCKV_PAGE_TOKENS != 0 || split > (1 << 24))
    return fail(DCKV_EINVAL, "%s: split_tokens %d is not 0 or a positive multiple of %d", where, split,
                DCKV_PAGE_TOKENS);
  return DCKV_OK;
}

int dckv_dense_page_elems(int32_t num_kv_heads, int32_t head_dim, int64_t* elems) {
  if (!elems) return fail(DCKV_EINVAL, "dense_page_elems: null output pointer");
  if (num_kv_heads < 1 || num_kv_heads > DCKV_MAX_HEADS || head_dim < 1 || head_dim > DCKV_MAX_HEAD_DIM)
    return fail(DCKV_EINVAL, "dense_page_elems: %d KV heads of dimension %d", num_kv_heads, head_dim);
  *elems = int64_t(2) * DCKV_PAGE_TOKENS * num_kv_heads * head_dim;
  return DCKV_OK;
}

int dckv_dense_workspace_bytes(int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                               int32_t split_tokens, int32_t batch, int32_t max_context,
                               size_t* bytes) {
  if (!bytes) return fail(DCKV_EINVAL, "dense_workspace_bytes: null bytes pointer");
  int st = dense_check("dense_workspace_bytes", num_q_heads, num_kv_heads, head_dim, split_tokens);
  if (st != DCKV_OK) return st;
  if (batch < 0 || max_context < 0)
    return fail(DCKV_EINVAL, "dense_workspace_bytes: negative batch %d or max_context %d", batch,
                max_context);
  *bytes = dckv::dense_shape(num_q_heads, num_kv_heads, head_dim, batch, max_context, split_tokens).bytes;
  return DCKV_OK;
}

int dckv_dense_decode(int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                      int32_t split_tokens, const float* q, int32_t batch, const void* kv_pool,
                      int64_t num_pages, const int32_t* page_table, int32_t max_pages,
                      const int32_t* seq_lens, int32_t max_context, float* out, void* workspace,
                      size_t workspace_bytes, void* before_event, void* after_event,
                      void* stream) {
  int st = dense_check("dense_decode", num_q_heads, num_kv_heads, head_dim, split_tokens);
  if (st != DCKV_OK) return st;
  if (batch < 0) return fail(DCKV_EINVAL, "dense_decode: batch %d < 0", batch);
  if (batch == 0) return DCKV_OK;
  if (batch > 65535) return fail(DCKV_EINVAL, "dense_decode: batch %d above 65535", batch);
  if (!q || !kv_pool || !page_table || !seq_lens || !out || !workspace)
    return fail(DCKV_EINVAL, "dense_decode: null device pointer");
  if ((before_event == nullptr) != (after_event == nullptr))
    return fail(DCKV_EINVAL, "dense_decode: give both events or neither");
  if (num_pages < 1) return fail(DCKV_EINVAL, "dense_decode: num_pages %lld < 1", (long long)num_pages);
  if (max_pages < 1) return fail(DCKV_EINVAL, "dense_decode: max_pages %d < 1", max_pages);
  if (max_context < 0 || int64_t(max_context) > int64_t(max_pages) * DCKV_PAGE_TOKENS)
    return fail(DCKV_EINVAL, "dense_decode: max_context %d outside [0, max_pages*64 = %lld]",
                max_context, (long long)max_pages * DCKV_PAGE_TOKENS);
  if (!aligned(q, 16) || !aligned(kv_pool, 16) || !aligned(out, 16) || !aligned(page_table, 4) ||
      !aligned(seq_lens, 4))
    return fail(DCKV_EALIGN, "dense_decode: q, kv_pool and out must be 16-byte aligned");
  if (!aligned(workspace, 256)) return fail(DCKV_EALIGN, "dense_decode: workspace must be 256-byte aligned");
  const dckv::DenseShape sh =
      dckv::dense_shape(num_q_heads, num_kv_heads, head_dim, batch, max_context, split_tokens);
  if (workspace_bytes < sh.bytes)
    return fail(DCKV_EWORKSPACE, "dense_decode: workspace of %zu bytes, %zu needed", workspace_bytes,
                sh.bytes);
  hipError_t e = dckv::launch_dense_decode(sh, q, kv_pool, num_pages, page_table, max_pages,
                                           seq_lens, out, workspace,
                                           static_cast<hipEvent_t>(before_event),
                                           static_cast<hipEvent_t>(after_event),
                                           static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(DCKV_EHIP, "dense_decode: %s", hipGetErrorString(e));
  return DCKV_OK;
}

}  // extern "C"
