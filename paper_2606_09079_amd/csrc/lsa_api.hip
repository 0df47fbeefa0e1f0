// Host side of the C ABI declared in include/lsa.h: argument validation, the
// per-call plan (sequence table, launch geometry, workspace carve-up) and the
// stream-ordered launches.  No allocation, no synchronisation, no exceptions.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>

#include "lsa_internal.h"

namespace lsa {
namespace {

thread_local char g_err[512] = "";

lsa_status fail(lsa_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

lsa_status hip_fail(hipError_t e, const char* what) {
  return fail(LSA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Plan {
  SeqTable t;
  int64_t total_chunks = 0;
  int32_t max_keep = 0, max_sel = 0;
  int32_t group = 0, rows = 0, rows_pad = 16;
  int64_t chunk_stride = 0, head_stride = 0;
  int64_t n_units = 0;
  size_t emb_elem = 0;
  // two-level path: history chunks (before the window) per sequence, and the
  // pitch of the recalled list
  int32_t n_hist[LSA_MAX_BATCH] = {};
  int32_t rec_pitch = 0;
  // workspace layout (byte offsets)
  size_t off_scores = 0, off_sel = 0, off_cnt = 0, off_pq = 0, off_ml = 0, off_o = 0, off_arrive = 0;
  size_t off_rec = 0, off_rec_cnt = 0, off_nat = 0, off_nat_all = 0;
  size_t ws_total = 0;
};

// tl != NULL plans the two-level path: contexts may end inside a chunk, and
// the kept set of sequence b is at most min(core_keep, keep, history) chunks
// plus the window.
// partial: contexts may end inside a chunk (attention alone).
lsa_status make_plan(const lsa_problem* p, Plan* pl, const lsa_two_level* tl = nullptr, bool partial = false) {
  if (p == nullptr) return fail(LSA_ERR_INVALID_ARG, "problem is NULL");
  const int B = p->batch;
  if (B < 1 || B > LSA_MAX_BATCH) return fail(LSA_ERR_INVALID_ARG, "batch %d not in [1, %d]", B, LSA_MAX_BATCH);
  if (p->chunk_size != 64 && p->chunk_size != 128)
    return fail(LSA_ERR_UNSUPPORTED, "chunk_size %d not in {64, 128}", p->chunk_size);
  if (p->head_dim != kHeadDim) return fail(LSA_ERR_UNSUPPORTED, "head_dim %d != 128", p->head_dim);
  if (p->emb_dim != 64 && p->emb_dim != 128 && p->emb_dim != 256 && p->emb_dim != 512)
    return fail(LSA_ERR_UNSUPPORTED, "emb_dim %d not in {64, 128, 256, 512}", p->emb_dim);
  if (p->n_kv_heads < 1 || p->n_q_heads < 1 || p->n_q_heads % p->n_kv_heads != 0)
    return fail(LSA_ERR_INVALID_ARG, "n_q_heads %d must be a positive multiple of n_kv_heads %d", p->n_q_heads,
                p->n_kv_heads);
  if (p->n_kv_heads > 1024) return fail(LSA_ERR_UNSUPPORTED, "n_kv_heads %d > 1024", p->n_kv_heads);
  if (p->n_lookahead < 1 || p->n_lookahead > LSA_MAX_LOOKAHEAD)
    return fail(LSA_ERR_INVALID_ARG, "n_lookahead %d not in [1, %d]", p->n_lookahead, LSA_MAX_LOOKAHEAD);
  if (p->n_qtok < 1 || p->n_qtok > LSA_MAX_QTOK)
    return fail(LSA_ERR_INVALID_ARG, "n_qtok %d not in [1, %d]", p->n_qtok, LSA_MAX_QTOK);
  if (p->emb_dtype != LSA_F32 && p->emb_dtype != LSA_BF16 && p->emb_dtype != LSA_I8)
    return fail(LSA_ERR_INVALID_ARG, "emb_dtype %d is not an lsa_dtype", p->emb_dtype);
  if (p->reserved != 0) return fail(LSA_ERR_INVALID_ARG, "reserved field must be 0");
  if (p->ctx_tokens == nullptr || p->keep == nullptr)
    return fail(LSA_ERR_INVALID_ARG, "ctx_tokens and keep must be host arrays of batch entries");
  if (tl != nullptr) {
    if (tl->native_heads != 16 && tl->native_heads != 32 && tl->native_heads != 64)
      return fail(LSA_ERR_UNSUPPORTED, "native_heads %d not in {16, 32, 64}", tl->native_heads);
    if (tl->reserved != 0) return fail(LSA_ERR_INVALID_ARG, "two-level reserved field must be 0");
    if (tl->core_keep == nullptr || tl->window_tokens == nullptr)
      return fail(LSA_ERR_INVALID_ARG, "core_keep and window_tokens must be host arrays of batch entries");
    if (p->n_lookahead != 1)
      return fail(LSA_ERR_INVALID_ARG, "the two-level path takes one query token: n_lookahead %d != 1",
                  p->n_lookahead);
  }
  const int G = p->n_q_heads / p->n_kv_heads;
  const int rows = G * p->n_qtok;
  if (rows > LSA_MAX_ROWS)
    return fail(LSA_ERR_UNSUPPORTED, "n_qtok * n_q_heads / n_kv_heads = %d > %d", rows, LSA_MAX_ROWS);

  Plan& P = *pl;
  SeqTable& t = P.t;
  memset(&t, 0, sizeof t);
  t.batch = B;
  t.n_lookahead = p->n_lookahead;
  const int C = p->chunk_size;
  const int srows = score_rows_per_wg(p->emb_dtype, p->emb_dim, p->n_lookahead);
  P.group = G;
  P.rows = rows;
  P.rows_pad = (rows + 15) / 16 * 16;  // partial rows per unit: whole 16-row MFMA blocks
  // Kept-chunk bound of sequence b (0 when its shape is invalid; the second
  // pass reports that).
  auto kept_bound = [&](int b) -> int64_t {
    const int64_t L = p->ctx_tokens[b];
    if (tl == nullptr) {
      if (L < 1 || (!partial && (L < C || L % C != 0)) || p->keep[b] < 1) return 0;
      return std::min<int64_t>((int64_t)p->n_lookahead * p->keep[b], (L + C - 1) / C);
    }
    if (L < 1 || p->keep[b] < 1 || tl->core_keep[b] < 1 || tl->window_tokens[b] < 0) return 0;
    const int64_t n = (L + C - 1) / C, full = L / C;
    const int64_t w0 = std::min<int64_t>(std::max<int64_t>(L - tl->window_tokens[b], 0) / C, full);
    return std::min<int64_t>({(int64_t)tl->core_keep[b], (int64_t)p->keep[b], w0}) + (n - w0);
  };
  // First pass: the total kept-chunk bound, which sizes the splits.
  int64_t sel_total = 0;
  for (int b = 0; b < B; ++b) sel_total += kept_bound(b);
  const int tpc = C / 32;
  const int target = rows <= 16 && B <= kFewSequences ? kTargetWorkgroupsFew : kTargetWorkgroups;
  int64_t chunk_off = 0, wg_off = 0, swg_off = 0;
  for (int b = 0; b < B; ++b) {
    const int64_t L = p->ctx_tokens[b];
    if (tl == nullptr && !partial && (L < C || L % C != 0))
      return fail(LSA_ERR_INVALID_ARG, "ctx_tokens[%d] = %lld is not a positive multiple of chunk_size %d", b,
                  (long long)L, C);
    if (L < 1) return fail(LSA_ERR_INVALID_ARG, "ctx_tokens[%d] = %lld < 1", b, (long long)L);
    const int64_t n = (L + C - 1) / C;
    if (n > INT32_MAX / 2) return fail(LSA_ERR_UNSUPPORTED, "sequence %d has too many chunks", b);
    if (p->n_lookahead > 1 && n > LSA_MAX_UNION_CHUNKS)
      return fail(LSA_ERR_UNSUPPORTED, "sequence %d: %lld chunks > %d with several lookahead queries", b,
                  (long long)n, LSA_MAX_UNION_CHUNKS);
    const int32_t k = p->keep[b];
    if (k < 1 || (tl == nullptr && k > n))
      return fail(LSA_ERR_INVALID_ARG, "keep[%d] = %d not in [1, n_b = %lld]", b, k, (long long)n);
    if (tl != nullptr) {
      if (tl->core_keep[b] < 1) return fail(LSA_ERR_INVALID_ARG, "core_keep[%d] = %d < 1", b, tl->core_keep[b]);
      if (tl->window_tokens[b] < 0)
        return fail(LSA_ERR_INVALID_ARG, "window_tokens[%d] = %lld < 0", b, (long long)tl->window_tokens[b]);
      const int64_t w0 = std::min<int64_t>(std::max<int64_t>(L - tl->window_tokens[b], 0) / C, L / C);
      t.w0[b] = (int32_t)w0;
      t.win[b] = (int32_t)(n - w0);
      P.n_hist[b] = (int32_t)w0;
      P.rec_pitch = std::max<int32_t>(P.rec_pitch, (int32_t)std::min<int64_t>(k, w0));
    }
    t.tail[b] = (int32_t)(L - (n - 1) * C);
    const int32_t msel = (int32_t)kept_bound(b);
    // splits of sequence b in proportion to its share of the kept chunks, so the
    // whole grid is about `target`; at least one 32-token tile per split
    const double share = (double)target * (double)msel /
                         ((double)p->n_kv_heads * (double)std::max<int64_t>(sel_total, 1));
    const int32_t ns = (int32_t)std::max<int64_t>(
        1, std::min<int64_t>({std::llround(share), (int64_t)kMaxSplits, (int64_t)msel * tpc}));
    t.n[b] = (int32_t)n;
    t.keep[b] = k;
    t.nsplit[b] = ns;
    t.chunk_off[b] = chunk_off;
    t.wg_off[b] = (int32_t)wg_off;
    t.score_wg_off[b] = (int32_t)swg_off;
    chunk_off += n;
    wg_off += (int64_t)p->n_kv_heads * ns;
    swg_off += (n + srows - 1) / srows;
    P.max_keep = std::max(P.max_keep, k);
    P.max_sel = std::max(P.max_sel, msel);
    if (chunk_off > INT32_MAX || wg_off > INT32_MAX || swg_off > INT32_MAX)
      return fail(LSA_ERR_UNSUPPORTED, "problem too large for one launch");
  }
  t.chunk_off[B] = chunk_off;
  t.wg_off[B] = (int32_t)wg_off;
  t.score_wg_off[B] = (int32_t)swg_off;
  P.total_chunks = chunk_off;
  P.n_units = wg_off;

  // KV cache strides: blocks of C*d elements must not overlap.
  const int64_t blk = (int64_t)C * kHeadDim;
  P.head_stride = p->kv_head_stride ? p->kv_head_stride : blk;
  P.chunk_stride = p->kv_chunk_stride ? p->kv_chunk_stride : (int64_t)p->n_kv_heads * P.head_stride;
  if (P.head_stride < 0 || P.chunk_stride < 0 || P.head_stride % 8 || P.chunk_stride % 8)
    return fail(LSA_ERR_INVALID_ARG, "kv strides must be non-negative multiples of 8 elements");
  const bool chunk_major = P.head_stride >= blk && P.chunk_stride >= (int64_t)p->n_kv_heads * P.head_stride;
  const bool head_major = P.chunk_stride >= blk && P.head_stride >= P.total_chunks * P.chunk_stride;
  if (!chunk_major && !head_major)
    return fail(LSA_ERR_INVALID_ARG, "kv strides (chunk %lld, head %lld) make (chunk, head) blocks overlap",
                (long long)P.chunk_stride, (long long)P.head_stride);

  P.emb_elem = p->emb_dtype == LSA_F32 ? 4 : p->emb_dtype == LSA_BF16 ? 2 : 1;

  size_t off = 0;
  P.off_scores = off;
  off = align_up(off + (size_t)p->n_lookahead * P.total_chunks * 4);
  P.off_sel = off;
  off = align_up(off + (size_t)B * P.max_sel * 4);
  P.off_cnt = off;
  off = align_up(off + (size_t)B * 4);
  P.off_pq = off;
  if (p->n_lookahead > 1) off = align_up(off + (size_t)B * p->n_lookahead * P.max_keep * 4);
  P.off_ml = off;
  off = align_up(off + (size_t)P.n_units * P.rows_pad * 2 * 4);
  P.off_o = off;
  off = align_up(off + (size_t)P.n_units * P.rows_pad * kHeadDim * 4);
  if (tl != nullptr) {
    P.rec_pitch = std::max(P.rec_pitch, 1);
    P.off_rec = off;
    off = align_up(off + (size_t)B * P.rec_pitch * 4);
    P.off_rec_cnt = off;
    off = align_up(off + (size_t)B * 4);
    P.off_nat = off;
    off = align_up(off + (size_t)B * P.rec_pitch * 4);
    P.off_nat_all = off;  // native keys of every chunk (the fused selection)
    off = align_up(off + (size_t)P.total_chunks * 4);
  }
  P.off_arrive = off;  // split arrival counters of the fused step, one per (b, g)
  off = align_up(off + (size_t)B * p->n_kv_heads * 4);
  P.ws_total = off;
  return LSA_OK;
}

lsa_status check_ptr(const void* ptr, const char* name) {
  if (ptr == nullptr) return fail(LSA_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned16(ptr)) return fail(LSA_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return LSA_OK;
}

lsa_status check_ws(const Plan& P, void* ws, size_t ws_bytes) {
  if (ws_bytes < P.ws_total)
    return fail(LSA_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, P.ws_total);
  if (P.ws_total > 0 && ws == nullptr) return fail(LSA_ERR_WORKSPACE, "workspace is NULL");
  if (!aligned16(ws)) return fail(LSA_ERR_WORKSPACE, "workspace is not 16-byte aligned");
  return LSA_OK;
}

#define LSA_TRY(expr)                  \
  do {                                 \
    const lsa_status st_ = (expr);     \
    if (st_ != LSA_OK) return st_;     \
  } while (0)

#define LSA_HIP(expr, what)                      \
  do {                                           \
    const hipError_t e_ = (expr);                \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

uint8_t* at(void* ws, size_t off) { return static_cast<uint8_t*>(ws) + off; }

lsa_status run_topk(const lsa_problem* p, const Plan& P, bool keys_ready, const void* scores, int32_t* sel_idx,
                    int32_t* sel_count, int32_t* per_query_idx, void* ws, hipStream_t s) {
  if (p->n_lookahead == 1) {
    LSA_HIP(launch_topk(P.t, p->emb_dtype, keys_ready, scores, sel_idx, P.max_sel, 0, sel_count, s),
            "topk launch");
    return LSA_OK;
  }
  int32_t* pq = per_query_idx ? per_query_idx : reinterpret_cast<int32_t*>(at(ws, P.off_pq));
  LSA_HIP(launch_topk(P.t, p->emb_dtype, keys_ready, scores, pq, (int64_t)p->n_lookahead * P.max_keep,
                      P.max_keep, nullptr, s),
          "topk launch");
  LSA_HIP(launch_union(P.t, pq, P.max_keep, sel_idx, P.max_sel, sel_count, s), "union launch");
  return LSA_OK;
}

int max_splits(const Plan& P) {
  int ns_max = 0;
  for (int b = 0; b < P.t.batch; ++b) ns_max = std::max(ns_max, P.t.nsplit[b]);
  return ns_max;
}

// Whether the split kernel merges its own splits (its last workgroup of each
// (b, g)) when an earlier kernel of the call zeroes the arrival counters: only
// where that measured faster than the combine launch, i.e. the split kernel
// (at most 16 rows) on the one-workgroup-per-CU grid with at most kFewSplits
// splits.  The merge of 32 splits in one workgroup, and one more wait in each
// of two workgroups per CU, cost more than the launch.
bool merge_in_split(const Plan& P) {
  return P.rows <= kAttnRowsPerWave && P.t.batch <= kFewSequences && max_splits(P) <= kFewSplits;
}

// count_is_keep: sel_count[b] is known to be min(keep[b], n_b) (the top-k of a
// fused step with one query embedding wrote it).
lsa_status run_attn(const lsa_problem* p, const Plan& P, const uint16_t* q, const uint16_t* k,
                    const uint16_t* v, const int32_t* sel_idx, const int32_t* sel_count, float scale,
                    float* out, float* lse, void* ws, hipStream_t s, bool count_is_keep = false) {
  AttnArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.sel_idx = sel_idx;
  a.sel_count = sel_count;
  a.out = out;
  a.lse = lse;
  a.part_o = reinterpret_cast<float*>(at(ws, P.off_o));
  a.part_ml = reinterpret_cast<float*>(at(ws, P.off_ml));
  a.chunk_stride = P.chunk_stride;
  a.head_stride = P.head_stride;
  const double sc = scale > 0.f ? (double)scale : 1.0 / std::sqrt((double)kHeadDim);
  a.scale_log2e = (float)(sc * 1.4426950408889634);
  a.sel_pitch = P.max_sel;
  a.count_is_keep = count_is_keep ? 1 : 0;
  a.n_q_heads = p->n_q_heads;
  a.n_kv_heads = p->n_kv_heads;
  a.group = P.group;
  a.n_qtok = p->n_qtok;
  a.rows = P.rows;
  a.rows_pad = P.rows_pad;
  a.few_splits = max_splits(P) <= kFewSplits ? 1 : 0;
  a.arrive = P.t.arrive;  // set (and zeroed by the scoring kernel) only where merge_in_split(P)
  LSA_HIP(launch_attn(P.t, a, p->chunk_size, s), "attention launch");
  return LSA_OK;
}

lsa_status check_indexer(const lsa_problem* p, const lsa_indexer* ix) {
  if (ix == nullptr) return fail(LSA_ERR_INVALID_ARG, "indexer is NULL");
  if (ix->n_layers < 1 || ix->n_layers > LSA_MAX_IDX_LAYERS)
    return fail(LSA_ERR_INVALID_ARG, "indexer n_layers %d not in [1, %d]", ix->n_layers, LSA_MAX_IDX_LAYERS);
  if (ix->n_heads != 16 && ix->n_heads != 32 && ix->n_heads != 64)
    return fail(LSA_ERR_UNSUPPORTED, "indexer n_heads %d not in {16, 32, 64}", ix->n_heads);
  if (ix->key_dim != 64 && ix->key_dim != 128)
    return fail(LSA_ERR_UNSUPPORTED, "indexer key_dim %d not in {64, 128}", ix->key_dim);
  if (ix->reserved != 0) return fail(LSA_ERR_INVALID_ARG, "indexer reserved field must be 0");
  if (p->n_lookahead != 1)
    return fail(LSA_ERR_INVALID_ARG, "the recall path takes one query token: n_lookahead %d != 1", p->n_lookahead);
  return LSA_OK;
}

// The sequence table with scoring workgroups of kRecallRowsPerWg entries.
SeqTable recall_table(const Plan& P) {
  SeqTable t = P.t;
  int32_t off = 0;
  for (int b = 0; b < t.batch; ++b) {
    t.score_wg_off[b] = off;
    off += (t.n[b] + kRecallRowsPerWg - 1) / kRecallRowsPerWg;
  }
  t.score_wg_off[t.batch] = off;
  return t;
}

RecallArgs recall_args(const Plan& P, const lsa_indexer* ix, const void* idx_q, const float* idx_w,
                       const void* idx_k) {
  RecallArgs r;
  r.q = static_cast<const uint16_t*>(idx_q);
  r.w = idx_w;
  r.k = static_cast<const uint16_t*>(idx_k);
  r.total = P.total_chunks;
  r.layer_stride = P.total_chunks * ix->key_dim;
  r.n_layers = ix->n_layers;
  r.n_heads = ix->n_heads;
  r.key_dim = ix->key_dim;
  return r;
}

lsa_status check_recall_inputs(const void* idx_q, const float* idx_w, const void* idx_k) {
  LSA_TRY(check_ptr(idx_q, "idx_q"));
  LSA_TRY(check_ptr(idx_w, "idx_w"));
  LSA_TRY(check_ptr(idx_k, "idx_k"));
  return LSA_OK;
}

// The host tier's plans: P for the full context (its kept lists and copies),
// R for the reserve, a problem whose sequence b has slots[b] chunks, so that
// the attention over slot ids is the attention over chunk ids with the
// reserve as the cache.  Both have the same kept bound min(keep[b], n) =
// keep[b], hence the same split-K plan.
struct TierPlan {
  Plan P, R;
  int32_t slot_off[LSA_MAX_BATCH + 1] = {};
  int64_t total_slots = 0;
  size_t off_keys = 0;  // lsa_tier_step: native order keys of the resident recalled chunks, [B][pitch]
  size_t ws_total = 0;
};

lsa_status make_tier_plan(const lsa_problem* p, const lsa_tier* tr, TierPlan* tp) {
  LSA_TRY(make_plan(p, &tp->P));
  if (tr == nullptr) return fail(LSA_ERR_INVALID_ARG, "tier is NULL");
  if (tr->reserved != 0) return fail(LSA_ERR_INVALID_ARG, "tier reserved field must be 0");
  if (tr->fetch_workgroups < 0 || tr->fetch_workgroups > 1024)
    return fail(LSA_ERR_INVALID_ARG, "tier fetch_workgroups %d not in [0, 1024]", tr->fetch_workgroups);
  if (tr->slots == nullptr) return fail(LSA_ERR_INVALID_ARG, "tier slots must be a host array of batch entries");
  if (p->n_lookahead != 1)
    return fail(LSA_ERR_INVALID_ARG, "the host tier takes one query token: n_lookahead %d != 1", p->n_lookahead);
  const int B = p->batch;
  int64_t rctx[LSA_MAX_BATCH];
  int64_t off = 0;
  for (int b = 0; b < B; ++b) {
    const int32_t n = tp->P.t.n[b], k = p->keep[b], S = tr->slots[b];
    if (n > LSA_MAX_TIER_CHUNKS)
      return fail(LSA_ERR_UNSUPPORTED, "sequence %d: %d chunks > %d in the host tier", b, n, LSA_MAX_TIER_CHUNKS);
    if (S < 2 * (int64_t)k || S > LSA_MAX_TIER_SLOTS)
      return fail(LSA_ERR_INVALID_ARG, "slots[%d] = %d not in [2 * keep = %lld, %d]", b, S, 2 * (long long)k,
                  LSA_MAX_TIER_SLOTS);
    tp->slot_off[b] = (int32_t)off;
    off += S;
    rctx[b] = (int64_t)S * p->chunk_size;
  }
  tp->slot_off[B] = (int32_t)off;
  tp->total_slots = off;
  lsa_problem r = *p;
  r.ctx_tokens = rctx;
  r.kv_chunk_stride = 0;
  r.kv_head_stride = 0;
  LSA_TRY(make_plan(&r, &tp->R));
  if (tp->R.max_sel != tp->P.max_sel || tp->R.n_units != tp->P.n_units)
    return fail(LSA_ERR_INVALID_ARG, "reserve plan differs from the context plan");
  tp->off_keys = align_up(tp->R.ws_total);
  tp->ws_total = align_up(tp->off_keys + (size_t)B * tp->P.max_sel * 4);
  return LSA_OK;
}

// Device-visible addresses of the pinned host mirror; fails unless both ends
// of each mirror lie in one pinned allocation mapped for the device.
lsa_status mirror_device_ptrs(const lsa_problem* p, const Plan& P, const uint16_t* host_k, const uint16_t* host_v,
                              const uint16_t* dev[2]) {
  // last element of the mirror: the final block of the last chunk and head
  const int64_t last = (P.total_chunks - 1) * P.chunk_stride + (int64_t)(p->n_kv_heads - 1) * P.head_stride +
                       (int64_t)p->chunk_size * kHeadDim - 1;
  const uint16_t* host[2] = {host_k, host_v};
  for (int i = 0; i < 2; ++i) {
    void* d0 = nullptr;
    void* d1 = nullptr;
    if (hipHostGetDevicePointer(&d0, const_cast<uint16_t*>(host[i]), 0) != hipSuccess || d0 == nullptr ||
        hipHostGetDevicePointer(&d1, const_cast<uint16_t*>(host[i] + last), 0) != hipSuccess ||
        static_cast<uint16_t*>(d1) != static_cast<uint16_t*>(d0) + last) {
      (void)hipGetLastError();  // clear the error the failed lookup recorded
      return fail(LSA_ERR_INVALID_ARG, "%s is not pinned host memory mapped for the device over the whole mirror",
                  i ? "host_v" : "host_k");
    }
    dev[i] = static_cast<const uint16_t*>(d0);
  }
  return LSA_OK;
}

// The golden-label pipeline's geometry and workspace layout.
struct GoldenPlan {
  GoldenTable t;
  int64_t row_words = 0;    // words of all row bitmaps
  int64_t label_words = 0;  // words of the label bitmaps
  size_t off_bits = 0, off_labels = 0, ws_total = 0;
};

lsa_status make_golden_plan(const lsa_golden* g, GoldenPlan* gp) {
  if (g == nullptr) return fail(LSA_ERR_INVALID_ARG, "golden problem is NULL");
  if (g->batch < 1 || g->batch > LSA_MAX_BATCH)
    return fail(LSA_ERR_INVALID_ARG, "batch %d not in [1, %d]", g->batch, LSA_MAX_BATCH);
  if (g->n_steps < 1) return fail(LSA_ERR_INVALID_ARG, "n_steps %d < 1", g->n_steps);
  if (g->n_layers < 1 || g->n_layers > LSA_MAX_GOLDEN_LAYERS)
    return fail(LSA_ERR_INVALID_ARG, "n_layers %d not in [1, %d]", g->n_layers, LSA_MAX_GOLDEN_LAYERS);
  if (g->theta < 1 || g->theta > 64) return fail(LSA_ERR_INVALID_ARG, "theta %d not in [1, 64]", g->theta);
  if (g->p_num < 1 || g->p_den < g->p_num || g->p_den > (1 << 30))
    return fail(LSA_ERR_INVALID_ARG, "top-p %d / %d is not a fraction in (0, 1] with denominator <= 2^30",
                g->p_num, g->p_den);
  if (g->n_entries == nullptr) return fail(LSA_ERR_INVALID_ARG, "n_entries must be a host array of batch entries");
  if ((int64_t)g->batch * g->n_steps * g->n_layers > INT32_MAX)
    return fail(LSA_ERR_UNSUPPORTED, "too many rows for one launch");
  GoldenTable& t = gp->t;
  memset(&t, 0, sizeof t);
  t.batch = g->batch;
  const int64_t rows = (int64_t)g->n_steps * g->n_layers;
  int64_t entries = 0, bits = 0, labels = 0;
  for (int b = 0; b < g->batch; ++b) {
    const int64_t n = g->n_entries[b];
    if (n < 1 || n > LSA_MAX_GOLDEN_ENTRIES)
      return fail(LSA_ERR_INVALID_ARG, "n_entries[%d] = %lld not in [1, %d]", b, (long long)n,
                  LSA_MAX_GOLDEN_ENTRIES);
    t.n[b] = (int32_t)n;
    t.words[b] = (int32_t)((n + 31) / 32);
    t.entry_off[b] = entries;
    t.logit_off[b] = rows * entries;
    t.bit_off[b] = bits;
    t.label_word_off[b] = labels;
    entries += n;
    bits += rows * t.words[b];
    labels += t.words[b];
  }
  gp->row_words = bits;
  gp->label_words = labels;
  gp->off_bits = 0;
  gp->off_labels = align_up((size_t)bits * 4);
  gp->ws_total = align_up(gp->off_labels + (size_t)labels * 4);
  return LSA_OK;
}

// Scratch of lsa_decode_step_noalloc: one array per GPU, held until the
// process ends.  In host code `scratch` only names the symbol; its device
// address on each GPU comes from hipGetSymbolAddress with that GPU current.
__device__ __align__(256) uint8_t scratch[LSA_SCRATCH_BYTES];
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

lsa_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(LSA_ERR_UNSUPPORTED, "device %d: the scratch array serves devices 0 .. %d", dev,
                kMaxScratchDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (ptr == nullptr) return fail(LSA_ERR_HIP, "hipGetSymbolAddress(scratch) gave no address");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return LSA_OK;
}

}  // namespace
}  // namespace lsa

using namespace lsa;

extern "C" {

int lsa_abi_version(void) { return LSA_ABI_VERSION; }

const char* lsa_status_string(lsa_status st) {
  switch (st) {
    case LSA_OK: return "LSA_OK";
    case LSA_ERR_INVALID_ARG: return "LSA_ERR_INVALID_ARG";
    case LSA_ERR_UNSUPPORTED: return "LSA_ERR_UNSUPPORTED";
    case LSA_ERR_WORKSPACE: return "LSA_ERR_WORKSPACE";
    case LSA_ERR_HIP: return "LSA_ERR_HIP";
    default: return "LSA_ERR_UNKNOWN";
  }
}

const char* lsa_last_error(void) { return g_err; }

lsa_status lsa_validate(const lsa_problem* p) {
  Plan P;
  return make_plan(p, &P);
}

lsa_status lsa_max_sel(const lsa_problem* p, int32_t* max_sel) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  if (!max_sel) return fail(LSA_ERR_INVALID_ARG, "max_sel is NULL");
  *max_sel = P.max_sel;
  return LSA_OK;
}

lsa_status lsa_max_keep(const lsa_problem* p, int32_t* max_keep) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  if (!max_keep) return fail(LSA_ERR_INVALID_ARG, "max_keep is NULL");
  *max_keep = P.max_keep;
  return LSA_OK;
}

lsa_status lsa_workspace_size(const lsa_problem* p, size_t* bytes) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  if (!bytes) return fail(LSA_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = P.ws_total;
  return LSA_OK;
}

lsa_status lsa_workspace_init(void* ws, size_t ws_bytes, void* stream) {
  if (ws_bytes == 0) return LSA_OK;
  LSA_TRY(check_ptr(ws, "ws"));
  LSA_HIP(launch_zero(ws, ws_bytes, (hipStream_t)stream), "zero-fill launch");
  return LSA_OK;
}

lsa_status lsa_kv_pack(const lsa_problem* p, const uint16_t* k_tok, const uint16_t* v_tok,
                       const int64_t* token_offsets, int64_t tok_stride, int64_t tok_head_stride,
                       const int64_t* first_token, uint16_t* k_cache, uint16_t* v_cache, void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P, nullptr, /*partial=*/true));
  LSA_TRY(check_ptr(k_tok, "k_tok"));
  LSA_TRY(check_ptr(v_tok, "v_tok"));
  LSA_TRY(check_ptr(token_offsets, "token_offsets"));
  LSA_TRY(check_ptr(k_cache, "k_cache"));
  LSA_TRY(check_ptr(v_cache, "v_cache"));
  const int64_t hs = tok_head_stride ? tok_head_stride : kHeadDim;
  const int64_t ts = tok_stride ? tok_stride : (int64_t)p->n_kv_heads * hs;
  if (ts < 0 || hs < 0 || ts % 8 || hs % 8)
    return fail(LSA_ERR_INVALID_ARG, "token-major strides (token %lld, head %lld) must be non-negative multiples of 8",
                (long long)ts, (long long)hs);
  PackArgs a{};
  a.k_tok = k_tok;
  a.v_tok = v_tok;
  a.tok_off = token_offsets;
  a.tok_stride = ts;
  a.tok_head_stride = hs;
  a.k = k_cache;
  a.v = v_cache;
  a.chunk_stride = P.chunk_stride;
  a.head_stride = P.head_stride;
  a.n_kv_heads = p->n_kv_heads;
  a.chunk = p->chunk_size;
  a.batch = p->batch;
  const int64_t C = p->chunk_size;
  int64_t units = 0;
  for (int b = 0; b < p->batch; ++b) {
    const int64_t L = p->ctx_tokens[b], f = first_token ? first_token[b] : 0;
    if (f < 0 || f > L)
      return fail(LSA_ERR_INVALID_ARG, "first_token[%d] = %lld not in [0, ctx_tokens = %lld]", b, (long long)f,
                  (long long)L);
    a.first[b] = f;
    a.ctx[b] = L;
    a.chunk_off[b] = P.t.chunk_off[b];
    a.unit_off[b] = units;
    if (f < L) units += (L - 1) / C - f / C + 1;
  }
  a.unit_off[p->batch] = units;
  if (units * p->n_kv_heads > INT32_MAX)
    return fail(LSA_ERR_UNSUPPORTED, "%lld chunk blocks to write in one launch", (long long)(units * p->n_kv_heads));
  LSA_HIP(launch_kv_pack(a, units, (hipStream_t)stream), "kv pack launch");
  return LSA_OK;
}

lsa_status lsa_score_chunks(const lsa_problem* p, const void* query_emb, const void* chunk_emb, void* scores,
                            void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  LSA_TRY(check_ptr(query_emb, "query_emb"));
  LSA_TRY(check_ptr(chunk_emb, "chunk_emb"));
  LSA_TRY(check_ptr(scores, "scores"));
  LSA_HIP(launch_score(P.t, p->emb_dtype, p->emb_dim, query_emb, chunk_emb, scores, false, (hipStream_t)stream),
          "score launch");
  return LSA_OK;
}

lsa_status lsa_topk_chunks(const lsa_problem* p, const void* scores, int32_t* sel_idx, int32_t* sel_count,
                           int32_t* per_query_idx, void* ws, size_t ws_bytes, void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  LSA_TRY(check_ptr(scores, "scores"));
  LSA_TRY(check_ptr(sel_idx, "sel_idx"));
  LSA_TRY(check_ptr(sel_count, "sel_count"));
  if (per_query_idx != nullptr) LSA_TRY(check_ptr(per_query_idx, "per_query_idx"));
  if (p->n_lookahead > 1 && per_query_idx == nullptr) LSA_TRY(check_ws(P, ws, ws_bytes));
  return run_topk(p, P, false, scores, sel_idx, sel_count, per_query_idx, ws, (hipStream_t)stream);
}

lsa_status lsa_sparse_decode_attn(const lsa_problem* p, const uint16_t* q, const uint16_t* k_cache,
                                  const uint16_t* v_cache, const int32_t* sel_idx, const int32_t* sel_count,
                                  float softmax_scale, float* out, float* lse, void* ws, size_t ws_bytes,
                                  void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P, nullptr, true));
  LSA_TRY(check_ptr(q, "q"));
  LSA_TRY(check_ptr(k_cache, "k_cache"));
  LSA_TRY(check_ptr(v_cache, "v_cache"));
  LSA_TRY(check_ptr(sel_idx, "sel_idx"));
  LSA_TRY(check_ptr(sel_count, "sel_count"));
  LSA_TRY(check_ptr(out, "out"));
  if (lse != nullptr && (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(LSA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if (!std::isfinite(softmax_scale)) return fail(LSA_ERR_INVALID_ARG, "softmax_scale is not finite");
  LSA_TRY(check_ws(P, ws, ws_bytes));
  return run_attn(p, P, q, k_cache, v_cache, sel_idx, sel_count, softmax_scale, out, lse, ws,
                  (hipStream_t)stream);
}

lsa_status lsa_decode_step(const lsa_problem* p, const void* query_emb, const void* chunk_emb, const uint16_t* q,
                           const uint16_t* k_cache, const uint16_t* v_cache, float softmax_scale, float* out,
                           float* lse, int32_t* sel_idx, int32_t* sel_count, void* ws, size_t ws_bytes,
                           void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  LSA_TRY(check_ptr(query_emb, "query_emb"));
  LSA_TRY(check_ptr(chunk_emb, "chunk_emb"));
  LSA_TRY(check_ptr(q, "q"));
  LSA_TRY(check_ptr(k_cache, "k_cache"));
  LSA_TRY(check_ptr(v_cache, "v_cache"));
  LSA_TRY(check_ptr(out, "out"));
  if (lse != nullptr && (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(LSA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if ((sel_idx == nullptr) != (sel_count == nullptr))
    return fail(LSA_ERR_INVALID_ARG, "sel_idx and sel_count must both be given or both be NULL");
  if (sel_idx != nullptr) {
    LSA_TRY(check_ptr(sel_idx, "sel_idx"));
    LSA_TRY(check_ptr(sel_count, "sel_count"));
  }
  if (!std::isfinite(softmax_scale)) return fail(LSA_ERR_INVALID_ARG, "softmax_scale is not finite");
  LSA_TRY(check_ws(P, ws, ws_bytes));
  const hipStream_t s = (hipStream_t)stream;
  void* scores = at(ws, P.off_scores);
  int32_t* sel = sel_idx ? sel_idx : reinterpret_cast<int32_t*>(at(ws, P.off_sel));
  int32_t* cnt = sel_count ? sel_count : reinterpret_cast<int32_t*>(at(ws, P.off_cnt));
  // the scores stay in the workspace, so the scoring kernel writes them as
  // order keys and the selection reads them without converting; it also
  // zeroes the split arrival counters, so that the attention's last split
  // workgroup of each (b, g) merges the splits without a combine launch
  if (merge_in_split(P)) {
    P.t.arrive = reinterpret_cast<uint32_t*>(at(ws, P.off_arrive));
    P.t.n_arrive = p->batch * p->n_kv_heads;
  }
  LSA_HIP(launch_score(P.t, p->emb_dtype, p->emb_dim, query_emb, chunk_emb, scores, true, s), "score launch");
  LSA_TRY(run_topk(p, P, true, scores, sel, cnt, nullptr, ws, s));
  return run_attn(p, P, q, k_cache, v_cache, sel, cnt, softmax_scale, out, lse, ws, s, p->n_lookahead == 1);
}

lsa_status lsa_decode_step_noalloc(const lsa_problem* p, const void* query_emb, const void* chunk_emb,
                                   const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                   float softmax_scale, float* out, float* lse, int32_t* sel_idx,
                                   int32_t* sel_count, void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  if (P.ws_total > LSA_SCRATCH_BYTES)
    return fail(LSA_ERR_WORKSPACE, "the step needs %zu bytes of scratch; the allocation-free call has %zu", P.ws_total,
                (size_t)LSA_SCRATCH_BYTES);
  void* ws = nullptr;
  LSA_TRY(scratch_of_current_device(&ws));
  return lsa_decode_step(p, query_emb, chunk_emb, q, k_cache, v_cache, softmax_scale, out, lse, sel_idx, sel_count,
                         ws, LSA_SCRATCH_BYTES, stream);
}

lsa_status lsa_recall_scores(const lsa_problem* p, const lsa_indexer* ix, const void* idx_q, const float* idx_w,
                             const void* idx_k, float* scores, void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  LSA_TRY(check_indexer(p, ix));
  LSA_TRY(check_recall_inputs(idx_q, idx_w, idx_k));
  LSA_TRY(check_ptr(scores, "scores"));
  LSA_HIP(launch_recall_score(recall_table(P), recall_args(P, ix, idx_q, idx_w, idx_k), scores, false,
                              (hipStream_t)stream),
          "recall score launch");
  return LSA_OK;
}

lsa_status lsa_recall_select(const lsa_problem* p, const lsa_indexer* ix, const float* scores, int32_t* sel_idx,
                             int32_t* sel_count, void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  LSA_TRY(check_indexer(p, ix));
  LSA_TRY(check_ptr(scores, "scores"));
  LSA_TRY(check_ptr(sel_idx, "sel_idx"));
  LSA_TRY(check_ptr(sel_count, "sel_count"));
  SelectArgs sa;
  sa.recall = true;
  sa.n_layers = ix->n_layers;
  sa.layer_stride = P.total_chunks;
  LSA_HIP(launch_topk(P.t, LSA_F32, false, scores, sel_idx, P.max_sel, 0, sel_count, (hipStream_t)stream, sa),
          "recall select launch");
  return LSA_OK;
}

lsa_status lsa_recall_step(const lsa_problem* p, const lsa_indexer* ix, const void* idx_q, const float* idx_w,
                           const void* idx_k, const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                           float softmax_scale, float* out, float* lse, int32_t* sel_idx, int32_t* sel_count,
                           void* ws, size_t ws_bytes, void* stream) {
  Plan P;
  LSA_TRY(make_plan(p, &P));
  LSA_TRY(check_indexer(p, ix));
  LSA_TRY(check_recall_inputs(idx_q, idx_w, idx_k));
  LSA_TRY(check_ptr(q, "q"));
  LSA_TRY(check_ptr(k_cache, "k_cache"));
  LSA_TRY(check_ptr(v_cache, "v_cache"));
  LSA_TRY(check_ptr(out, "out"));
  if (lse != nullptr && (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(LSA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if ((sel_idx == nullptr) != (sel_count == nullptr))
    return fail(LSA_ERR_INVALID_ARG, "sel_idx and sel_count must both be given or both be NULL");
  if (sel_idx != nullptr) {
    LSA_TRY(check_ptr(sel_idx, "sel_idx"));
    LSA_TRY(check_ptr(sel_count, "sel_count"));
  }
  if (!std::isfinite(softmax_scale)) return fail(LSA_ERR_INVALID_ARG, "softmax_scale is not finite");
  LSA_TRY(check_ws(P, ws, ws_bytes));
  const hipStream_t s = (hipStream_t)stream;
  void* keys = at(ws, P.off_scores);  // n_lookahead == 1: one key per chunk
  int32_t* sel = sel_idx ? sel_idx : reinterpret_cast<int32_t*>(at(ws, P.off_sel));
  int32_t* cnt = sel_count ? sel_count : reinterpret_cast<int32_t*>(at(ws, P.off_cnt));
  // the scoring kernel writes the order key of max_l x_l, which the selection
  // reads as ready keys
  LSA_HIP(launch_recall_score(recall_table(P), recall_args(P, ix, idx_q, idx_w, idx_k), keys, true, s),
          "recall score launch");
  SelectArgs sa;
  sa.recall = true;
  LSA_HIP(launch_topk(P.t, LSA_F32, true, keys, sel, P.max_sel, 0, cnt, s, sa), "recall select launch");
  return run_attn(p, P, q, k_cache, v_cache, sel, cnt, softmax_scale, out, lse, ws, s);
}

lsa_status lsa_two_level_sizes(const lsa_problem* p, const lsa_two_level* tl, int32_t* max_sel,
                               size_t* ws_bytes) {
  if (tl == nullptr) return fail(LSA_ERR_INVALID_ARG, "two-level description is NULL");
  Plan P;
  LSA_TRY(make_plan(p, &P, tl));
  if (max_sel != nullptr) *max_sel = P.max_sel;
  if (ws_bytes != nullptr) *ws_bytes = P.ws_total;
  return LSA_OK;
}

lsa_status lsa_two_level_step(const lsa_problem* p, const lsa_indexer* ix, const lsa_two_level* tl,
                              const void* idx_q, const float* idx_w, const void* idx_k, const void* nat_q,
                              const float* nat_w, const void* nat_k, const uint16_t* q, const uint16_t* k_cache,
                              const uint16_t* v_cache, float softmax_scale, float* out, float* lse, int32_t* sel_idx,
                              int32_t* sel_count, void* ws, size_t ws_bytes, void* stream) {
  if (tl == nullptr) return fail(LSA_ERR_INVALID_ARG, "two-level description is NULL");
  Plan P;
  LSA_TRY(make_plan(p, &P, tl));
  LSA_TRY(check_indexer(p, ix));
  LSA_TRY(check_recall_inputs(idx_q, idx_w, idx_k));
  LSA_TRY(check_ptr(nat_q, "nat_q"));
  LSA_TRY(check_ptr(nat_w, "nat_w"));
  LSA_TRY(check_ptr(nat_k, "nat_k"));
  LSA_TRY(check_ptr(q, "q"));
  LSA_TRY(check_ptr(k_cache, "k_cache"));
  LSA_TRY(check_ptr(v_cache, "v_cache"));
  LSA_TRY(check_ptr(out, "out"));
  if (lse != nullptr && (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(LSA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if ((sel_idx == nullptr) != (sel_count == nullptr))
    return fail(LSA_ERR_INVALID_ARG, "sel_idx and sel_count must both be given or both be NULL");
  if (sel_idx != nullptr) {
    LSA_TRY(check_ptr(sel_idx, "sel_idx"));
    LSA_TRY(check_ptr(sel_count, "sel_count"));
  }
  if (!std::isfinite(softmax_scale)) return fail(LSA_ERR_INVALID_ARG, "softmax_scale is not finite");
  LSA_TRY(check_ws(P, ws, ws_bytes));
  const hipStream_t s = (hipStream_t)stream;
  const int B = p->batch;
  void* keys = at(ws, P.off_scores);
  int32_t* rec = reinterpret_cast<int32_t*>(at(ws, P.off_rec));
  int32_t* rec_cnt = reinterpret_cast<int32_t*>(at(ws, P.off_rec_cnt));
  uint32_t* nat = reinterpret_cast<uint32_t*>(at(ws, P.off_nat));
  int32_t* sel = sel_idx ? sel_idx : reinterpret_cast<int32_t*>(at(ws, P.off_sel));
  int32_t* cnt = sel_count ? sel_count : reinterpret_cast<int32_t*>(at(ws, P.off_cnt));

  // Level 1 over the history chunks: scores -> recalled ids (at most K_max)
  SeqTable th = P.t;
  for (int b = 0; b < B; ++b) th.n[b] = P.n_hist[b];
  SeqTable ths = th;
  {
    int32_t off = 0;
    for (int b = 0; b < B; ++b) {
      ths.score_wg_off[b] = off;
      off += (th.n[b] + kRecallRowsPerWg - 1) / kRecallRowsPerWg;
    }
    ths.score_wg_off[B] = off;
  }
  // Fused form: one scoring pass for both indexers (the native one as an extra
  // layer of the same head count), then both selections and the window in one
  // workgroup per sequence.
  int max_hist = 0;
  for (int b = 0; b < B; ++b) max_hist = std::max(max_hist, P.n_hist[b]);
  if (tl->native_heads == ix->n_heads && ix->n_layers + 1 <= kMaxIdxLayers &&
      (ix->n_layers + 1) * ix->n_heads <= kRecallThreads && max_hist <= kTwoLevelSelMaxN) {
    uint32_t* nat_all = reinterpret_cast<uint32_t*>(at(ws, P.off_nat_all));
    RecallArgs r = recall_args(P, ix, idx_q, idx_w, idx_k);
    r.nat_q = static_cast<const uint16_t*>(nat_q);
    r.nat_w = nat_w;
    r.nat_k = static_cast<const uint16_t*>(nat_k);
    r.nat_out = nat_all;
    LSA_HIP(launch_recall_score(ths, r, keys, true, s), "recall score launch");
    TwoLevelSelArgs a;
    a.l1 = static_cast<const uint32_t*>(keys);
    a.l2 = nat_all;
    a.out = sel;
    a.pitch = P.max_sel;
    a.count = cnt;
    for (int b = 0; b < B; ++b) a.keep2[b] = tl->core_keep[b];
    LSA_HIP(launch_two_level_select(th, a, s), "two-level select launch");
    return run_attn(p, P, q, k_cache, v_cache, sel, cnt, softmax_scale, out, lse, ws, s);
  }

  LSA_HIP(launch_recall_score(ths, recall_args(P, ix, idx_q, idx_w, idx_k), keys, true, s), "recall score launch");
  SelectArgs sa1;
  sa1.recall = true;
  LSA_HIP(launch_topk(th, LSA_F32, true, keys, rec, P.rec_pitch, 0, rec_cnt, s, sa1), "recall select launch");

  // Level 2: native scores of the recalled ids, then their top-k2 positions
  SeqTable tn = P.t;
  {
    int32_t off = 0;
    for (int b = 0; b < B; ++b) {
      tn.n[b] = std::min(p->keep[b], P.n_hist[b]);  // list capacity
      tn.score_wg_off[b] = off;
      off += (tn.n[b] + kRecallRowsPerWg - 1) / kRecallRowsPerWg;
    }
    tn.score_wg_off[B] = off;
  }
  RecallArgs rn;
  rn.q = static_cast<const uint16_t*>(nat_q);
  rn.w = nat_w;
  rn.k = static_cast<const uint16_t*>(nat_k);
  rn.total = P.total_chunks;
  rn.layer_stride = 0;
  rn.n_layers = 1;
  rn.n_heads = tl->native_heads;
  rn.key_dim = ix->key_dim;
  rn.list = rec;
  rn.list_count = rec_cnt;
  rn.list_pitch = P.rec_pitch;
  LSA_HIP(launch_recall_score(tn, rn, nat, true, s), "native score launch");
  // the compact [B][rec_pitch] native keys as sequences of capacity tn.n[b];
  // the selection writes the recalled ids it keeps, then the window chunks
  SeqTable tc = tn;
  for (int b = 0; b < B; ++b) {
    tc.keep[b] = tl->core_keep[b];
    tc.chunk_off[b] = (int64_t)b * P.rec_pitch;
  }
  SelectArgs sa2;
  sa2.dev_n = rec_cnt;
  sa2.map = rec;
  sa2.map_pitch = P.rec_pitch;
  LSA_HIP(launch_topk(tc, LSA_F32, true, nat, sel, P.max_sel, 0, cnt, s, sa2), "native top-k launch");
  return run_attn(p, P, q, k_cache, v_cache, sel, cnt, softmax_scale, out, lse, ws, s);
}

lsa_status lsa_tier_sizes(const lsa_problem* p, const lsa_tier* tr, int32_t* pitch, int64_t* total_slots,
                          size_t* ws_bytes) {
  TierPlan T;
  LSA_TRY(make_tier_plan(p, tr, &T));
  if (pitch != nullptr) *pitch = T.P.max_sel;
  if (total_slots != nullptr) *total_slots = T.total_slots;
  if (ws_bytes != nullptr) *ws_bytes = T.ws_total;
  return LSA_OK;
}

lsa_status lsa_tier_reset(const lsa_problem* p, const lsa_tier* tr, int32_t* owner, void* stream) {
  TierPlan T;
  LSA_TRY(make_tier_plan(p, tr, &T));
  LSA_TRY(check_ptr(owner, "owner"));
  LSA_HIP(launch_tier_reset(owner, T.total_slots, (hipStream_t)stream), "tier reset launch");
  return LSA_OK;
}

lsa_status lsa_tier_plan(const lsa_problem* p, const lsa_tier* tr, const int32_t* kept_idx,
                         const int32_t* kept_count, const int32_t* prev_slots, const int32_t* prev_count,
                         int32_t* owner, int32_t* slot_idx, int32_t* fetch, int32_t* fetch_count, void* stream) {
  TierPlan T;
  LSA_TRY(make_tier_plan(p, tr, &T));
  LSA_TRY(check_ptr(kept_idx, "kept_idx"));
  LSA_TRY(check_ptr(kept_count, "kept_count"));
  if ((prev_slots == nullptr) != (prev_count == nullptr))
    return fail(LSA_ERR_INVALID_ARG, "prev_slots and prev_count must both be given or both be NULL");
  if (prev_slots != nullptr) {
    LSA_TRY(check_ptr(prev_slots, "prev_slots"));
    LSA_TRY(check_ptr(prev_count, "prev_count"));
  }
  LSA_TRY(check_ptr(owner, "owner"));
  LSA_TRY(check_ptr(slot_idx, "slot_idx"));
  LSA_TRY(check_ptr(fetch, "fetch"));
  LSA_TRY(check_ptr(fetch_count, "fetch_count"));
  if (slot_idx == kept_idx || slot_idx == prev_slots)
    return fail(LSA_ERR_INVALID_ARG, "slot_idx must not alias kept_idx or prev_slots");
  TierArgs a;
  a.kept = kept_idx;
  a.kept_count = kept_count;
  a.prev_slots = prev_slots;
  a.prev_count = prev_count;
  a.owner = owner;
  a.slot_idx = slot_idx;
  a.fetch = fetch;
  a.fetch_count = fetch_count;
  a.pitch = T.P.max_sel;
  for (int b = 0; b < p->batch; ++b) a.slots[b] = tr->slots[b];
  memcpy(a.slot_off, T.slot_off, sizeof a.slot_off);
  LSA_HIP(launch_tier_plan(T.P.t, a, (hipStream_t)stream), "tier plan launch");
  return LSA_OK;
}

lsa_status lsa_tier_fetch(const lsa_problem* p, const lsa_tier* tr, const uint16_t* host_k,
                          const uint16_t* host_v, const int32_t* fetch, const int32_t* fetch_count,
                          uint16_t* res_k, uint16_t* res_v, void* stream) {
  TierPlan T;
  LSA_TRY(make_tier_plan(p, tr, &T));
  LSA_TRY(check_ptr(host_k, "host_k"));
  LSA_TRY(check_ptr(host_v, "host_v"));
  LSA_TRY(check_ptr(fetch, "fetch"));
  LSA_TRY(check_ptr(fetch_count, "fetch_count"));
  LSA_TRY(check_ptr(res_k, "res_k"));
  LSA_TRY(check_ptr(res_v, "res_v"));
  const uint16_t* dev[2] = {nullptr, nullptr};
  LSA_TRY(mirror_device_ptrs(p, T.P, host_k, host_v, dev));
  const Plan& P = T.P;
  TierFetchArgs a;
  a.host_k = dev[0];
  a.host_v = dev[1];
  a.res_k = res_k;
  a.res_v = res_v;
  a.fetch = fetch;
  a.fetch_count = fetch_count;
  a.chunk_stride = P.chunk_stride;
  a.head_stride = P.head_stride;
  a.res_slot_stride = (int64_t)p->n_kv_heads * p->chunk_size * kHeadDim;
  a.pitch = P.max_sel;
  a.n_kv_heads = p->n_kv_heads;
  for (int b = 0; b < p->batch; ++b) a.slots[b] = tr->slots[b];
  memcpy(a.slot_off, T.slot_off, sizeof a.slot_off);
  a.workgroups = tr->fetch_workgroups;
  LSA_HIP(launch_tier_fetch(P.t, a, p->chunk_size, (hipStream_t)stream), "tier fetch launch");
  return LSA_OK;
}

lsa_status lsa_tier_fetch_dma(const lsa_problem* p, const lsa_tier* tr, const uint16_t* host_k,
                              const uint16_t* host_v, const int32_t* h_fetch, const int32_t* h_fetch_count,
                              uint16_t* res_k, uint16_t* res_v, void* stream) {
  TierPlan T;
  LSA_TRY(make_tier_plan(p, tr, &T));
  LSA_TRY(check_ptr(host_k, "host_k"));
  LSA_TRY(check_ptr(host_v, "host_v"));
  LSA_TRY(check_ptr(res_k, "res_k"));
  LSA_TRY(check_ptr(res_v, "res_v"));
  if (h_fetch == nullptr || h_fetch_count == nullptr)
    return fail(LSA_ERR_INVALID_ARG, "h_fetch and h_fetch_count must be host arrays");
  const Plan& P = T.P;
  const int32_t pitch = P.max_sel;
  for (int b = 0; b < p->batch; ++b) {
    const int32_t nf = h_fetch_count[b];
    if (nf < 0 || nf > pitch)
      return fail(LSA_ERR_INVALID_ARG, "h_fetch_count[%d] = %d not in [0, %d]", b, nf, pitch);
    for (int f = 0; f < nf; ++f) {
      const int32_t c = h_fetch[((int64_t)b * pitch + f) * 2], s = h_fetch[((int64_t)b * pitch + f) * 2 + 1];
      if (c < 0 || c >= P.t.n[b] || s < 0 || s >= tr->slots[b])
        return fail(LSA_ERR_INVALID_ARG, "copy %d of sequence %d: chunk %d / slot %d out of range", f, b, c, s);
    }
  }
  const uint16_t* dev[2] = {nullptr, nullptr};
  LSA_TRY(mirror_device_ptrs(p, P, host_k, host_v, dev));
  const hipStream_t st = (hipStream_t)stream;
  const int64_t blk = (int64_t)p->chunk_size * kHeadDim;     // elements of one chunk-head block
  const int64_t slot = (int64_t)p->n_kv_heads * blk;          // elements of one reserve slot
  const bool packed = P.head_stride == blk && P.chunk_stride == slot;  // a chunk's heads adjacent in the mirror
  for (int b = 0; b < p->batch; ++b) {
    const int32_t* fl = h_fetch + (int64_t)b * pitch * 2;
    for (int f = 0; f < h_fetch_count[b];) {
      const int32_t c = fl[2 * f], s = fl[2 * f + 1];
      int r = 1;  // adjacent chunks into adjacent slots
      while (packed && f + r < h_fetch_count[b] && fl[2 * (f + r)] == c + r && fl[2 * (f + r) + 1] == s + r) ++r;
      for (int kv = 0; kv < 2; ++kv) {
        const uint16_t* src = (kv ? host_v : host_k) + (P.t.chunk_off[b] + c) * P.chunk_stride;
        uint16_t* dst = (kv ? res_v : res_k) + ((int64_t)T.slot_off[b] + s) * slot;
        if (packed) {
          LSA_HIP(hipMemcpyAsync(dst, src, (size_t)r * slot * 2, hipMemcpyHostToDevice, st), "tier DMA copy");
        } else {
          LSA_HIP(hipMemcpy2DAsync(dst, (size_t)blk * 2, src, (size_t)P.head_stride * 2, (size_t)blk * 2,
                                   (size_t)p->n_kv_heads, hipMemcpyHostToDevice, st),
                  "tier DMA copy");
        }
      }
      f += r;
    }
  }
  return LSA_OK;
}

lsa_status lsa_tier_step(const lsa_problem* p, const lsa_tier* tr, const lsa_indexer* nat, const int32_t* core_keep,
                         const void* nat_q, const float* nat_w, const void* nat_k, const int32_t* kept_idx,
                         const int32_t* kept_count, const int32_t* slot_idx, const uint16_t* q,
                         const uint16_t* res_k, const uint16_t* res_v, float softmax_scale, float* out, float* lse,
                         int32_t* sel_slots, int32_t* sel_count, void* ws, size_t ws_bytes, void* stream) {
  TierPlan T;
  LSA_TRY(make_tier_plan(p, tr, &T));
  LSA_TRY(check_indexer(p, nat));
  if (nat->n_layers != 1) return fail(LSA_ERR_INVALID_ARG, "native indexer n_layers %d != 1", nat->n_layers);
  if (core_keep == nullptr) return fail(LSA_ERR_INVALID_ARG, "core_keep must be a host array of batch entries");
  for (int b = 0; b < p->batch; ++b)
    if (core_keep[b] < 1) return fail(LSA_ERR_INVALID_ARG, "core_keep[%d] = %d < 1", b, core_keep[b]);
  LSA_TRY(check_ptr(nat_q, "nat_q"));
  LSA_TRY(check_ptr(nat_w, "nat_w"));
  LSA_TRY(check_ptr(nat_k, "nat_k"));
  LSA_TRY(check_ptr(kept_idx, "kept_idx"));
  LSA_TRY(check_ptr(kept_count, "kept_count"));
  LSA_TRY(check_ptr(slot_idx, "slot_idx"));
  LSA_TRY(check_ptr(q, "q"));
  LSA_TRY(check_ptr(res_k, "res_k"));
  LSA_TRY(check_ptr(res_v, "res_v"));
  LSA_TRY(check_ptr(out, "out"));
  LSA_TRY(check_ptr(sel_slots, "sel_slots"));
  LSA_TRY(check_ptr(sel_count, "sel_count"));
  if (sel_slots == slot_idx || sel_slots == kept_idx)
    return fail(LSA_ERR_INVALID_ARG, "sel_slots aliases kept_idx or slot_idx");
  if (lse != nullptr && (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(LSA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if (!std::isfinite(softmax_scale)) return fail(LSA_ERR_INVALID_ARG, "softmax_scale is not finite");
  if (ws_bytes < T.ws_total)
    return fail(LSA_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, T.ws_total);
  LSA_TRY(check_ws(T.R, ws, ws_bytes));
  const hipStream_t s = (hipStream_t)stream;
  const int B = p->batch;
  const int32_t pitch = T.P.max_sel;
  uint32_t* keys = reinterpret_cast<uint32_t*>(at(ws, T.off_keys));

  // native scores of the resident recalled chunks (list mode over kept_idx)
  SeqTable tn = T.P.t;
  {
    int32_t off = 0;
    for (int b = 0; b < B; ++b) {
      tn.n[b] = std::min(pitch, T.P.t.n[b]);  // list capacity
      tn.score_wg_off[b] = off;
      off += (tn.n[b] + kRecallRowsPerWg - 1) / kRecallRowsPerWg;
    }
    tn.score_wg_off[B] = off;
  }
  RecallArgs rn;
  rn.q = static_cast<const uint16_t*>(nat_q);
  rn.w = nat_w;
  rn.k = static_cast<const uint16_t*>(nat_k);
  rn.total = T.P.total_chunks;
  rn.layer_stride = 0;
  rn.n_layers = 1;
  rn.n_heads = nat->n_heads;
  rn.key_dim = nat->key_dim;
  rn.list = kept_idx;
  rn.list_count = kept_count;
  rn.list_pitch = pitch;
  LSA_HIP(launch_recall_score(tn, rn, keys, true, s), "native score launch");
  // the k2 largest of them, mapped to their reserve slots, in chunk order
  SeqTable tc = tn;
  for (int b = 0; b < B; ++b) {
    tc.keep[b] = core_keep[b];
    tc.chunk_off[b] = (int64_t)b * pitch;
    tc.win[b] = 0;
  }
  SelectArgs sa;
  sa.dev_n = kept_count;
  sa.map = slot_idx;
  sa.map_pitch = pitch;
  LSA_HIP(launch_topk(tc, LSA_F32, true, keys, sel_slots, pitch, 0, sel_count, s, sa), "native top-k launch");
  return run_attn(p, T.R, q, res_k, res_v, sel_slots, sel_count, softmax_scale, out, lse, ws, s);
}

lsa_status lsa_tier_attend(const lsa_problem* p, const lsa_tier* tr, const uint16_t* q, const uint16_t* res_k,
                           const uint16_t* res_v, const int32_t* slot_idx, const int32_t* slot_count,
                           float softmax_scale, float* out, float* lse, void* ws, size_t ws_bytes, void* stream) {
  TierPlan T;
  LSA_TRY(make_tier_plan(p, tr, &T));
  LSA_TRY(check_ptr(q, "q"));
  LSA_TRY(check_ptr(res_k, "res_k"));
  LSA_TRY(check_ptr(res_v, "res_v"));
  LSA_TRY(check_ptr(slot_idx, "slot_idx"));
  LSA_TRY(check_ptr(slot_count, "slot_count"));
  LSA_TRY(check_ptr(out, "out"));
  if (lse != nullptr && (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(LSA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if (!std::isfinite(softmax_scale)) return fail(LSA_ERR_INVALID_ARG, "softmax_scale is not finite");
  if (ws_bytes < T.ws_total)
    return fail(LSA_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, T.ws_total);
  LSA_TRY(check_ws(T.R, ws, ws_bytes));
  return run_attn(p, T.R, q, res_k, res_v, slot_idx, slot_count, softmax_scale, out, lse, ws, (hipStream_t)stream);
}

lsa_status lsa_golden_sizes(const lsa_golden* g, size_t* ws_bytes) {
  GoldenPlan G;
  LSA_TRY(make_golden_plan(g, &G));
  if (ws_bytes != nullptr) *ws_bytes = G.ws_total;
  return LSA_OK;
}

lsa_status lsa_golden_labels(const lsa_golden* g, const float* logits, int32_t* labels, int32_t* label_count,
                             int32_t* nucleus_size, int32_t* golden_count, void* ws, size_t ws_bytes, void* stream) {
  GoldenPlan G;
  LSA_TRY(make_golden_plan(g, &G));
  LSA_TRY(check_ptr(logits, "logits"));
  LSA_TRY(check_ptr(labels, "labels"));
  LSA_TRY(check_ptr(label_count, "label_count"));
  if (nucleus_size != nullptr) LSA_TRY(check_ptr(nucleus_size, "nucleus_size"));
  if (golden_count != nullptr) LSA_TRY(check_ptr(golden_count, "golden_count"));
  if (ws_bytes < G.ws_total)
    return fail(LSA_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, G.ws_total);
  if (ws == nullptr || !aligned16(ws)) return fail(LSA_ERR_WORKSPACE, "workspace is NULL or not 16-byte aligned");
  GoldenArgs a;
  a.logits = logits;
  a.bits = reinterpret_cast<uint32_t*>(at(ws, G.off_bits));
  a.nucleus_size = nucleus_size;
  a.p_num = g->p_num;
  a.p_den = g->p_den;
  a.tau = g->n_steps;
  a.layers = g->n_layers;
  a.theta = g->theta;
  LSA_HIP(launch_golden(G.t, a, reinterpret_cast<uint32_t*>(at(ws, G.off_labels)), G.label_words, labels,
                        label_count, golden_count, (hipStream_t)stream),
          "golden-label launch");
  return LSA_OK;
}

}  // extern "C"
