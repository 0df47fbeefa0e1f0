/*
 * lsa.h -- C ABI of the MI355X (gfx950) decode hot path of Lookahead Sparse
 * Attention (LSA).
 *
 * One decode step has three parts (paper Sec. 2.1):
 *   1. score   -- the Memory Indexer scores every compressed chunk of the context
 *                 against the query embedding (Eq. 4, taken as the dual-encoder
 *                 dot product s_c = qe . E_c of one indexer head with unit gate);
 *   2. select  -- keep the k highest-scoring chunks (the Top-k of Eq. 6,
 *                 with the recall bound K_max of Sec. 2.5 as the keep budget k);
 *                 with several lookahead query embeddings the kept set is the
 *                 union of the per-query top-k sets (set union as in Eq. 13);
 *   3. attend  -- softmax(q K^T * scale) V over the tokens of the kept chunks
 *                 only, gathered by chunk id from the full cache (the core
 *                 attention over the selected entries, Sec. 2.1).
 *
 * Conventions shared by every entry point
 *  - All device pointers are caller-owned HBM buffers, 16-byte aligned.  The
 *    library never allocates, frees or synchronises.  Every call is
 *    asynchronous on `stream` (a hipStream_t; NULL is the default stream);
 *    outputs are valid once the stream has reached the call.
 *  - Arguments are validated on the host before any launch; on failure the
 *    call returns a status, records a message for lsa_last_error() and writes
 *    nothing.  A failed launch returns LSA_ERR_HIP.  No C++ exception crosses
 *    the ABI.  Device contents (scores, chunk ids) are not validated: inputs
 *    must be finite and produced by the preceding steps.
 *  - Sequences are packed back to back.  Sequence b holds n_b = ctx_tokens[b] /
 *    chunk_size chunks (rounded up where the context may end inside a chunk,
 *    the last chunk then partial); its chunks have global ids chunk_off[b] ..
 *    chunk_off[b] + n_b - 1 where chunk_off is the exclusive prefix sum of n_b.
 *  - Chunk embeddings E: [sum_b n_b][emb_dim] row-major, row = global chunk id.
 *    Query embeddings: [batch][n_lookahead][emb_dim].
 *  - Scores: sequence b's block starts at element n_lookahead * chunk_off[b] and
 *    is [n_lookahead][n_b] row-major; float32 for F32/BF16 embeddings, int32
 *    (exact) for I8 embeddings.
 *  - Kept chunk ids: sel_idx [batch][max_sel] int32, per-sequence chunk ids in
 *    ascending order in the first sel_count[b] entries (sel_count is a device
 *    int32 [batch]); max_sel = max_b min(n_lookahead * keep[b], n_b).
 *  - KV cache (bf16, raw 16-bit patterns), paged by chunk.  The block of global
 *    chunk c and KV head g starts at element c * kv_chunk_stride + g *
 *    kv_head_stride and holds the chunk_size x 128 values of that chunk and
 *    head in MFMA operand order, so that every 1 KiB of the block is exactly
 *    what one wavefront load feeds to one v_mfma_f32_16x16x32_bf16.  Token t
 *    (0 <= t < chunk_size) and dimension e (0 <= e < 128) sit at element
 *        K block: ((((t/32*2 + t/4%2)*4 + e/32)*4 + e/8%4)*16 + t%32/8*4 + t%4)*8 + e%8
 *        V block: (((t/32*8 + e/16)*4 + t%32/8)*16 + e%16)*8 + t%8
 *    (integer division).  A serving system writes each new token's K and V
 *    rows into these positions once; every decode step then streams whole,
 *    contiguous 16 KiB (C = 64) or 32 KiB (C = 128) blocks.
 *  - q: bf16 [batch][n_qtok][n_q_heads][head_dim].  Query head h reads KV head
 *    h / (n_q_heads / n_kv_heads).  out: float32, same shape as q.  lse: float32
 *    [batch][n_qtok][n_q_heads], the natural-log log-sum-exp of the scaled
 *    logits over the kept tokens.
 *  - All n_qtok query tokens of a sequence attend the same kept set; there is
 *    no mask inside it.
 *
 * Recall path (lsa_recall_*): the paper's full Memory Indexer in place of
 * steps 1 and 2 -- a gated multi-head score per indexer layer (Eq. 4), the
 * sigmoid threshold 1/2 (Eq. 5), the OR over L indexer layers (Eq. 13) and
 * the bound K_max on the recalled set (Sec. 2.5) -- followed by step 3.
 *
 * Two-level path (lsa_two_level_*): that recall over the history before an
 * always-resident window (Level 1), the native indexer's top-k inside the
 * recalled set (Level 2, Eq. 6), and the window chunks added (Sec. 2.5); the
 * context may end inside a chunk, whose missing tokens get no weight.
 *
 * Host tier (lsa_tier_*): the decode-side offload of Sec. 2.5 -- the whole
 * cache stays in a pinned host mirror, each sequence has a GPU reserve of
 * chunk slots, a residency plan maps the recalled chunks to slots, the missing
 * ones are copied in from the mirror (a side-band step that can overlap
 * decode), and attention runs over the reserve.
 *
 * Golden labels (lsa_golden_*): the offline label pipeline of Sec. 2.2 over
 * raw indexer logits -- softmax, top-p set, votes across layers, golden set,
 * union over the look-ahead window.
 */
#ifndef LSA_H_
#define LSA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LSA_ABI_VERSION 1
#define LSA_MAX_BATCH 64           /* sequences per call */
#define LSA_MAX_LOOKAHEAD 16       /* query embeddings per sequence */
#define LSA_MAX_QTOK 16            /* attention query tokens per sequence */
#define LSA_MAX_ROWS 128           /* n_qtok * n_q_heads / n_kv_heads */
#define LSA_MAX_UNION_CHUNKS 262144 /* n_b limit when n_lookahead > 1 */
#define LSA_MAX_IDX_LAYERS 4       /* indexer layers OR-ed by the recall path */
#define LSA_MAX_TIER_CHUNKS 131072 /* n_b limit of the host tier's residency plan */
#define LSA_MAX_TIER_SLOTS 65536   /* reserve slots per sequence */
#define LSA_MAX_GOLDEN_ENTRIES 4194304 /* entries per sequence of the golden-label pipeline */
#define LSA_MAX_GOLDEN_LAYERS 63   /* layers voting in the golden-label pipeline */
#define LSA_SCRATCH_BYTES (64u << 20) /* device scratch of lsa_decode_step_noalloc, per GPU */

typedef enum {
  LSA_OK = 0,
  LSA_ERR_INVALID_ARG = 1, /* a shape, pointer, alignment or size is out of contract */
  LSA_ERR_UNSUPPORTED = 2, /* valid, but this build has no kernel for it */
  LSA_ERR_WORKSPACE = 3,   /* workspace missing or smaller than lsa_workspace_size() */
  LSA_ERR_HIP = 4          /* a HIP launch failed; see lsa_last_error() */
} lsa_status;

typedef enum { LSA_F32 = 0, LSA_BF16 = 1, LSA_I8 = 2 } lsa_dtype;

/* Shape of one decode step.  Host memory only; read during the call. */
typedef struct lsa_problem {
  int32_t batch;        /* B, 1 .. LSA_MAX_BATCH */
  int32_t chunk_size;   /* C, tokens per compressed chunk: 64 or 128 */
  int32_t n_q_heads;    /* Hq */
  int32_t n_kv_heads;   /* Hkv, divides Hq */
  int32_t head_dim;     /* d, 128 */
  int32_t emb_dim;      /* D, indexer embedding width: 64, 128, 256 or 512 */
  int32_t n_lookahead;  /* Q, query embeddings per sequence, 1 .. 16 */
  int32_t n_qtok;       /* Tq, attention query tokens per sequence, 1 .. 16 */
  int32_t emb_dtype;    /* lsa_dtype of E and of the query embeddings */
  int32_t reserved;     /* must be 0 */
  const int64_t* ctx_tokens; /* HOST [B]: context tokens of each sequence, a positive multiple of C
                                (lsa_sparse_decode_attn, lsa_two_level_step and lsa_kv_pack also take
                                any positive count: the last chunk may be partial) */
  const int32_t* keep;       /* HOST [B]: keep budget k_b, 1 <= k_b <= n_b (per query when Q > 1) */
  int64_t kv_chunk_stride;   /* elements between chunks in K and V; 0 selects n_kv_heads*C*d */
  int64_t kv_head_stride;    /* elements between KV heads in K and V; 0 selects C*d */
} lsa_problem;

/* Memory Indexer of the recall path.  Host memory only; read during the call. */
typedef struct lsa_indexer {
  int32_t n_layers;  /* L, indexer layers whose recalls are OR-ed, 1 .. LSA_MAX_IDX_LAYERS */
  int32_t n_heads;   /* n_h, indexer heads per layer: 16, 32 or 64 */
  int32_t key_dim;   /* c, width of the indexer queries and compressed index keys: 64 or 128 */
  int32_t reserved;  /* must be 0 */
} lsa_indexer;

/* Host tier.  Host memory only; read during the call. */
typedef struct lsa_tier {
  const int32_t* slots;  /* HOST [B]: reserve slots of sequence b, 2 * keep[b] .. LSA_MAX_TIER_SLOTS */
  int32_t reserved;      /* must be 0 */
  int32_t fetch_workgroups; /* workgroups of lsa_tier_fetch's copy kernel, 0 .. 1024; 0 selects 32, the
                               fastest copy (for a cold fill).  The copy reads the mirror through the memory
                               path a concurrent decode uses, and each copy workgroup slows that decode:
                               fewer move less per second but disturb it less. */
} lsa_tier;

/* Golden-label pipeline.  Host memory only; read during the call. */
typedef struct lsa_golden {
  int32_t batch;              /* B, 1 .. LSA_MAX_BATCH windows (one per sequence) */
  int32_t n_steps;            /* tau, decoding steps of a window, >= 1 */
  int32_t n_layers;           /* L, layers that vote, 1 .. LSA_MAX_GOLDEN_LAYERS */
  int32_t theta;              /* votes an entry needs, 1 .. 64 (above L no entry qualifies) */
  int32_t p_num, p_den;       /* top-p mass p = p_num / p_den, 1 <= p_num <= p_den <= 2^30 */
  const int64_t* n_entries;   /* HOST [B]: entries of each sequence, 1 .. LSA_MAX_GOLDEN_ENTRIES */
} lsa_golden;

/* Two-level selection.  Host memory only; read during the call. */
typedef struct lsa_two_level {
  int32_t native_heads;          /* heads of the native indexer of Level 2: 16, 32 or 64 (key width as the
                                    lsa_indexer's key_dim) */
  int32_t reserved;              /* must be 0 */
  const int32_t* core_keep;      /* HOST [B]: Level-2 budget k2_b >= 1 */
  const int64_t* window_tokens;  /* HOST [B]: always-resident context tail in tokens, >= 0 */
} lsa_two_level;

int lsa_abi_version(void);
const char* lsa_status_string(lsa_status status);
/* Message of the last failed call on this host thread ("" if none). */
const char* lsa_last_error(void);

/* Validate a problem without launching anything. */
lsa_status lsa_validate(const lsa_problem* p);
/* Row pitch of sel_idx: max_b min(Q * k_b, n_b). */
lsa_status lsa_max_sel(const lsa_problem* p, int32_t* max_sel);
/* Row pitch of the optional per-query lists of lsa_topk_chunks: max_b k_b. */
lsa_status lsa_max_keep(const lsa_problem* p, int32_t* max_keep);
/* Bytes of device workspace that any entry point below needs for p. */
lsa_status lsa_workspace_size(const lsa_problem* p, size_t* bytes);
/* Zero-fill a workspace on `stream` (a fill kernel, safe under graph capture).
 * Optional: no entry point needs a zeroed workspace; it only makes the
 * workspace contents deterministic before a first call. */
lsa_status lsa_workspace_init(void* ws, size_t ws_bytes, void* stream);

/*
 * Step 1 -- score every chunk (Sec. 2.1, Eq. 4 with one head and unit gate):
 *   scores[b][j][c] = sum_i query_emb[b][j][i] * E[chunk_off[b] + c][i]
 * float32 accumulation for F32/BF16 embeddings, exact int32 for I8.
 */
lsa_status lsa_score_chunks(const lsa_problem* p, const void* query_emb, const void* chunk_emb,
                            void* scores, void* stream);

/*
 * Step 2 -- keep the top-k chunks (Sec. 2.1, Eq. 6; union of Eq. 13):
 * for each (b, j) the k_b chunk ids with the largest score, ties broken towards
 * the lower chunk id, -0.0 equal to +0.0.  Q == 1: sel_idx[b][0..k_b) ascending
 * and sel_count[b] = k_b.  Q > 1: sel_idx[b] holds the ascending union of the Q
 * per-query sets and sel_count[b] its size.  per_query_idx (nullable) receives
 * each ascending per-query set, [B][Q][max_keep].  The workspace is used only
 * when Q > 1 and per_query_idx is NULL.
 */
lsa_status lsa_topk_chunks(const lsa_problem* p, const void* scores, int32_t* sel_idx,
                           int32_t* sel_count, int32_t* per_query_idx, void* ws, size_t ws_bytes,
                           void* stream);

/*
 * Step 3 -- sparse decode attention over the kept chunks (Sec. 2.1): for every
 * (b, t, h) with g = h / G, out = softmax(scale * q K_sel^T) V_sel over the
 * tokens of chunks sel_idx[b][0 .. sel_count[b]).  softmax_scale <= 0 selects
 * 1/sqrt(head_dim).  bf16 inputs, float32 softmax and accumulation.  lse is
 * nullable.  Split-K partials live in the workspace and are merged in a fixed
 * order, so results are bitwise reproducible.  Chunk ids must be < n_b and
 * sel_count[b] must be in 0 .. max_sel; an empty kept set (which only the
 * recall path produces) gives out = 0 and lse = -inf.  Unlike the other
 * entry points of steps 1 and 2 this one also takes a context that ends
 * inside a chunk (n_b = ceil(ctx_tokens[b] / chunk_size)); tokens past the
 * context end get no weight, and their K and V slots may hold any bits,
 * NaN included.
 */
lsa_status lsa_sparse_decode_attn(const lsa_problem* p, const uint16_t* q, const uint16_t* k_cache,
                                  const uint16_t* v_cache, const int32_t* sel_idx,
                                  const int32_t* sel_count, float softmax_scale, float* out,
                                  float* lse, void* ws, size_t ws_bytes, void* stream);

/*
 * Cache re-layout for callers whose K/V are token-major (the paged cache of
 * Sec. 2.1 and the KV layout of Sec. 2.5, one row per token): write the K and
 * V rows of tokens first_token[b] .. ctx_tokens[b] - 1 of every sequence b into
 * the chunk-paged, MFMA-ordered blocks that lsa_sparse_decode_attn and the
 * fused steps read (layout above, strides kv_chunk_stride / kv_head_stride of
 * p).  Once at prefill with first_token NULL (every token), then each step
 * for the tokens decoded since (first_token[b] = the old ctx_tokens[b]).
 *   k_tok, v_tok   bf16 source rows: token i of sequence b, KV head g starts at
 *                  element (token_offsets[b] + i) * tok_stride + g * tok_head_stride
 *                  and holds head_dim contiguous values.  tok_stride 0 selects
 *                  n_kv_heads * head_dim, tok_head_stride 0 selects head_dim
 *                  ([tokens][Hkv][d]); both non-negative multiples of 8.
 *   token_offsets  DEVICE int64 [B]: source row of token 0 of sequence b (a
 *                  [B + 1] prefix sum of the context lengths works as is; for a
 *                  buffer holding only the new rows it is the row of the first
 *                  new token minus first_token[b], which may be negative).
 *   first_token    HOST int64 [B], 0 <= first_token[b] <= ctx_tokens[b], or NULL
 *                  for 0.  Sequences with first_token[b] == ctx_tokens[b] are
 *                  left alone.
 * ctx_tokens may end inside a chunk: the positions of that block past the
 * context end are set to zero (a later call fills them).  No other position
 * changes; source rows must not overlap the caches.
 */
lsa_status lsa_kv_pack(const lsa_problem* p, const uint16_t* k_tok, const uint16_t* v_tok,
                       const int64_t* token_offsets, int64_t tok_stride, int64_t tok_head_stride,
                       const int64_t* first_token, uint16_t* k_cache, uint16_t* v_cache, void* stream);

/*
 * The whole step: score -> select -> attend on one stream with no host
 * synchronisation.  sel_idx / sel_count are nullable (then they live in the
 * workspace); when given they receive the kept chunk ids as lsa_topk_chunks
 * writes them.
 */
lsa_status lsa_decode_step(const lsa_problem* p, const void* query_emb, const void* chunk_emb,
                           const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                           float softmax_scale, float* out, float* lse, int32_t* sel_idx,
                           int32_t* sel_count, void* ws, size_t ws_bytes, void* stream);

/*
 * lsa_decode_step for callers that cannot allocate device memory (code under
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same step, with the same kernels and results, but no workspace argument.
 * Its scratch (scores, kept ids when sel_idx is NULL, split-K partials) lives
 * in one file-scope device array of LSA_SCRATCH_BYTES bytes, which every GPU
 * the library runs on holds until the process ends.  The call allocates and
 * frees nothing; on its first call on a device (the current one) it looks up
 * that device's address of the array.  A problem whose lsa_workspace_size
 * exceeds LSA_SCRATCH_BYTES returns LSA_ERR_WORKSPACE before any launch.
 * Every call on one GPU uses that GPU's one array: calls that overlap in time
 * on one GPU (other streams, other host threads) race, and the caller must
 * order them.  The array keeps the last call's contents; no call depends on
 * them.
 */
lsa_status lsa_decode_step_noalloc(const lsa_problem* p, const void* query_emb, const void* chunk_emb,
                                   const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                   float softmax_scale, float* out, float* lse, int32_t* sel_idx,
                                   int32_t* sel_count, void* stream);

/*
 * Recall path.  Shapes: the problem must have n_lookahead == 1 (one query token
 * fires the indexers) and keep[b] is the bound K_max of sequence b; emb_dim and
 * emb_dtype are not used.  Inputs, all device memory:
 *   idx_q  bf16 [B][L][n_h][c]        indexer queries q_{t,h} of every layer
 *   idx_w  float32 [B][L][n_h]        gate weights w_{t,h} of every layer
 *   idx_k  bf16 [L][sum_b n_b][c]     compressed index keys, row = global chunk id
 * R1 -- gated multi-head index score (Sec. 2.1, Eq. 4, the argument of the
 * sigmoid), float32 accumulation of exact bf16 products:
 *   scores[l][chunk_off[b] + s] = sum_h idx_w[b][l][h] * ReLU(idx_q[b][l][h] . idx_k[l][chunk_off[b] + s])
 */
lsa_status lsa_recall_scores(const lsa_problem* p, const lsa_indexer* ix, const void* idx_q, const float* idx_w,
                             const void* idx_k, float* scores, void* stream);

/*
 * R2 -- recall from scores as lsa_recall_scores writes them, float32
 * [L][sum_b n_b]: layer l recalls entry s when sigmoid(x) >= 1/2, i.e. x >= 0
 * (Eq. 5; -0.0 counts as 0), and s is recalled when any layer recalls it
 * (Eq. 13).  When more than keep[b] entries are recalled, the keep[b] with the
 * largest max_l x stay, ties towards the lower chunk id (K_max, Sec. 2.5).
 * sel_idx[b] receives the recalled ids in ascending order (row pitch
 * lsa_max_sel()) and sel_count[b] their number, 0 .. keep[b].  No workspace.
 */
lsa_status lsa_recall_select(const lsa_problem* p, const lsa_indexer* ix, const float* scores, int32_t* sel_idx,
                             int32_t* sel_count, void* stream);

/*
 * R1 -> R2 -> step 3 on one stream with no host synchronisation.  The scores
 * stay in the workspace; sel_idx / sel_count are nullable as in
 * lsa_decode_step.  Sequences with nothing recalled get out = 0, lse = -inf.
 */
lsa_status lsa_recall_step(const lsa_problem* p, const lsa_indexer* ix, const void* idx_q, const float* idx_w,
                           const void* idx_k, const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                           float softmax_scale, float* out, float* lse, int32_t* sel_idx, int32_t* sel_count,
                           void* ws, size_t ws_bytes, void* stream);

/*
 * Two-level path.  The problem must have n_lookahead == 1; ctx_tokens[b] may be
 * any positive count: sequence b has n_b = ceil(ctx_tokens[b] / chunk_size)
 * chunks (every chunk-indexed tensor counts them all), the last one possibly
 * partial.  keep[b] is the Level-1 bound K_max.  The window is the chunks
 * w0_b .. n_b - 1 with w0_b = min(floor(max(ctx - window_tokens, 0) / C),
 * floor(ctx / C)), so it always holds a partial last chunk; the history is
 * the complete chunks 0 .. w0_b - 1.  Per sequence:
 *   Level 1  recalled = the recall of lsa_recall_select over the history
 *            (idx_q, idx_w, idx_k as for lsa_recall_scores)
 *   Level 2  native[s] = sum_h nat_w[b][h] * ReLU(nat_q[b][h] . nat_k[chunk_off[b] + s])
 *            for the recalled s; the k2_b recalled chunks with the largest
 *            native score stay (all of them when there are at most k2_b;
 *            ties towards the lower id)
 *   kept     those chunks, ascending, then w0_b .. n_b - 1
 * then step 3 over the kept chunks; tokens past ctx_tokens[b] in the last
 * chunk get no weight.  Layouts: nat_q bf16 [B][native_heads][key_dim],
 * nat_w float32 [B][native_heads], nat_k bf16 [sum_b n_b][key_dim].
 */
/* Row pitch of sel_idx and the workspace size of lsa_two_level_step (either
 * output pointer may be NULL). */
lsa_status lsa_two_level_sizes(const lsa_problem* p, const lsa_two_level* tl, int32_t* max_sel,
                               size_t* ws_bytes);
lsa_status lsa_two_level_step(const lsa_problem* p, const lsa_indexer* ix, const lsa_two_level* tl,
                              const void* idx_q, const float* idx_w, const void* idx_k, const void* nat_q,
                              const float* nat_w, const void* nat_k, const uint16_t* q, const uint16_t* k_cache,
                              const uint16_t* v_cache, float softmax_scale, float* out, float* lse, int32_t* sel_idx,
                              int32_t* sel_count, void* ws, size_t ws_bytes, void* stream);

/*
 * Host tier (Sec. 2.5, decode-side offload and asynchronous recall).  The
 * problem is the one of the full context (ctx_tokens[b] a multiple of
 * chunk_size, n_b <= LSA_MAX_TIER_CHUNKS, n_lookahead == 1) with keep[b] the
 * bound K_max on the kept set.  Sequence b owns slots[b] reserve slots; slot
 * ids are local to the sequence and reserve slot s of sequence b is global
 * slot slot_off[b] + s, slot_off the exclusive prefix sum of slots.
 *   owner    device int32 [sum_b slots[b]]: the chunk id each slot holds, -1
 *            when it holds none (the residency table; the library keeps it up
 *            to date, the caller allocates it and resets it once)
 *   res_k, res_v   device bf16 reserve, [sum_b slots[b]][n_kv_heads][C x 128]:
 *            global slot j and KV head g start at element (j * n_kv_heads + g)
 *            * C * 128 and hold that chunk-head block exactly as the cache
 *            stores it (the MFMA operand order above)
 *   host_k, host_v  the mirror: pinned host memory (hipHostMalloc, or a pinned
 *            torch tensor) laid out as the cache, with the problem's strides
 * Kept lists, slot lists and copy lists are [B][pitch] with pitch = lsa_max_sel()
 * (copy lists [B][pitch][2] of (chunk id, local slot id)).
 */
/* Pitch of the lists, slots in the reserve, and the workspace of
 * lsa_tier_attend and lsa_tier_step (any output pointer may be NULL). */
lsa_status lsa_tier_sizes(const lsa_problem* p, const lsa_tier* tr, int32_t* pitch, int64_t* total_slots,
                          size_t* ws_bytes);
/* owner[0 .. sum_b slots[b]) = -1: an empty reserve (a fill kernel on stream). */
lsa_status lsa_tier_reset(const lsa_problem* p, const lsa_tier* tr, int32_t* owner, void* stream);
/*
 * Residency plan of one firing.  kept_idx[b][0 .. kept_count[b]) are distinct
 * chunk ids < n_b in ascending order (as the selections write them);
 * prev_slots[b][0 .. prev_count[b]) are the slots the previous kept set reads
 * (the previous call's slot_idx; both NULL at the first firing).  Per sequence:
 *  - a kept chunk that a slot already holds keeps that slot;
 *  - the other kept chunks, in ascending order, take the free slots in
 *    ascending order, a free slot being one that holds no kept chunk and that
 *    the previous set does not read (so decode may go on reading the previous
 *    set until the copies are done);
 *  - slot_idx[b][i] = slot of kept_idx[b][i]; fetch[b][f] = (chunk, slot) for
 *    f < fetch_count[b], ascending in both; owner is updated.
 * slots[b] >= 2 * keep[b] guarantees enough free slots.  Should that fail
 * anyway, fetch_count[b] = -1 and owner is left as it was.  A kept id
 * outside 0 .. n_b - 1 gets slot -1 and no copy.
 */
lsa_status lsa_tier_plan(const lsa_problem* p, const lsa_tier* tr, const int32_t* kept_idx,
                         const int32_t* kept_count, const int32_t* prev_slots, const int32_t* prev_count,
                         int32_t* owner, int32_t* slot_idx, int32_t* fetch, int32_t* fetch_count, void* stream);
/*
 * Copy the chunks of a plan's copy list from the mirror into the reserve: for
 * f < fetch_count[b], the K and V blocks of every KV head of chunk fetch[b][f][0]
 * into slot fetch[b][f][1].  The GPU reads the mirror over PCIe (no host
 * synchronisation; the copy list stays on the device).  LSA_ERR_INVALID_ARG
 * when host_k or host_v is not pinned, device-visible host memory.
 */
lsa_status lsa_tier_fetch(const lsa_problem* p, const lsa_tier* tr, const uint16_t* host_k,
                          const uint16_t* host_v, const int32_t* fetch, const int32_t* fetch_count,
                          uint16_t* res_k, uint16_t* res_v, void* stream);
/*
 * The copies of lsa_tier_fetch made by the GPU's DMA engines and issued from
 * the host: h_fetch [B][pitch][2] and h_fetch_count [B] are HOST copies of a
 * plan's copy list (the caller brings them over once the plan has run, in a
 * side band off the decode path).  One asynchronous host-to-device copy per
 * chunk and K/V (per chunk and KV head plane for a mirror whose heads of a
 * chunk are not adjacent), copies of adjacent chunks into adjacent slots
 * merged.  The DMA engines take no compute units, so a decode running at the
 * same time is hardly slowed, but they move fewer bytes per second than
 * lsa_tier_fetch.  Every entry is validated before the first copy is issued
 * (chunk < n_b, slot < slots[b], 0 <= count <= pitch); a copy that fails to
 * issue returns LSA_ERR_HIP with the earlier copies already queued.
 */
lsa_status lsa_tier_fetch_dma(const lsa_problem* p, const lsa_tier* tr, const uint16_t* host_k,
                              const uint16_t* host_v, const int32_t* h_fetch, const int32_t* h_fetch_count,
                              uint16_t* res_k, uint16_t* res_v, void* stream);
/*
 * One decode step over the resident set (Sec. 2.5, the fixed-shape part that
 * runs every step between firings): Level 2 of the two-level selection
 * (Sec. 2.1 after Eq. 5, Eq. 6) over the chunks that the last firing made
 * resident, then step 3 over their reserve slots.  kept_idx / kept_count are
 * that firing's kept list (as given to lsa_tier_plan) and slot_idx the slots
 * lsa_tier_plan assigned to it.  nat describes the native indexer (n_layers
 * must be 1); nat_q bf16 [B][n_h][c], nat_w float32 [B][n_h], nat_k bf16
 * [total chunks][c], all device memory.  Per sequence:
 *   native[i] = sum_h nat_w[b][h] * ReLU(nat_q[b][h] . nat_k[chunk_off[b] + kept_idx[b][i]]),
 * the core_keep[b] (HOST [B], >= 1) kept chunks with the largest native score
 * stay (all when there are fewer; equal scores by the lower position in the
 * kept list, which is ascending); sel_slots[b] (device, row pitch as
 * lsa_tier_sizes) receives their reserve slots in ascending chunk order and
 * sel_count[b] their number; out / lse are the attention over those slots
 * (layouts as lsa_tier_attend); sel_slots must not be kept_idx or slot_idx.
 * No window is added: chunks that must always
 * be attended belong in the kept list.  Kept ids outside 0 .. n_b - 1 give
 * unspecified but in-bounds results.  The workspace is the one lsa_tier_sizes
 * reports; the call only enqueues work on `stream`.
 */
lsa_status lsa_tier_step(const lsa_problem* p, const lsa_tier* tr, const lsa_indexer* nat, const int32_t* core_keep,
                         const void* nat_q, const float* nat_w, const void* nat_k, const int32_t* kept_idx,
                         const int32_t* kept_count, const int32_t* slot_idx, const uint16_t* q,
                         const uint16_t* res_k, const uint16_t* res_v, float softmax_scale, float* out, float* lse,
                         int32_t* sel_slots, int32_t* sel_count, void* ws, size_t ws_bytes, void* stream);
/*
 * Step 3 over the reserve: the attention of lsa_sparse_decode_attn for the
 * chunks held in slots slot_idx[b][0 .. slot_count[b]) (the remapped kept
 * set), reading res_k / res_v only.  The kept chunks in the same order give
 * the same result, bit for bit, as lsa_sparse_decode_attn on the full cache
 * with sel_idx = the kept ids.
 */
lsa_status lsa_tier_attend(const lsa_problem* p, const lsa_tier* tr, const uint16_t* q, const uint16_t* res_k,
                           const uint16_t* res_v, const int32_t* slot_idx, const int32_t* slot_count,
                           float softmax_scale, float* out, float* lse, void* ws, size_t ws_bytes, void* stream);

/*
 * Golden labels (Sec. 2.2, Eqs. 7-11).  logits: device float32, sequence b's
 * block [tau][L][n_b] at element tau * L * entry_off[b] (entry_off the
 * exclusive prefix sum of n_entries); row (i, l) holds the raw indexer logits
 * S_{i,l,s} of decoding step i and layer l over the n_b entries.  Per row:
 * P = softmax(S) (Eq. 7) and its top-p set (Eq. 8), the smallest set of the
 * most probable entries whose probability mass reaches p, more probable first
 * and lower index first among equal logits (-0.0 equal to +0.0).  Per step:
 * V_s = the number of layers whose set holds s (Eq. 9) and the golden set
 * {s : V_s >= theta} (Eq. 10).  Per sequence: the label set, the union of the
 * golden sets of the tau steps (Eq. 11).
 * The decision is exact: weights exp(S - max S) come from one fixed float32
 * method (S - max S rounded to float32, Cody-Waite reduction, Taylor series
 * of degree 7 with fused multiply-adds) as integers floor(w * 2^40), and a set
 * reaches p when
 * (its mass) * p_den >= p_num * (total mass) in integers.  Logits must be
 * finite.
 * Outputs (device): labels [sum_b n_b] int32, sequence b's label ids ascending
 * from element entry_off[b], label_count [B] their number; nucleus_size
 * [B][tau][L] int32 the size of every top-p set and golden_count [B][tau] the
 * size of every golden set (both nullable).  The workspace holds the
 * membership bitmaps of every row.
 */
lsa_status lsa_golden_sizes(const lsa_golden* g, size_t* ws_bytes);
lsa_status lsa_golden_labels(const lsa_golden* g, const float* logits, int32_t* labels, int32_t* label_count,
                             int32_t* nucleus_size, int32_t* golden_count, void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LSA_H_ */
