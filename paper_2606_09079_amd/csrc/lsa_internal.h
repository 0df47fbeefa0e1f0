// Internal interface between the host dispatch (lsa_api.hip) and the gfx950
// kernels.  Per-sequence metadata travels by value in kernel arguments, so a
// launch needs no device-side offset table and nothing is read back to size
// the grids.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/lsa.h"

namespace lsa {

// Per-sequence table computed on the host for one call.
struct SeqTable {
  int32_t batch;
  int32_t n_lookahead;
  int32_t n[LSA_MAX_BATCH];            // chunks of sequence b (a partial last chunk included)
  int32_t tail[LSA_MAX_BATCH];         // tokens in the last chunk of sequence b (the chunk size when complete)
  int32_t w0[LSA_MAX_BATCH];           // two-level path: first chunk of the always-resident window
  int32_t win[LSA_MAX_BATCH];          // two-level path: chunks in that window
  int32_t keep[LSA_MAX_BATCH];         // keep budget k_b
  int32_t nsplit[LSA_MAX_BATCH];       // attention splits per (b, kv head)
  int32_t wg_off[LSA_MAX_BATCH + 1];   // first attention workgroup of sequence b
  int32_t score_wg_off[LSA_MAX_BATCH + 1];  // first scoring workgroup of sequence b
  int64_t chunk_off[LSA_MAX_BATCH + 1];     // first global chunk id of sequence b
  uint32_t* arrive;                    // fused step: split arrival counters, zeroed by the scoring kernel
  int32_t n_arrive;                    //   (B * Hkv words; NULL / 0 otherwise)
};

// Attention launch parameters.
struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* sel_idx;
  const int32_t* sel_count;
  float* out;
  float* lse;            // nullable
  float* part_o;         // [unit][rows_pad][128]
  float* part_ml;        // [unit][rows_pad][2]
  int64_t chunk_stride;
  int64_t head_stride;
  float scale_log2e;     // softmax scale * log2(e)
  int32_t sel_pitch;
  int32_t count_is_keep; // 1: sel_count[b] is min(keep[b], n_b), known on the host (the fused step with Q = 1),
                         // so the kernel need not wait for it
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t group;         // G = Hq / Hkv
  int32_t n_qtok;
  int32_t rows;          // G * n_qtok
  int32_t rows_pad;      // partial rows per (b, g, split): rows rounded up to 16
  uint32_t* arrive;      // NULL: a combine kernel merges the splits.  Else one counter per (b, g), zero on
                         // entry: the last split workgroup of (b, g) to finish merges them (split kernel only)
  int32_t few_splits;    // 1: every sequence has at most 16 splits (the merge order of the few-split combine)
};

// Geometry of the attention launch shared by dispatch and kernels.
constexpr int kAttnWaves = 4;          // waves per workgroup
constexpr int kAttnRowsPerWave = 16;   // MFMA tile rows
constexpr int kHeadDim = 128;
// Split-K sizing: the attention grid is sized to one resident round of the
// MI355X (256 CUs x 2 workgroups of 256 threads at <= 256 registers).  With
// at most kFewSequences sequences the split kernel (<= 16 rows) runs one
// workgroup per CU instead: the second workgroup of a CU lags the first by
// ~10 us, and one per CU measured 0.4-1.5 us faster per step.  Ragged batches
// keep two per CU, whose finer splits balance unequal sequences.
constexpr int kTargetWorkgroups = 512;
constexpr int kTargetWorkgroupsFew = 256;
constexpr int kFewSequences = 8;
constexpr int kFewSplits = 16;   // splits per (sequence, kv head) up to which the few-split merge order holds
constexpr int kMaxSplits = 256;  // splits per (sequence, kv head, row group)

// How the selection reads its scores: raw float32 scores, raw int32 scores, or
// scores the scoring kernel has already mapped to keys (the fused step).
enum KeyMode : int { kKeysFromF32 = 0, kKeysFromI32 = 1, kKeysReady = 2 };

// 32-bit key whose unsigned order is the score order.  float32: -0.0 is folded
// onto +0.0, then positives get the sign bit set and negatives have every bit
// flipped; int32: the sign bit is flipped.
template <int MODE>
__device__ __forceinline__ uint32_t order_key(uint32_t bits) {
  if constexpr (MODE == kKeysReady) {
    return bits;
  } else if constexpr (MODE == kKeysFromI32) {
    return bits ^ 0x80000000u;
  } else {
    if (bits == 0x80000000u) bits = 0u;
    return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
  }
}

// Order key of an exact int32 score of int8 embeddings, |s| <= 512 * 128^2 =
// 2^23: (s + 2^24) << 7 is increasing and spreads the scores over the 32-bit
// range, so the selection's first 12-bit digit tells them apart.  (With the
// sign flip of order_key, every score below 2^20 in magnitude falls in one of
// two bins, and the last digits then run over all the keys.)
__device__ __forceinline__ uint32_t int_score_key(int32_t s) { return ((uint32_t)s + (1u << 24)) << 7; }

// Sequence b of workgroup wg of a grid laid out by wg_off (first workgroup
// of each sequence, wg_off[0] = 0) and the per-sequence numbers the kernels
// read.  Those of sequence 0 are loaded together with the search's first
// bound (the empty asm statements keep the compiler from deferring the loads
// past the branch), so a workgroup of sequence 0 -- every one, with one
// sequence -- waits for one round of kernel-argument loads before it can
// address memory, not two or three.
struct SeqData {
  int b, n, keep, tail, ns, wg0;
  int64_t chunk_off;
};
__device__ __forceinline__ SeqData seq_data(const SeqTable& t, const int32_t* wg_off, int wg) {
  int n0 = t.n[0], k0 = t.keep[0], tl0 = t.tail[0], ns0 = t.nsplit[0], off1 = wg_off[1];
  int64_t c0 = t.chunk_off[0];
  asm volatile("" : "+s"(n0), "+s"(k0), "+s"(tl0), "+s"(ns0), "+s"(off1));
  asm volatile("" : "+s"(c0));
  SeqData r{0, n0, k0, tl0, ns0, 0, c0};
  if (wg >= off1) {
    int b = 1;
    while (wg >= wg_off[b + 1]) ++b;
    r = SeqData{b, t.n[b], t.keep[b], t.tail[b], t.nsplit[b], wg_off[b], t.chunk_off[b]};
  }
  return r;
}

// The fused step's first kernel (the scoring) zeroes the attention's split
// arrival counters of the same call: wave 0 of workgroup 0, at its end (so
// that the check does not delay the kernel's first loads), with stores that
// are coherent across the XCDs' caches.
__device__ __forceinline__ void zero_arrivals(const SeqTable& t) {
  if (blockIdx.x == 0 && threadIdx.x < 64 && t.arrive != nullptr)
    for (int i = threadIdx.x; i < t.n_arrive; i += 64)
      __hip_atomic_store(t.arrive + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// keys == true writes order keys instead of scores (for the fused step).
hipError_t launch_score(const SeqTable& t, int32_t emb_dtype, int32_t emb_dim, const void* qe,
                        const void* E, void* scores, bool keys, hipStream_t s);
int score_rows_per_wg(int32_t emb_dtype, int32_t emb_dim, int32_t n_lookahead);

// Selection variants.  recall: k_b becomes min(keep[b], number of keys >= the
// key of +0.0), i.e. the entries whose sigmoid score reaches 1/2, bounded by
// K_max = keep[b]; n_layers > 1 reads that many score arrays layer_stride
// elements apart and selects on their per-entry maximum (the OR over layers).
// dev_n (nullable): per-sequence key counts in device memory, read by the
// kernel (at most t.n[b]); k_b is then min(keep[b], that count).
// map (nullable): write map[b * map_pitch + i] for each selected key i instead
// of i, then append the window chunks t.w0[b] .. t.w0[b] + t.win[b] - 1, and
// count them in sel_count (the two-level path's Level 2).
struct SelectArgs {
  bool recall = false;
  int32_t n_layers = 1;
  int64_t layer_stride = 0;
  const int32_t* dev_n = nullptr;
  const int32_t* map = nullptr;
  int64_t map_pitch = 0;
};

// keys_ready == true: `scores` holds keys written by launch_score(keys = true)
// or launch_recall_score(keys = true).
hipError_t launch_topk(const SeqTable& t, int32_t emb_dtype, bool keys_ready, const void* scores,
                       int32_t* out_idx, int64_t out_pitch_seq, int64_t out_pitch_query, int32_t* sel_count,
                       hipStream_t s, const SelectArgs& sa = SelectArgs());
hipError_t launch_union(const SeqTable& t, const int32_t* per_query, int32_t k_pitch,
                        int32_t* sel_idx, int32_t sel_pitch, int32_t* sel_count, hipStream_t s);

hipError_t launch_attn(const SeqTable& t, const AttnArgs& a, int32_t chunk_size, hipStream_t s);

// Re-layout of token-major K/V rows into the chunk-paged blocks; a unit is
// one chunk of a sequence's range, one workgroup per (unit, KV head).
struct PackArgs {
  const uint16_t* k_tok;
  const uint16_t* v_tok;
  const int64_t* tok_off;         // device [B]: source row of token 0 of sequence b
  int64_t tok_stride;             // source elements between tokens
  int64_t tok_head_stride;        // source elements between KV heads
  uint16_t* k;
  uint16_t* v;
  int64_t chunk_stride, head_stride;  // destination block strides
  int32_t n_kv_heads, chunk, batch;
  int64_t unit_off[LSA_MAX_BATCH + 1];  // first unit of sequence b
  int64_t first[LSA_MAX_BATCH];         // first token written
  int64_t ctx[LSA_MAX_BATCH];           // one past the last token written
  int64_t chunk_off[LSA_MAX_BATCH];     // first global chunk id of sequence b
};
hipError_t launch_kv_pack(const PackArgs& a, int64_t units, hipStream_t s);

// Recall path: the full Memory Indexer score of L layers.
constexpr int kMaxIdxLayers = LSA_MAX_IDX_LAYERS;
constexpr int kRecallRowsPerWg = 64;  // entries per scoring workgroup (4 waves x 16)
constexpr int kRecallThreads = 256;   // threads per scoring workgroup
struct RecallArgs {
  const uint16_t* q;     // bf16 [B][L][n_h][c]
  const float* w;        // [B][L][n_h]
  const uint16_t* k;     // bf16 [L][total][c]
  int64_t layer_stride;  // total * c
  int64_t total;         // sum_b n_b
  int32_t n_layers, n_heads, key_dim;
  // list mode (nullable list): score only the entries list[b * list_pitch + i],
  // i < list_count[b], and write the keys to out[b * list_pitch + i]
  const int32_t* list = nullptr;
  const int32_t* list_count = nullptr;
  int64_t list_pitch = 0;
  // keys mode, optional: a second indexer of the same head count scored in
  // the same pass (one more staged layer, outside the max over layers), whose
  // order keys go to nat_out[total] (the two-level path's native indexer)
  const uint16_t* nat_q = nullptr;  // bf16 [B][n_h][c]
  const float* nat_w = nullptr;     // [B][n_h]
  const uint16_t* nat_k = nullptr;  // bf16 [total][c]
  uint32_t* nat_out = nullptr;
};
// t.score_wg_off must count kRecallRowsPerWg entries per workgroup.  keys ==
// false writes x [L][total] float32; keys == true writes the order key of
// max_l x_l per entry, [total] (the input of the recall selection).
hipError_t launch_recall_score(const SeqTable& t, const RecallArgs& r, void* out, bool keys, hipStream_t s);

// Two-level selection in one kernel: the recall over the Level-1 keys (order
// keys of max_l x, ready), then the top-k2 of the native keys (order keys)
// among the recalled chunks, then the window chunks.  t.n[b] is the history
// length (at most 16384), t.keep[b] K_max, t.w0 / t.win the window.
struct TwoLevelSelArgs {
  const uint32_t* l1;     // [total] indexed by chunk_off[b] + s
  const uint32_t* l2;     // [total] likewise
  int32_t* out;           // [B][pitch]
  int64_t pitch;
  int32_t* count;         // [B]
  int32_t keep2[LSA_MAX_BATCH];
};
constexpr int kTwoLevelSelMaxN = 16384;
hipError_t launch_two_level_select(const SeqTable& t, const TwoLevelSelArgs& a, hipStream_t s);


// Host tier: residency plan and copies between a pinned host mirror of the
// cache and a GPU reserve of chunk slots.  Sequence b owns reserve slots
// slot_off[b] .. slot_off[b] + slots[b] - 1; slot ids in the lists are local
// to the sequence.
constexpr int kMaxTierChunks = LSA_MAX_TIER_CHUNKS;
constexpr int kMaxTierSlots = LSA_MAX_TIER_SLOTS;
struct TierArgs {
  const int32_t* kept;        // [B][pitch] ascending chunk ids
  const int32_t* kept_count;  // [B]
  const int32_t* prev_slots;  // nullable [B][pitch]: slots the previous kept set reads
  const int32_t* prev_count;  // [B]
  int32_t* owner;             // [sum_b slots[b]] chunk held by each slot, -1 when none
  int32_t* slot_idx;          // [B][pitch] slot of each kept chunk
  int32_t* fetch;             // [B][pitch][2] (chunk, slot) copies
  int32_t* fetch_count;       // [B]
  int32_t pitch;
  int32_t slots[LSA_MAX_BATCH];
  int32_t slot_off[LSA_MAX_BATCH + 1];
};
struct TierFetchArgs {
  const uint16_t* host_k;     // device-visible addresses of the pinned mirror
  const uint16_t* host_v;
  uint16_t* res_k;
  uint16_t* res_v;
  const int32_t* fetch;
  const int32_t* fetch_count;
  int64_t chunk_stride, head_stride;  // mirror strides (the cache's)
  int64_t res_slot_stride;            // n_kv_heads * C * 128
  int32_t pitch;
  int32_t n_kv_heads;
  int32_t workgroups;                 // copy workgroups per launch, 0: the default
  int32_t slots[LSA_MAX_BATCH];
  int32_t slot_off[LSA_MAX_BATCH + 1];
};
hipError_t launch_tier_plan(const SeqTable& t, const TierArgs& a, hipStream_t s);
hipError_t launch_tier_fetch(const SeqTable& t, const TierFetchArgs& a, int32_t chunk_size, hipStream_t s);
hipError_t launch_tier_reset(int32_t* owner, int64_t n, hipStream_t s);

// Golden-label pipeline: per-sequence geometry (by value) and launch arguments.
struct GoldenTable {
  int32_t batch;
  int32_t n[LSA_MAX_BATCH];                // entries n_b
  int32_t words[LSA_MAX_BATCH];            // 32-bit bitmap words per row, ceil(n_b / 32)
  int64_t entry_off[LSA_MAX_BATCH];        // first entry of sequence b (labels)
  int64_t logit_off[LSA_MAX_BATCH];        // first logit of sequence b, tau * L * entry_off[b]
  int64_t bit_off[LSA_MAX_BATCH];          // first word of sequence b's row bitmaps
  int64_t label_word_off[LSA_MAX_BATCH];   // first word of sequence b's label bitmap
};
struct GoldenArgs {
  const float* logits;
  uint32_t* bits;          // [sum_b tau * L * words_b] top-p membership per row
  int32_t* nucleus_size;   // nullable [B][tau][L]
  uint32_t* label_bits = nullptr;    // [label_words] zeroed by the row kernel's first workgroup
  int64_t label_words = 0;
  int32_t* golden_count = nullptr;   // nullable [B][tau], zeroed likewise
  int64_t p_num, p_den;
  int32_t tau, layers, theta;
};
hipError_t launch_golden(const GoldenTable& gt, const GoldenArgs& a, uint32_t* label_bits, int64_t label_words,
                         int32_t* labels, int32_t* label_count, int32_t* golden_count, hipStream_t s);

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

}  // namespace lsa
