/*
 * Host side of the seeded input generator for the LSA decode hot path.
 *
 * Test and benchmark infrastructure: it produces input bytes only and holds
 * none of the method's arithmetic (no scoring, selection or attention).
 *
 * Random numbers come from SplitMix64 used as a counter-based generator: the
 * value at counter i of a stream is mix64(key + (i + 1) * GAMMA), where
 * mix64 is the SplitMix64 output finaliser (Steele, Lea, Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014).  The device
 * fill in synth_dev.hip evaluates the same function, so any element of the
 * K/V cache can be regenerated on the host from its logical coordinates.
 */
#include <stdint.h>

#define SYNTH_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t synth_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t synth_stream_key(uint64_t seed, uint64_t stream) {
  return synth_mix64(seed * SYNTH_GAMMA + stream * 0xD1B54A32D192ED03ULL + 1ULL);
}

uint64_t synth_draw(uint64_t key, uint64_t i) {
  return synth_mix64(key + (i + 1ULL) * SYNTH_GAMMA);
}

/*
 * Fill the listed chunks of one KV head of a cache with table-mapped normal
 * draws.  The element at global token tau, head h, dimension e has counter
 * (tau * hkv + h) * d + e; its value is table[draw >> 48].  Output is the
 * logical token-major slab out[j][t][e] for chunk j of the list, token t of
 * that chunk and dimension e.
 */
void synth_kv_chunks(uint64_t key, const uint16_t* table, int32_t hkv, int32_t h,
                     int32_t d, int32_t chunk, const int64_t* chunks, int64_t n_list,
                     uint16_t* out) {
  for (int64_t j = 0; j < n_list; ++j) {
    const int64_t tau0 = chunks[j] * (int64_t)chunk;
    for (int32_t t = 0; t < chunk; ++t) {
      const uint64_t base = (uint64_t)(((tau0 + t) * hkv + h) * (int64_t)d);
      uint16_t* row = out + ((j * chunk) + t) * (int64_t)d;
      for (int32_t e = 0; e < d; ++e) row[e] = table[synth_draw(key, base + (uint64_t)e) >> 48];
    }
  }
}

/* Raw draws for counters [start, start + n): used by the Python side for the
 * small tensors (embeddings, queries, lengths). */
void synth_draws(uint64_t key, uint64_t start, int64_t n, uint64_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = synth_draw(key, start + (uint64_t)i);
}

/*
 * Logits of the golden-label workload, rows x n entries starting at counter
 * start (row r, entry s at counter start + r * n + s).  Every value is built
 * from exact or single correctly rounded float32 operations, so the device
 * fill produces the same bytes:
 *   z    = table[draw >> 48] + ((draw >> 32) & 0xFFFF) * 2^-26
 *   v    = z * sigma                          (sigma a power of two: exact)
 *   v   += beta   when entry s of sequence b is relevant (a per-sequence draw
 *                 below rel_thr) and boosted in this row (a per-element draw
 *                 below boost_thr)
 */
void synth_golden_logits(uint64_t key_noise, uint64_t key_rel, uint64_t key_boost, const float* table,
                         uint64_t start, int64_t rows, int64_t n, int32_t b, float sigma, float beta,
                         uint32_t rel_thr, uint32_t boost_thr, float* out) {
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t s = 0; s < n; ++s) {
      const uint64_t c = start + (uint64_t)(r * n + s);
      const uint64_t d = synth_draw(key_noise, c);
      const float z = table[d >> 48] + (float)((d >> 32) & 0xFFFFu) * 0x1p-26f;
      float v = z * sigma;
      const int relevant = (uint32_t)(synth_draw(key_rel, ((uint64_t)b << 32) | (uint64_t)s) >> 32) < rel_thr;
      if (relevant && (uint32_t)(synth_draw(key_boost, c) >> 32) < boost_thr) v = v + beta;
      out[r * n + s] = v;
    }
}
