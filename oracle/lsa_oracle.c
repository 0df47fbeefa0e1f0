/*
 * CPU oracle for the LSA decode hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct reference for what one decode step of
 * Lookahead Sparse Attention computes: score every compressed chunk with the
 * Memory Indexer, keep the top-k chunks, attend over the kept chunks only.
 * Only the test suite, the smoke check and the benchmark's CPU baseline may
 * load this library; the product path never links or calls it.
 *
 * Arithmetic is float64 (int64 for int8 embeddings), every loop runs in index
 * order, and nothing is blocked, fused or reordered beyond the definitions.
 * Inputs in bf16 are passed as their raw 16-bit patterns and widened here.
 *
 * Readings of the paper that this file encodes:
 *  - Score (Sec. 2.1, Eq. 4): the gated multi-head form with one indexer head
 *    and unit gate, i.e. the dual-encoder dot product s_c = qe . E_c.  The
 *    sigmoid and ReLU of Eq. 4 are non-decreasing, so they cannot reorder
 *    chunks with positive dot products; the keep-budget selection is taken on
 *    the raw dot product.
 *  - Selection (Sec. 2.1, Eq. 6; Sec. 2.5 bound K_max): the k chunks with
 *    the largest score, ties broken towards the lower chunk index, reported in
 *    ascending chunk order.  With several lookahead queries the kept set is the
 *    union of the per-query top-k sets (the set union of Eq. 13).
 *  - Attention (Sec. 2.1, core attention over the selected entries):
 *    softmax(q K^T * scale) V over the tokens of the kept chunks, with query
 *    head h reading KV head floor(h / G).  An empty kept set gives out = 0 and
 *    lse = -inf (the empty sum), which only the recall path below can produce.
 *  - Two-level selection (Sec. 2.1 after Eq. 5; Sec. 2.5): the history is the
 *    complete entries before the always-resident window; Level 1 recalls from
 *    it as below, Level 2 keeps the k2 recalled entries with the largest native
 *    indexer score (Eq. 6, lower id first on ties), and the kept set is those
 *    plus every chunk of the window, the last one possibly partial.
 *  - Recall (the full Memory Indexer of Sec. 2.1 Eq. 4, the threshold of Eq. 5,
 *    the OR over indexer layers of Eq. 13 and the K_max bound of Sec. 2.5):
 *    layer l recalls entry s when sigma(x_l(s)) >= 1/2 with
 *    x_l(s) = sum_h w_h ReLU(q_h . K_s); the recalled set is the OR over the
 *    layers; when it holds more than K_max entries, the K_max with the largest
 *    max_l x_l(s) are kept (lower id first on ties).
 *  - Golden labels (Sec. 2.2, Eqs. 7-11): the top-p set of Eq. 8 is read as
 *    the text states it, the smallest set of the most probable entries whose
 *    probability mass reaches p (entries ordered by probability, then by lower
 *    index); Eq. 8 as printed (cumulative mass <= p) would leave the set empty
 *    whenever the most probable entry alone exceeds p.  The softmax of Eq. 7
 *    is taken in float64 with the C library's exp, and "the first j entries
 *    reach p" is decided in the equivalent form (1 - p) * head >= p * tail of
 *    the two float64 sums of positive weights, so that p = 1 needs every
 *    entry and a set whose mass is exactly p (equal weights) is enough.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double bf16_to_f64(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* ---------------------------------------------------------------- O1 score */

/* s[c] = sum_i qe[i] * E[c][i], float32 inputs, float64 sum (Sec. 2.1, Eq. 4). */
void oracle_score_f32(const float* qe, const float* E, int64_t n, int32_t D, double* out) {
  for (int64_t c = 0; c < n; ++c) {
    double s = 0.0;
    for (int32_t i = 0; i < D; ++i) s += (double)qe[i] * (double)E[c * D + i];
    out[c] = s;
  }
}

/* Same, bf16 inputs given as bit patterns. */
void oracle_score_bf16(const uint16_t* qe, const uint16_t* E, int64_t n, int32_t D, double* out) {
  for (int64_t c = 0; c < n; ++c) {
    double s = 0.0;
    for (int32_t i = 0; i < D; ++i) s += bf16_to_f64(qe[i]) * bf16_to_f64(E[c * D + i]);
    out[c] = s;
  }
}

/* Same, int8 inputs, exact int64 sum. */
void oracle_score_i8(const int8_t* qe, const int8_t* E, int64_t n, int32_t D, int64_t* out) {
  for (int64_t c = 0; c < n; ++c) {
    int64_t s = 0;
    for (int32_t i = 0; i < D; ++i) s += (int64_t)qe[i] * (int64_t)E[c * D + i];
    out[c] = s;
  }
}

/* ----------------------------------------------------------------- O2 top-k */

typedef struct { double s; int64_t c; } scored_f;
typedef struct { int64_t s; int64_t c; } scored_i;

/* Larger score first; equal scores: lower chunk index first. */
static int by_score_desc_f(const void* a, const void* b) {
  const scored_f* x = (const scored_f*)a;
  const scored_f* y = (const scored_f*)b;
  if (x->s > y->s) return -1;
  if (x->s < y->s) return 1;
  return (x->c > y->c) - (x->c < y->c);
}

static int by_score_desc_i(const void* a, const void* b) {
  const scored_i* x = (const scored_i*)a;
  const scored_i* y = (const scored_i*)b;
  if (x->s > y->s) return -1;
  if (x->s < y->s) return 1;
  return (x->c > y->c) - (x->c < y->c);
}

static int ascending_i32(const void* a, const void* b) {
  const int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  return (x > y) - (x < y);
}

/* Top-k of float64 scores: writes the k kept chunk ids in ascending order and
 * returns k, or -1 on a bad argument or allocation failure. */
int64_t oracle_topk_f64(const double* s, int64_t n, int64_t k, int32_t* out) {
  if (n <= 0 || k < 1 || k > n) return -1;
  scored_f* v = (scored_f*)malloc((size_t)n * sizeof *v);
  if (!v) return -1;
  for (int64_t c = 0; c < n; ++c) { v[c].s = s[c]; v[c].c = c; }
  qsort(v, (size_t)n, sizeof *v, by_score_desc_f);
  for (int64_t j = 0; j < k; ++j) out[j] = (int32_t)v[j].c;
  free(v);
  qsort(out, (size_t)k, sizeof *out, ascending_i32);
  return k;
}

/* Top-k of int64 scores (int8 embeddings). */
int64_t oracle_topk_i64(const int64_t* s, int64_t n, int64_t k, int32_t* out) {
  if (n <= 0 || k < 1 || k > n) return -1;
  scored_i* v = (scored_i*)malloc((size_t)n * sizeof *v);
  if (!v) return -1;
  for (int64_t c = 0; c < n; ++c) { v[c].s = s[c]; v[c].c = c; }
  qsort(v, (size_t)n, sizeof *v, by_score_desc_i);
  for (int64_t j = 0; j < k; ++j) out[j] = (int32_t)v[j].c;
  free(v);
  qsort(out, (size_t)k, sizeof *out, ascending_i32);
  return k;
}

/* Union of n_lists chunk-id lists of length k each (row-major), ascending.
 * Returns the union size, or -1 on a bad argument. */
int64_t oracle_union(const int32_t* lists, int32_t n_lists, int64_t k, int64_t n, int32_t* out) {
  if (n <= 0 || n_lists < 1 || k < 0) return -1;
  unsigned char* in = (unsigned char*)calloc((size_t)n, 1);
  if (!in) return -1;
  for (int64_t j = 0; j < (int64_t)n_lists * k; ++j) {
    if (lists[j] < 0 || lists[j] >= n) { free(in); return -1; }
    in[lists[j]] = 1;
  }
  int64_t u = 0;
  for (int64_t c = 0; c < n; ++c)
    if (in[c]) out[u++] = (int32_t)c;
  free(in);
  return u;
}

/* ------------------------------------------------------------- O3 attention */

/*
 * Attention of R query rows against the tokens of the selected chunks of one
 * KV head.
 *   q     [R][d]        bf16 bits
 *   Kh,Vh [n_tok][d]    bf16 bits, logical token-major for this KV head
 *   sel   [nsel]        chunk ids; the token list is the concatenation, over
 *                       sel in the given order, of tokens [c*C, c*C + C)
 *   out   [R][d]        float64,  out = sum_i w_i V_i / sum_i w_i
 *   lse   [R]           float64,  m + log(sum_i w_i)
 * where l_i = scale * q . K_i, m = max_i l_i and w_i = exp(l_i - m).
 * Returns 0, or -1 on a bad argument or allocation failure.
 */
int oracle_attention(const uint16_t* q, int32_t R, const uint16_t* Kh, const uint16_t* Vh,
                     int64_t n_tok, int32_t d, int32_t C, const int32_t* sel, int64_t nsel,
                     double scale, double* out, double* lse) {
  if (R < 1 || d < 1 || C < 1 || nsel < 0) return -1;
  if (nsel == 0) { /* nothing to attend: the empty sum */
    for (int64_t i = 0; i < (int64_t)R * d; ++i) out[i] = 0.0;
    for (int32_t r = 0; r < R; ++r) lse[r] = -INFINITY;
    return 0;
  }
  for (int64_t j = 0; j < nsel; ++j)
    if (sel[j] < 0 || (int64_t)(sel[j] + 1) * C > n_tok) return -1;
  const int64_t T = nsel * C;
  double* logit = (double*)malloc((size_t)T * sizeof *logit);
  if (!logit) return -1;
  for (int32_t r = 0; r < R; ++r) {
    const uint16_t* qr = q + (int64_t)r * d;
    for (int64_t i = 0; i < T; ++i) {
      const int64_t tok = (int64_t)sel[i / C] * C + i % C;
      double dot = 0.0;
      for (int32_t e = 0; e < d; ++e) dot += bf16_to_f64(qr[e]) * bf16_to_f64(Kh[tok * d + e]);
      logit[i] = dot * scale;
    }
    double m = logit[0];
    for (int64_t i = 1; i < T; ++i)
      if (logit[i] > m) m = logit[i];
    double Z = 0.0;
    for (int64_t i = 0; i < T; ++i) {
      logit[i] = exp(logit[i] - m); /* the weight w_i from here on */
      Z += logit[i];
    }
    for (int32_t e = 0; e < d; ++e) {
      double acc = 0.0;
      for (int64_t i = 0; i < T; ++i) {
        const int64_t tok = (int64_t)sel[i / C] * C + i % C;
        acc += logit[i] * bf16_to_f64(Vh[tok * d + e]);
      }
      out[(int64_t)r * d + e] = acc / Z;
    }
    lse[r] = m + log(Z);
  }
  free(logit);
  return 0;
}

/*
 * Attention of R query rows over an explicit list of tokens of one KV head
 * (the token-level form of the function above, for kept sets whose last
 * chunk is partial).  toks [ntoks] are token indices < n_tok, attended in the
 * given order.  Returns 0, or -1 on a bad argument or allocation failure.
 */
int oracle_attention_tokens(const uint16_t* q, int32_t R, const uint16_t* Kh, const uint16_t* Vh, int64_t n_tok,
                            int32_t d, const int64_t* toks, int64_t ntoks, double scale, double* out, double* lse) {
  if (R < 1 || d < 1 || ntoks < 0) return -1;
  for (int64_t i = 0; i < ntoks; ++i)
    if (toks[i] < 0 || toks[i] >= n_tok) return -1;
  if (ntoks == 0) { /* nothing to attend: the empty sum */
    for (int64_t i = 0; i < (int64_t)R * d; ++i) out[i] = 0.0;
    for (int32_t r = 0; r < R; ++r) lse[r] = -INFINITY;
    return 0;
  }
  double* w = (double*)malloc((size_t)ntoks * sizeof *w);
  if (!w) return -1;
  for (int32_t r = 0; r < R; ++r) {
    const uint16_t* qr = q + (int64_t)r * d;
    for (int64_t i = 0; i < ntoks; ++i) {
      double dot = 0.0;
      for (int32_t e = 0; e < d; ++e) dot += bf16_to_f64(qr[e]) * bf16_to_f64(Kh[toks[i] * d + e]);
      w[i] = dot * scale;
    }
    double m = w[0];
    for (int64_t i = 1; i < ntoks; ++i)
      if (w[i] > m) m = w[i];
    double Z = 0.0;
    for (int64_t i = 0; i < ntoks; ++i) {
      w[i] = exp(w[i] - m);
      Z += w[i];
    }
    for (int32_t e = 0; e < d; ++e) {
      double acc = 0.0;
      for (int64_t i = 0; i < ntoks; ++i) acc += w[i] * bf16_to_f64(Vh[toks[i] * d + e]);
      out[(int64_t)r * d + e] = acc / Z;
    }
    lse[r] = m + log(Z);
  }
  free(w);
  return 0;
}

/* ---------------------------------------------------------------- R recall */

/*
 * Gated multi-head index score of one indexer layer, the argument of the
 * sigmoid in Sec. 2.1 Eq. 4:
 *   x[s] = sum_h w[h] * ReLU(q[h] . K[s])
 *   q [n_h][c] bf16 bits, w [n_h] float32, K [n][c] bf16 bits, x [n] float64.
 */
void oracle_index_score_bf16(const uint16_t* q, const float* w, const uint16_t* K, int64_t n, int32_t n_h,
                             int32_t c, double* out) {
  for (int64_t s = 0; s < n; ++s) {
    double x = 0.0;
    for (int32_t h = 0; h < n_h; ++h) {
      double dot = 0.0;
      for (int32_t i = 0; i < c; ++i) dot += bf16_to_f64(q[(int64_t)h * c + i]) * bf16_to_f64(K[s * c + i]);
      const double relu = dot > 0.0 ? dot : 0.0;
      x += (double)w[h] * relu;
    }
    out[s] = x;
  }
}

/*
 * Recall of the Memory Indexers of L layers over n entries (Sec. 2.1 Eq. 5,
 * the OR of Eq. 13, the K_max bound of Sec. 2.5).  x [L][n] float64 holds the
 * sigmoid arguments.  Layer l recalls entry s when sigma(x[l][s]) >= 1/2; the
 * sigmoid is increasing with sigma(0) = 1/2, so that is exactly x[l][s] >= 0
 * (-0.0 included), and taking it on x keeps the decision free of the rounding
 * of a computed sigmoid.  An entry is recalled when any layer recalls it.  If
 * more than kmax entries are recalled, the kmax with the largest max_l x[l][s]
 * stay (lower id first on ties).  Writes the kept ids in ascending order and
 * returns their count, 0 .. kmax, or -1 on a bad argument or allocation failure.
 */
int64_t oracle_recall(const double* x, int32_t L, int64_t n, int64_t kmax, int32_t* out) {
  if (L < 1 || n <= 0 || kmax < 1) return -1;
  scored_f* v = (scored_f*)malloc((size_t)n * sizeof *v);
  if (!v) return -1;
  int64_t m = 0;
  for (int64_t s = 0; s < n; ++s) {
    int recalled = 0;
    double best = x[s];
    for (int32_t l = 0; l < L; ++l) {
      const double xl = x[(int64_t)l * n + s];
      if (xl >= 0.0) recalled = 1;
      if (xl > best) best = xl;
    }
    if (recalled) {
      v[m].s = best;
      v[m].c = s;
      ++m;
    }
  }
  if (m > kmax) {
    qsort(v, (size_t)m, sizeof *v, by_score_desc_f);
    m = kmax;
  }
  for (int64_t j = 0; j < m; ++j) out[j] = (int32_t)v[j].c;
  free(v);
  qsort(out, (size_t)m, sizeof *out, ascending_i32);
  return m;
}

/*
 * Level 2 of the two-level selection and the window (Sec. 2.1 after Eq. 5,
 * Eq. 6; Sec. 2.5).  recalled [m] are the ascending ids that Level 1 kept from
 * the history (entries before w0); native [n_hist] is the native indexer's
 * score of every history entry.  The k2 recalled entries with the largest
 * native score stay (all of them when m <= k2; lower id first on ties); the
 * kept set is those plus the window chunks w0 .. n_total - 1.  Writes the kept
 * ids in ascending order and returns their count, or -1 on a bad argument or
 * allocation failure.
 */
int64_t oracle_two_level(const int32_t* recalled, int64_t m, const double* native, int64_t n_hist, int64_t k2,
                         int64_t w0, int64_t n_total, int32_t* out) {
  if (m < 0 || k2 < 1 || n_hist < 0 || w0 < n_hist || w0 > n_total) return -1;
  for (int64_t j = 0; j < m; ++j)
    if (recalled[j] < 0 || recalled[j] >= n_hist || (j > 0 && recalled[j] <= recalled[j - 1])) return -1;
  int64_t core = m;
  if (m > 0) {
    scored_f* v = (scored_f*)malloc((size_t)m * sizeof *v);
    if (!v) return -1;
    for (int64_t j = 0; j < m; ++j) {
      v[j].s = native[recalled[j]];
      v[j].c = recalled[j];
    }
    if (m > k2) {
      qsort(v, (size_t)m, sizeof *v, by_score_desc_f);
      core = k2;
    }
    for (int64_t j = 0; j < core; ++j) out[j] = (int32_t)v[j].c;
    free(v);
    qsort(out, (size_t)core, sizeof *out, ascending_i32);
  }
  for (int64_t c = w0; c < n_total; ++c) out[core + (c - w0)] = (int32_t)c;
  return core + (n_total - w0);
}

/* ------------------------------------------------------------ golden labels */

typedef struct { float s; int64_t c; } logit_entry;

/* Larger logit first (so larger probability first); equal logits, -0.0 and
 * +0.0 included: lower entry index first. */
static int by_logit_desc(const void* a, const void* b) {
  const logit_entry* x = (const logit_entry*)a;
  const logit_entry* y = (const logit_entry*)b;
  if (x->s > y->s) return -1;
  if (x->s < y->s) return 1;
  return (x->c > y->c) - (x->c < y->c);
}

/*
 * Top-p set of one row of logits (Eq. 7 softmax, Eq. 8 nucleus).  Entries are
 * ordered by (logit desc, index asc); w_j = exp(S_j - max S) in float64 is the
 * softmax numerator of the j-th of them (dividing by the sum does not change
 * which prefix reaches p).  The set is the shortest prefix j = 0 .. J whose
 * mass head = w_0 + .. + w_J reaches p of the total head + tail, tail =
 * w_{J+1} + .. + w_{n-1}, i.e. (p_den - p_num) * head >= p_num * tail.
 * mark[s] = 1 for the entries of the set.  order (nullable) receives the entry
 * order and cum (nullable) the mass fraction head / (head + tail) of every
 * prefix.  Returns the size of the set, or -1 on a bad argument or allocation
 * failure.  Logits must be finite; a weight below the smallest double (a
 * logit more than about 745 below the maximum) counts as 0.
 */
int64_t oracle_top_p(const float* S, int64_t n, int64_t p_num, int64_t p_den, uint8_t* mark, int64_t* order,
                     double* cum) {
  if (n < 1 || p_num < 1 || p_den < p_num) return -1;
  double m = (double)S[0];
  for (int64_t s = 1; s < n; ++s)
    if ((double)S[s] > m) m = (double)S[s];
  logit_entry* v = (logit_entry*)malloc((size_t)n * sizeof *v);
  double* w = (double*)malloc((size_t)n * sizeof *w);
  double* tail = (double*)malloc((size_t)(n + 1) * sizeof *tail);
  if (!v || !w || !tail) { free(v); free(w); free(tail); return -1; }
  for (int64_t s = 0; s < n; ++s) {
    v[s].s = S[s];
    v[s].c = s;
  }
  qsort(v, (size_t)n, sizeof *v, by_logit_desc);
  for (int64_t j = 0; j < n; ++j) w[j] = exp((double)v[j].s - m);
  tail[n] = 0.0; /* tail[j] = w_j + .. + w_{n-1}, summed from the smallest */
  for (int64_t j = n - 1; j >= 0; --j) tail[j] = tail[j + 1] + w[j];
  memset(mark, 0, (size_t)n);
  double head = 0.0;
  int64_t size = -1;
  for (int64_t j = 0; j < n; ++j) {
    head += w[j];
    if (order) order[j] = v[j].c;
    if (cum) cum[j] = head / (head + tail[j + 1]);
    if (size < 0) {
      mark[v[j].c] = 1;
      if ((double)(p_den - p_num) * head >= (double)p_num * tail[j + 1]) size = j + 1;
    }
  }
  free(v);
  free(w);
  free(tail);
  return size;
}

/*
 * The label pipeline of one window: logits [tau][L][n] (row (i, l) holds
 * S_{i,l,.}).  For each step i the top-p set of every layer, the vote count
 * V_{i,s} = number of layers whose set holds s (Eq. 9), the golden set
 * A_i = {s : V_{i,s} >= theta} (Eq. 10), and the label set Y = the union of
 * the A_i over the window (Eq. 11).  Writes label[s] = 1 for s in Y,
 * nucleus_size[i * L + l] = size of the top-p set of row (i, l) and
 * golden_count[i] = |A_i| (both nullable), and returns |Y| (-1 on a bad
 * argument or allocation failure).
 */
int64_t oracle_golden_labels(const float* logits, int32_t tau, int32_t L, int64_t n, int64_t p_num, int64_t p_den,
                             int32_t theta, uint8_t* label, int32_t* nucleus_size, int32_t* golden_count) {
  if (tau < 1 || L < 1 || n < 1 || theta < 1) return -1;
  uint8_t* mark = (uint8_t*)malloc((size_t)n);
  int32_t* votes = (int32_t*)malloc((size_t)n * sizeof *votes);
  if (!mark || !votes) { free(mark); free(votes); return -1; }
  memset(label, 0, (size_t)n);
  for (int32_t i = 0; i < tau; ++i) {
    memset(votes, 0, (size_t)n * sizeof *votes);
    for (int32_t l = 0; l < L; ++l) {
      const int64_t size = oracle_top_p(logits + ((int64_t)i * L + l) * n, n, p_num, p_den, mark, NULL, NULL);
      if (size < 0) { free(mark); free(votes); return -1; }
      if (nucleus_size) nucleus_size[(int64_t)i * L + l] = (int32_t)size;
      for (int64_t s = 0; s < n; ++s) votes[s] += mark[s];
    }
    int32_t golden = 0;
    for (int64_t s = 0; s < n; ++s)
      if (votes[s] >= theta) {
        ++golden;
        label[s] = 1;
      }
    if (golden_count) golden_count[i] = golden;
  }
  int64_t count = 0;
  for (int64_t s = 0; s < n; ++s) count += label[s];
  free(mark);
  free(votes);
  return count;
}
