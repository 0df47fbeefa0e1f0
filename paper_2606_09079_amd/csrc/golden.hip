// Golden-label pipeline (Sec. 2.2, Eqs. 7-11) over raw indexer logits
// S[i][l][s] of one window: for every decoding step i and layer l the
// softmax over the entries s (Eq. 7) and its top-p set (Eq. 8: the smallest
// set of the most probable entries whose mass reaches p, more probable first,
// lower index first among equals), the votes of the L layers per entry
// (Eq. 9), the golden set of entries with at least theta votes (Eq. 10), and
// the union of the golden sets over the window (Eq. 11).
//
// The top-p decision is exact: a weight is exp(S - max S) evaluated by one
// fixed float32 method (Cody-Waite reduction with the fdlibm split of ln 2,
// Taylor series of degree 7 in Horner form with fused multiply-adds), held as
// the integer q = floor(w * 2^40); masses are integer sums, so their order
// does not matter, and a set reaches p = num / den when
// (its mass) * den >= num * Z in 128-bit integers.
//
// golden_row_kernel -- one 512-thread workgroup per (step, layer) row, three
//   passes over the row: (1) the maximum; (2) a 4096-bin LDS histogram of the
//   masses by the top 12 bits of each logit's order key, whose descending
//   scan finds the bin where the cumulative mass reaches p; (3) the row's
//   membership bitmap for the bins above it (wavefront ballots), the entries
//   of that bin staged in LDS.  Two 10-bit digit rounds over the staged
//   entries give the exact threshold key T and the number of entries equal to
//   T that the set needs (those with the lowest indices).  A bin with more
//   entries than LDS holds is refined by passes over the row instead.  The
//   first two passes read through the caches (the next pass finds part of the
//   row in the Infinity Cache); the last one streams.
// golden_vote_kernel -- one thread per (sequence, step, bitmap word): the
//   votes of the L layers for 32 entries as bit-sliced counters, the theta
//   test, an OR into the label bitmap and the golden-set size.
// golden_compact_kernel -- one workgroup per sequence: label bitmap to
//   ascending entry ids.
#include "lsa_internal.h"

namespace lsa {
namespace {

constexpr int kThreads = 512;   // three rows per compute unit at a time
constexpr int kWaves = kThreads / 64;
constexpr int kBins = 4096;     // first digit: top 12 bits of the order key
constexpr int kSubBins = 1024;  // two more digits of 10 bits
constexpr int kBinsPerThread = kBins / kThreads;
constexpr int kSubPerThread = kSubBins / kThreads;
constexpr int kCand = 1024;     // entries of the threshold bin staged in LDS
constexpr int kUnroll = 16;     // 64-entry groups per wavefront per round

struct u128 {
  uint64_t hi, lo;
};

__device__ __forceinline__ u128 mul64(uint64_t a, uint64_t b) { return {__umul64hi(a, b), a * b}; }
__device__ __forceinline__ bool ge128(u128 a, u128 b) { return a.hi > b.hi || (a.hi == b.hi && a.lo >= b.lo); }

// exp(x) for x <= 0 by the fixed float32 method described above.
__device__ __forceinline__ float exp_fixed(float x) {
  x = x > 0.0f ? 0.0f : x;
  if (x < -64.0f) return 0.0f;
  const float log2e = 1.44269502e+00f;
  const float ln2_hi = 6.9314575195e-01f;
  const float ln2_lo = 1.4286067653e-06f;
  const float k = __builtin_rintf(x * log2e);
  float r = __builtin_fmaf(-k, ln2_hi, x);
  r = __builtin_fmaf(-k, ln2_lo, r);
  float p = 1.0f / 5040.0f;
  p = __builtin_fmaf(p, r, 1.0f / 720.0f);
  p = __builtin_fmaf(p, r, 1.0f / 120.0f);
  p = __builtin_fmaf(p, r, 1.0f / 24.0f);
  p = __builtin_fmaf(p, r, 1.0f / 6.0f);
  p = __builtin_fmaf(p, r, 1.0f / 2.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  return __builtin_ldexpf(p, (int)k);
}

// Weight of a logit in units of 2^-40 of the largest weight: floor(w * 2^40)
// taken exactly from w's bits, w = M 2^(E - 23) with a 24-bit mantissa M and
// -93 <= E <= 0 (w is 0 or normal), so that floor(w 2^40) = M shifted by E + 17.
__device__ __forceinline__ uint64_t mass_of(float s, float m) {
  const uint32_t bits = __float_as_uint(exp_fixed(__fsub_rn(s, m)));
  if (bits == 0u) return 0ull;
  const int sh = (int)(bits >> 23) - 127 + 17;
  const uint64_t M = (uint64_t)((bits & 0x7FFFFFu) | 0x800000u);
  return sh >= 0 ? M << sh : (sh > -24 ? M >> -sh : 0ull);
}

__device__ __forceinline__ uint32_t key_of(float f) { return order_key<kKeysFromF32>(__float_as_uint(f)); }

__device__ __forceinline__ float logit_of(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = op(v, __shfl_xor(v, off));
  return v;
}

// Exclusive prefix sum over the workgroup in thread order; *total gets the sum.
__device__ __forceinline__ uint64_t block_scan_u64(uint64_t v, uint64_t* wave_tot, uint64_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint64_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wave_tot[wave] = incl;
  __syncthreads();
  uint64_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint64_t x = wave_tot[w];
    before += w < wave ? x : 0ull;
    all += x;
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

__global__ void __launch_bounds__(kThreads)
golden_row_kernel(GoldenTable gt, GoldenArgs a) {
  __shared__ unsigned long long hist[kBins];
  __shared__ uint32_t sub_cnt[kSubBins];
  __shared__ uint32_t cand_key[kCand];
  __shared__ uint32_t cand_idx[kCand];
  __shared__ uint64_t wave_tot[kWaves];
  __shared__ float wave_max[kWaves];
  __shared__ uint32_t sh_cnt, sh_digit;
  __shared__ uint64_t sh_above;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (blockIdx.x == 0) {  // the label bitmap and golden-set sizes start at zero (the vote kernel runs after)
    for (int64_t i = tid; i < a.label_words; i += kThreads) a.label_bits[i] = 0u;
    if (a.golden_count != nullptr)
      for (int64_t i = tid; i < (int64_t)gt.batch * a.tau; i += kThreads) a.golden_count[i] = 0;
  }
  const int rows_per_seq = a.tau * a.layers;
  const int b = blockIdx.x / rows_per_seq, row = blockIdx.x % rows_per_seq;
  const int n = gt.n[b], words = gt.words[b];
  const float* S = a.logits + gt.logit_off[b] + (int64_t)row * n;
  uint32_t* bm = a.bits + gt.bit_off[b] + (int64_t)row * words;

  // entry of group u of round base for this lane: 64 consecutive entries per
  // wavefront load, kUnroll consecutive groups per wavefront
  auto entry = [&](int base, int u) { return base + (wave * kUnroll + u) * 64 + lane; };
  constexpr int kRound = kThreads * kUnroll;

  // ---- pass 1: maximum
  float mx = -INFINITY;
  for (int base = 0; base < n; base += kRound) {
    float v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int e = entry(base, u);
      v[u] = e < n ? S[e] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) mx = fmaxf(mx, v[u]);
  }
  mx = wave_reduce(mx, [](float x, float y) { return fmaxf(x, y); });
  for (int i = tid; i < kBins; i += kThreads) hist[i] = 0ull;
  if (lane == 0) wave_max[wave] = mx;
  if (tid == 0) sh_cnt = 0u;
  __syncthreads();
  float m = wave_max[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) m = fmaxf(m, wave_max[w]);

  // ---- pass 2: mass histogram by the top 12 bits of the order key
  for (int base = 0; base < n; base += kRound) {
    float v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int e = entry(base, u);
      v[u] = e < n ? S[e] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (entry(base, u) < n) {
        const uint64_t q = mass_of(v[u], m);
        if (q) atomicAdd(&hist[key_of(v[u]) >> 20], (unsigned long long)q);
      }
    }
  }
  __syncthreads();

  // descending scan of the bins: thread t owns the kBinsPerThread bins below
  // kBins - 1 - kBinsPerThread * t
  uint64_t own[kBinsPerThread], own_sum = 0;
#pragma unroll
  for (int j = 0; j < kBinsPerThread; ++j) {
    own[j] = hist[kBins - 1 - kBinsPerThread * tid - j];
    own_sum += own[j];
  }
  uint64_t Z;
  uint64_t before = block_scan_u64(own_sum, wave_tot, &Z);
  const u128 need = mul64(Z, (uint64_t)a.p_num);
  const uint64_t den = (uint64_t)a.p_den;
#pragma unroll
  for (int j = 0; j < kBinsPerThread; ++j) {
    if (!ge128(mul64(before, den), need) && ge128(mul64(before + own[j], den), need)) {
      sh_digit = (uint32_t)(kBins - 1 - kBinsPerThread * tid - j);
      sh_above = before;
    }
    before += own[j];
  }
  __syncthreads();
  const uint32_t bstar = sh_digit;
  uint64_t above = sh_above;  // mass of every key above the current prefix

  // ---- pass 3: bitmap of the bins above bstar, entries of bstar to LDS
  uint32_t n_in = 0;
  for (int base = 0; base < n; base += kRound) {
    float v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int e = entry(base, u);
      v[u] = e < n ? __builtin_nontemporal_load(S + e) : -INFINITY;
    }
    // the wavefront's kUnroll groups are 2 * kUnroll consecutive bitmap
    // words; lane j < 2 * kUnroll collects word j and stores it
    uint32_t word = 0u;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int e = entry(base, u);
      const uint32_t key = key_of(v[u]);
      const bool valid = e < n;
      const uint64_t in = __ballot(valid && (key >> 20) > bstar);
      const uint64_t cnd = __ballot(valid && (key >> 20) == bstar);
      word = (lane == 2 * u) ? (uint32_t)in : (lane == 2 * u + 1) ? (uint32_t)(in >> 32) : word;
      n_in += lane == 0 ? (uint32_t)__popcll(in) : 0u;
      if (cnd) {
        uint32_t first = 0;
        if (lane == 0) first = atomicAdd(&sh_cnt, (uint32_t)__popcll(cnd));
        first = __shfl(first, 0);
        if (valid && (key >> 20) == bstar) {
          const uint32_t pos = first + (uint32_t)__popcll(cnd & ((1ull << lane) - 1ull));
          if (pos < kCand) {
            cand_key[pos] = key;
            cand_idx[pos] = (uint32_t)e;
          }
        }
      }
    }
    const int w0 = (base >> 5) + wave * 2 * kUnroll;  // first word of this wavefront's groups
    if (lane < 2 * kUnroll && w0 + lane < words) bm[w0 + lane] = word;
  }
  n_in = wave_reduce(n_in, [](uint32_t x, uint32_t y) { return x + y; });
  if (lane == 0) wave_tot[wave] = n_in;
  __syncthreads();
  uint32_t count_in = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) count_in += (uint32_t)wave_tot[w];
  const uint32_t nc = sh_cnt;
  const bool staged = nc <= (uint32_t)kCand;
  __syncthreads();  // wave_tot and sh_cnt are reused below

  // the entries whose key has the given prefix: staged ones, or the row
  auto each = [&](uint32_t prefix, int shift, auto&& f) {
    if (staged) {
      for (uint32_t i = tid; i < nc; i += kThreads) {
        const uint32_t key = cand_key[i];
        if ((key >> shift) == prefix) f(key, cand_idx[i]);
      }
    } else {
      for (int e = tid; e < n; e += kThreads) {
        const uint32_t key = key_of(S[e]);
        if ((key >> shift) == prefix) f(key, (uint32_t)e);
      }
    }
  };

  // ---- two 10-bit digits inside the threshold bin
  uint32_t prefix = bstar;
  for (int round = 0; round < 2; ++round) {
    const int shift = 10 - 10 * round;  // digit bits [shift, shift + 10)
    for (int i = tid; i < kSubBins; i += kThreads) {
      hist[i] = 0ull;
      sub_cnt[i] = 0u;
    }
    __syncthreads();
    each(prefix, shift + 10, [&](uint32_t key, uint32_t) {
      const uint32_t d = (key >> shift) & (kSubBins - 1);
      atomicAdd(&hist[d], (unsigned long long)mass_of(logit_of(key), m));
      atomicAdd(&sub_cnt[d], 1u);
    });
    __syncthreads();
    // descending: thread t owns the kSubPerThread digits below 1023 - kSubPerThread * t
    uint64_t mine[kSubPerThread], mine_sum = 0;
#pragma unroll
    for (int j = 0; j < kSubPerThread; ++j) {
      mine[j] = hist[kSubBins - 1 - kSubPerThread * tid - j];
      mine_sum += mine[j];
    }
    uint64_t tot;
    uint64_t ex = above + block_scan_u64(mine_sum, wave_tot, &tot);
#pragma unroll
    for (int j = 0; j < kSubPerThread; ++j) {
      const int d = kSubBins - 1 - kSubPerThread * tid - j;
      if (sub_cnt[d] != 0u && !ge128(mul64(ex, den), need) && ge128(mul64(ex + mine[j], den), need)) {
        sh_digit = (uint32_t)d;
        sh_above = ex;
      }
      ex += mine[j];
    }
    __syncthreads();
    prefix = (prefix << 10) | sh_digit;
    above = sh_above;
  }
  const uint32_t T = prefix;
  const uint32_t ties = sub_cnt[T & (kSubBins - 1)];
  const uint64_t qT = mass_of(logit_of(T), m);
  // the fewest entries equal to T that reach the mass (1 .. ties)
  uint32_t lo = 1, hi = ties;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) / 2;
    if (ge128(mul64(above + (uint64_t)mid * qT, den), need)) hi = mid;
    else lo = mid + 1;
  }
  const uint32_t r = lo;

  // ---- the threshold bin's members: keys above T, and T itself when all of
  // its entries are needed
  uint32_t n_mid = 0;
  each(bstar, 20, [&](uint32_t key, uint32_t idx) {
    if (key > T || (key == T && r == ties)) {
      atomicOr(&bm[idx >> 5], 1u << (idx & 31));
      ++n_mid;
    }
  });
  if (r != ties && wave == 0) {
    // only r of the entries equal to T, the lowest indices first
    uint32_t run = 0;
    for (int g0 = 0; g0 < n && run < r; g0 += 64) {
      const int e = g0 + lane;
      const bool tie = e < n && key_of(S[e]) == T;
      const uint64_t bal = __ballot(tie);
      const uint32_t rank = run + (uint32_t)__popcll(bal & ((1ull << lane) - 1ull));
      if (tie && rank < r) atomicOr(&bm[e >> 5], 1u << (e & 31));
      run += (uint32_t)__popcll(bal);
    }
  }
  n_mid = wave_reduce(n_mid, [](uint32_t x, uint32_t y) { return x + y; });
  __syncthreads();
  if (lane == 0) wave_tot[wave] = n_mid;
  __syncthreads();
  if (tid == 0 && a.nucleus_size != nullptr) {
    uint32_t tot = count_in + (r == ties ? 0u : r);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += (uint32_t)wave_tot[w];
    a.nucleus_size[(int64_t)b * rows_per_seq + row] = (int32_t)tot;
  }
}

// Bit-sliced vote counters: c[k] holds bit k of the count of each of 32 entries.
constexpr int kCountBits = 7;  // counts up to 127 >= LSA_MAX_GOLDEN_LAYERS

__global__ void __launch_bounds__(256)
golden_vote_kernel(GoldenTable gt, GoldenArgs a, uint32_t* __restrict__ label_bits, int32_t* golden_count) {
  const int b = blockIdx.z, i = blockIdx.y;
  const int w = blockIdx.x * 256 + threadIdx.x;
  const int words = gt.words[b];
  uint32_t A = 0u;
  if (w < words) {
    uint32_t c[kCountBits] = {};
    const uint32_t* src = a.bits + gt.bit_off[b] + (int64_t)i * a.layers * words + w;
    // the layers' words eight at a time, every load of a batch in flight at once
    for (int l0 = 0; l0 < a.layers; l0 += 8) {
      uint32_t x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = l0 + j < a.layers ? src[(int64_t)(l0 + j) * words] : 0u;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint32_t carry = x[j];
#pragma unroll
        for (int k = 0; k < kCountBits; ++k) {
          const uint32_t t = c[k] & carry;
          c[k] ^= carry;
          carry = t;
        }
      }
    }
    // count >= theta, bit-sliced, from the most significant bit down
    uint32_t gt_ = 0u, eq = 0xFFFFFFFFu;
#pragma unroll
    for (int k = kCountBits - 1; k >= 0; --k) {
      if ((a.theta >> k) & 1) {
        eq &= c[k];
      } else {
        gt_ |= eq & c[k];
        eq &= ~c[k];
      }
    }
    A = gt_ | eq;
    if (A) atomicOr(&label_bits[gt.label_word_off[b] + w], A);
  }
  if (golden_count != nullptr) {
    uint32_t cnt = (uint32_t)__popc(A);
    cnt = wave_reduce(cnt, [](uint32_t x, uint32_t y) { return x + y; });
    if ((threadIdx.x & 63) == 0 && cnt) atomicAdd(&golden_count[b * a.tau + i], (int32_t)cnt);
  }
}

__global__ void __launch_bounds__(kThreads)
golden_compact_kernel(GoldenTable gt, const uint32_t* __restrict__ label_bits, int32_t* labels,
                      int32_t* label_count) {
  __shared__ uint64_t wave_tot[kWaves];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int words = gt.words[b];
  const uint32_t* src = label_bits + gt.label_word_off[b];
  const int seg = (words + kThreads - 1) / kThreads;
  const int w0 = min(tid * seg, words), w1 = min(w0 + seg, words);
  uint64_t cnt = 0;
  for (int w = w0; w < w1; ++w) cnt += __popc(src[w]);
  uint64_t total;
  uint64_t pos = block_scan_u64(cnt, wave_tot, &total);
  int32_t* out = labels + gt.entry_off[b];
  for (int w = w0; w < w1; ++w) {
    uint32_t x = src[w];
    while (x) {
      const int bit = __builtin_ctz(x);
      x &= x - 1u;
      out[pos++] = 32 * w + bit;
    }
  }
  if (tid == 0) label_count[b] = (int32_t)total;
}

}  // namespace

hipError_t launch_golden(const GoldenTable& gt, const GoldenArgs& a, uint32_t* label_bits, int64_t label_words,
                         int32_t* labels, int32_t* label_count, int32_t* golden_count, hipStream_t s) {
  GoldenArgs ra = a;
  ra.label_bits = label_bits;
  ra.label_words = label_words;
  ra.golden_count = golden_count;
  hipLaunchKernelGGL(golden_row_kernel, dim3((unsigned)(gt.batch * a.tau * a.layers)), dim3(kThreads), 0, s, gt, ra);
  int max_words = 0;
  for (int b = 0; b < gt.batch; ++b) max_words = std::max(max_words, gt.words[b]);
  hipLaunchKernelGGL(golden_vote_kernel, dim3((unsigned)((max_words + 255) / 256), (unsigned)a.tau, (unsigned)gt.batch),
                     dim3(256), 0, s, gt, a, label_bits, golden_count);
  hipLaunchKernelGGL(golden_compact_kernel, dim3((unsigned)gt.batch), dim3(kThreads), 0, s, gt,
                     (const uint32_t*)label_bits, labels, label_count);
  return hipGetLastError();
}

}  // namespace lsa
