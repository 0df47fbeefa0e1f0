// Step 2 of the decode hot path: keep the k highest-scoring chunks (the Top-k
// of Sec. 2.1, Eq. 6, with the K_max recall bound of Sec. 2.5 as k) and,
// with several lookahead queries, the union of the per-query sets (the set
// union of Sec. 2.4, Eq. 13).
//
// One 1024-thread workgroup per (sequence, query).  Scores map to 32-bit keys
// whose unsigned order is the score order (order_key; the fused step receives
// them already mapped from the scoring kernel).  A radix select finds the k-th
// largest key T and how many keys equal to T must be taken; every key above T
// is kept, and keys equal to T in chunk order while the tie quota lasts, so
// ties go to the lower chunk id and the output is ascending with no sort.
//
// topk_select_kernel (up to 16384 chunks) runs on one compute unit, where every
// instruction executed by all 1024 threads costs 16 cycles, so the design
// minimises per-key work:
//   - keys stay in registers (up to 16 per thread, coalesced buffer loads);
//   - first digit: top 12 bits into an LDS histogram whose atomic return
//     values double as each key's rank in its bin, so the keys of the
//     threshold bin are packed into a candidate list without a scan;
//   - the last 20 bits: two 10-bit digits resolved by one wavefront over the
//     candidates, with no barriers;
//   - the kept set is built as bitmaps straight from wavefront ballots, and
//     512 threads emit the set bits of their 32-chunk words in order.
// topk_kernel (longer contexts): 8-bit digits, with the keys staged in LDS when
//   they fit and re-read from memory in every pass otherwise.
#include "lsa_internal.h"

namespace lsa {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kLdsKeys = 16384;
constexpr int kSubHist = 4;

// Exclusive block-wide prefix sum of a 64-bit value (two 32-bit counters).
__device__ __forceinline__ uint64_t block_exclusive_scan(uint64_t v, uint64_t* wave_tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t lo = __shfl_up((uint32_t)incl, off);
    const uint32_t hi = __shfl_up((uint32_t)(incl >> 32), off);
    if (lane >= off) incl += ((uint64_t)hi << 32) | lo;
  }
  if (lane == 63) wave_tot[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t run = 0;
    for (int w = 0; w < kWaves; ++w) {
      const uint64_t x = wave_tot[w];
      wave_tot[w] = run;
      run += x;
    }
  }
  __syncthreads();
  return incl - v + wave_tot[wave];
}

// Selected key i as written: i itself, or its mapped id (two-level Level 2).
__device__ __forceinline__ int32_t emitted(const SelectArgs& sa, int b, int i) {
  return sa.map != nullptr ? sa.map[b * sa.map_pitch + i] : i;
}

// Count of the selection of sequence b, after the window chunks that follow
// the k selected ones in mapped mode (all threads of the workgroup call it).
__device__ __forceinline__ void finish_count(const SeqTable& t, const SelectArgs& sa, int b, int k, int32_t* out,
                                             int32_t* sel_count, int tid, int nthreads) {
  int total = k;
  if (sa.map != nullptr) {
    const int w0 = t.w0[b], nw = t.win[b];
    for (int i = tid; i < nw; i += nthreads) out[k + i] = w0 + i;
    total += nw;
  }
  if (sel_count != nullptr && tid == 0) sel_count[b] = total;
}

template <int MODE, bool RECALL>
__global__ void __launch_bounds__(kThreads)
topk_kernel(SeqTable t, const uint32_t* __restrict__ scores, int32_t* __restrict__ out_idx,
            int64_t pitch_seq, int64_t pitch_q, int32_t* __restrict__ sel_count, SelectArgs sa) {
  __shared__ uint32_t keys[kLdsKeys];
  __shared__ uint32_t hist[kSubHist][256];
  __shared__ uint64_t wave_tot[kWaves];
  __shared__ uint32_t sh_digit, sh_krem, sh_k;

  const int Q = t.n_lookahead;
  const int b = blockIdx.x / Q, j = blockIdx.x % Q;
  // keys of this (sequence, query): t.n[b], or fewer when the count is on the device
  const int n = sa.dev_n != nullptr ? min(t.n[b], max(sa.dev_n[b], 0)) : t.n[b];
  int k = min(t.keep[b], n);
  const int tid = threadIdx.x;
  const uint32_t* s = scores + (int64_t)Q * t.chunk_off[b] + (int64_t)j * t.n[b];
  int32_t* out = out_idx + b * pitch_seq + j * pitch_q;
  if (k == 0) {  // no keys (uniform across the workgroup)
    finish_count(t, sa, b, 0, out, sel_count, tid, kThreads);
    return;
  }
  const bool staged = n <= kLdsKeys;
  // key of entry i; for the recall, the largest over the indexer layers
  auto key_at = [&](int i) -> uint32_t {
    uint32_t key = order_key<MODE>(s[i]);
    if constexpr (RECALL)
      for (int l = 1; l < sa.n_layers; ++l) key = max(key, order_key<MODE>(s[l * sa.layer_stride + i]));
    return key;
  };

  if (staged)
    for (int i = tid; i < n; i += kThreads) keys[i] = key_at(i);

  uint32_t prefix = 0, pmask = 0, krem = (uint32_t)k;
  uint32_t* hflat = &hist[0][0];
  const int sub = (tid >> 6) & (kSubHist - 1);
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < kSubHist * 256; i += kThreads) hflat[i] = 0u;
    __syncthreads();
    for (int i = tid; i < n; i += kThreads) {
      const uint32_t key = staged ? keys[i] : key_at(i);
      if ((key & pmask) == prefix) atomicAdd(&hist[sub][(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane l owns bins 4l .. 4l+3; find the bin holding the krem-th largest key
      uint32_t c[4], tot = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[q] = 0;
#pragma unroll
        for (int h = 0; h < kSubHist; ++h) c[q] += hist[h][4 * tid + q];
        tot += c[q];
      }
      uint32_t suffix = tot;  // sum over lanes >= this lane
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_down(suffix, off);
        if (tid + off < 64) suffix += y;
      }
      uint32_t cum = suffix - tot;  // keys in higher bins
      if constexpr (RECALL) {
        if (shift == 24) {
          // keys at or above the key of +0.0 fill bins 128 .. 255 (lanes 32 .. 63)
          krem = min(krem, (uint32_t)__shfl((int)suffix, 32));
          if (tid == 0) sh_k = krem;
        }
      }
#pragma unroll
      for (int q = 3; q >= 0; --q) {
        if (cum < krem && cum + c[q] >= krem) {
          sh_digit = 4u * tid + q;
          sh_krem = krem - cum;
        }
        cum += c[q];
      }
    }
    __syncthreads();
    if constexpr (RECALL) {
      if (shift == 24) {
        k = (int)sh_k;
        if (k == 0) {  // nothing recalled (uniform across the workgroup)
          finish_count(t, sa, b, 0, out, sel_count, tid, kThreads);
          return;
        }
      }
    }
    prefix |= sh_digit << shift;
    pmask |= 0xFFu << shift;
    krem = sh_krem;
  }
  const uint32_t T = prefix;  // k-th largest key; krem keys equal to T are kept

  // Index-order compaction over contiguous per-thread segments.
  const int seg = (n + kThreads - 1) / kThreads;
  const int i0 = min(tid * seg, n), i1 = min(i0 + seg, n);
  uint32_t gt = 0, eq = 0;
  for (int i = i0; i < i1; ++i) {
    const uint32_t key = key_at(i);
    gt += key > T;
    eq += key == T;
  }
  const uint64_t base = block_exclusive_scan(((uint64_t)gt << 32) | eq, wave_tot);
  uint32_t pgt = (uint32_t)(base >> 32), peq = (uint32_t)base;
  for (int i = i0; i < i1; ++i) {
    const uint32_t key = key_at(i);
    if (key > T) {
      const uint32_t pos = pgt + min(peq, krem);
      if (pos < (uint32_t)k) out[pos] = emitted(sa, b, i);
      ++pgt;
    } else if (key == T) {
      if (peq < krem && pgt + peq < (uint32_t)k) out[pgt + peq] = emitted(sa, b, i);
      ++peq;
    }
  }
  finish_count(t, sa, b, k, out, sel_count, tid, kThreads);
}

// ---------------------------------------------------------------------------
// LDS-resident selection for up to 16384 chunks per (sequence, query).  The
// kernel runs once per step on a single compute unit, so what it waits on is
// latency: every phase is a short chain of independent memory operations, and
// the tail of the radix select runs in one wavefront with no barriers.
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelMaxN = 16384;
constexpr int kSelKPT = kSelMaxN / kSelThreads;  // 16 keys per thread
// topk_select_kernel holds KPT keys per thread: 16 up to 16384 keys, 8 up to
// 8192, 4 up to 4096, 2 up to 2048.  On one CU every per-key instruction of the 1024 threads
// costs 16 cycles, so a short sequence does not pay for 16 slots of padding.
constexpr int kSelCand = 4096;                   // threshold-bin keys packed for the last digits
constexpr int kSelSub = 4;                       // sub-histograms of the first digit (lane / 16)

// Inclusive prefix sum across the 64 lanes of a wave with DPP row shifts and
// row broadcasts (no LDS round trips).
__device__ __forceinline__ uint32_t wave_scan_incl(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

__device__ __forceinline__ uint32_t lane_bcast(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

// One wavefront: among the keys src[0 .. m) that match (prefix, pmask), find
// the bin of the next 10-bit digit (below bit `shift`) holding the kr-th
// largest; h is a private LDS area of 1024 words and src is readable up to the
// next multiple of 512 past m.  Returns the digit and updates kr to the number
// of keys still to take from that bin.
__device__ __forceinline__ uint32_t wave_digit(const uint32_t* src, int m, uint32_t prefix, uint32_t pmask,
                                               int shift, uint32_t& kr, uint32_t* h) {
  const int lane = threadIdx.x & 63;
  uint4* h4 = reinterpret_cast<uint4*>(h) + lane * 4;  // lane l owns bins 16l .. 16l+15
#pragma unroll
  for (int q = 0; q < 4; ++q) h4[q] = make_uint4(0u, 0u, 0u, 0u);
  __builtin_amdgcn_wave_barrier();
  // candidates in batches of 8 per lane: all reads of a batch are issued
  // before its atomics
  for (int c0 = 0; c0 < m; c0 += 8 * 64) {
    uint32_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = src[c0 + u * 64 + lane];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (c0 + u * 64 + lane < m && (v[u] & pmask) == prefix) atomicAdd(&h[(v[u] >> shift) & 1023u], 1u);
  }
  __builtin_amdgcn_wave_barrier();
  uint32_t sum = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint4 x = h4[q];
    sum += x.x + x.y + x.z + x.w;
  }
  const uint32_t incl = wave_scan_incl(sum);
  const uint32_t above = lane_bcast(incl, 63) - incl;  // keys in the bins of higher lanes
  const int L = __builtin_ctzll(__ballot(above < kr && above + sum >= kr));
  const uint32_t krl = kr - lane_bcast(above, L);
  // lane i < 16 takes bin 16L + 15 - i (descending), then a row scan
  const uint32_t c = lane < 16 ? h[16 * L + 15 - lane] : 0u;
  uint32_t ci = c;
  ci += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)ci, 0x111, 0xF, 0xF, false);  // row_shr:1
  ci += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)ci, 0x112, 0xF, 0xF, false);  // row_shr:2
  ci += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)ci, 0x114, 0xF, 0xF, false);  // row_shr:4
  ci += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)ci, 0x118, 0xF, 0xF, false);  // row_shr:8
  const int i = __builtin_ctzll(__ballot(lane < 16 && ci >= krl && ci - c < krl));
  kr = krl - (lane_bcast(ci, i) - lane_bcast(c, i));
  return (uint32_t)(16 * L + 15 - i);
}

// Raw 32-bit buffer view of `bytes` bytes at p (gfx9 buffer descriptor: no
// stride, 32-bit data format); loads past the end return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_buffer(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

template <int MODE, bool RECALL, int KPT>
__global__ void __launch_bounds__(kSelThreads)
topk_select_kernel(SeqTable t, const uint32_t* __restrict__ scores, int32_t* __restrict__ out_idx,
                   int64_t pitch_seq, int64_t pitch_q, int32_t* __restrict__ sel_count, SelectArgs sa) {
  // First-digit histogram, 4 counters per bin (one per lane quarter, adjacent
  // words so that equal bins of different quarters fall in different banks).
  __shared__ __align__(16) uint32_t hist[4096 * kSelSub];
  __shared__ uint32_t cand[kSelCand + 512];  // + the read-ahead of the last batch
  __shared__ uint32_t keys[kSelMaxN];  // used only when the threshold bin is too large to pack
  __shared__ __align__(16) uint32_t tot[kSelWaves];
  __shared__ __align__(16) uint32_t bm_gt[kSelMaxN / 32];  // chunks above T, bit i % 32 of word i / 32
  __shared__ __align__(16) uint32_t bm_eq[kSelMaxN / 32];  // chunks equal to T
  __shared__ uint32_t sh[4];
  __shared__ uint32_t nonneg[kSelWaves];  // recall: keys >= the key of +0.0, per wave

  // (sequence, query) of this workgroup; the numbers of sequence 0 are loaded
  // with the query count, in one round (see seq_data)
  int Q = t.n_lookahead, nb = t.n[0], kb = t.keep[0];
  int64_t cb = t.chunk_off[0], ps = pitch_seq, pq = pitch_q;
  const uint32_t* sc = scores;
  int32_t* oi = out_idx;
  asm volatile("" : "+s"(Q), "+s"(nb), "+s"(kb));
  asm volatile("" : "+s"(cb), "+s"(ps), "+s"(pq), "+s"(sc), "+s"(oi));
  int b = 0, j = blockIdx.x;
  if (j >= Q) {
    b = j / Q;
    j -= b * Q;
    nb = t.n[b];
    kb = t.keep[b];
    cb = t.chunk_off[b];
  }
  // keys of this (sequence, query): n_b, or fewer when the count is on the device
  const int n = sa.dev_n != nullptr ? min(nb, max(sa.dev_n[b], 0)) : nb;
  int k = min(kb, n);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, sub = lane >> 4;
  const uint32_t* s = sc + (int64_t)Q * cb + (int64_t)j * nb;
  int32_t* out = oi + b * ps + j * pq;
  if (k == 0) {  // no keys (uniform across the workgroup)
    finish_count(t, sa, b, 0, out, sel_count, tid, kSelThreads);
    return;
  }

  // Key i = q * 1024 + tid sits in slot q of thread tid: coalesced buffer loads,
  // all in flight while the histogram is cleared.  Slots past the end hold key
  // 0, which no finite score maps to.  They stay out of the histogram (with
  // few real keys they would all land in bin 0 and serialise its atomics),
  // never fall in the threshold bin, and the emission drops their chunk ids.
  const __amdgpu_buffer_rsrc_t src = raw_buffer(s, (uint32_t)n * 4u);
  uint32_t kk[KPT];
#pragma unroll
  for (int q = 0; q < KPT; ++q)
    kk[q] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(src, tid * 4, q * kSelThreads * 4, 0);
  // mapped mode: the ids that the keys stand for, loaded with them and staged
  // in LDS (in the histogram's space, once it is free) for the emission
  uint32_t mp[KPT];
  if (sa.map != nullptr) {
    const __amdgpu_buffer_rsrc_t msrc = raw_buffer(sa.map + b * sa.map_pitch, (uint32_t)n * 4u);
#pragma unroll
    for (int q = 0; q < KPT; ++q)
      mp[q] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(msrc, tid * 4, q * kSelThreads * 4, 0);
  }
  if constexpr (RECALL) {
    // keys of the first layer, then the largest over the other indexer layers
#pragma unroll
    for (int q = 0; q < KPT; ++q) kk[q] = q * kSelThreads + tid < n ? order_key<MODE>(kk[q]) : 0u;
    for (int l = 1; l < sa.n_layers; ++l) {
      const __amdgpu_buffer_rsrc_t srcl = raw_buffer(s + l * sa.layer_stride, (uint32_t)n * 4u);
#pragma unroll
      for (int q = 0; q < KPT; ++q) {
        const uint32_t v = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(srcl, tid * 4, q * kSelThreads * 4, 0);
        if (q * kSelThreads + tid < n) kk[q] = max(kk[q], order_key<MODE>(v));
      }
    }
  }
#pragma unroll
  for (int q = 0; q < kSelSub; ++q)
    reinterpret_cast<uint4*>(hist)[q * kSelThreads + tid] = make_uint4(0u, 0u, 0u, 0u);
  if (tid < kSelMaxN / 128) reinterpret_cast<uint4*>(bm_eq)[tid] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();

  // First digit (top 12 bits).  The atomic returns the key's rank among the
  // keys of its bin and quarter, which later places it in the candidate list.
  // Slots past n are padding and stay out.  In the recall the keys below the
  // key of +0.0 cannot be kept (k is at most the number of the others): they
  // are set to 0, which no kept key equals there, and stay out too.
  if constexpr (RECALL) {
    uint32_t nn = 0;
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
      nn += (uint32_t)__popcll(__ballot(kk[q] >= 0x80000000u));
      kk[q] = kk[q] >= 0x80000000u ? kk[q] : 0u;
    }
    if (lane == 0) nonneg[wave] = nn;
  }
  uint32_t bin[KPT], rk[KPT];
  bool in[KPT];
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    if constexpr (MODE != kKeysReady && !RECALL) kk[q] = q * kSelThreads + tid < n ? order_key<MODE>(kk[q]) : 0u;
    in[q] = RECALL ? kk[q] != 0u : q * kSelThreads + tid < n;
    bin[q] = kk[q] >> 20;
    rk[q] = in[q] ? atomicAdd(&hist[bin[q] * kSelSub + sub], 1u) : 0u;
  }
  __syncthreads();
  if constexpr (RECALL) {
    // recalled entries: sigmoid >= 1/2, i.e. key >= key(+0.0); at most K_max = keep[b]
    const uint32_t c = lane < kSelWaves ? nonneg[lane] : 0u;
    k = min(k, (int)lane_bcast(wave_scan_incl(c), 63));
    if (k == 0) {  // nothing recalled (uniform across the workgroup)
      finish_count(t, sa, b, 0, out, sel_count, tid, kSelThreads);
      return;
    }
  }

  // Bin B0 holding the k-th largest key: thread t owns bins 4t .. 4t+3.
  {
    const uint4* h4 = reinterpret_cast<const uint4*>(hist) + 4 * tid;
    uint32_t c[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 x = h4[q];
      c[q] = x.x + x.y + x.z + x.w;
    }
    const uint32_t mine = c[0] + c[1] + c[2] + c[3];
    const uint32_t incl = wave_scan_incl(mine);
    if (lane == 63) tot[wave] = incl;
    __syncthreads();
    // keys in the bins of higher waves: lane w < 16 holds wave w's total
    const uint32_t wt = lane < kSelWaves ? tot[lane] : 0u;
    const uint32_t after = lane_bcast(wave_scan_incl(lane > wave ? wt : 0u), 63);
    uint32_t cum = after + lane_bcast(incl, 63) - incl;  // keys in the bins above this thread's
    const uint32_t kr = (uint32_t)k;
#pragma unroll
    for (int q = 3; q >= 0; --q) {
      if (cum < kr && cum + c[q] >= kr) {
        sh[0] = 4u * tid + q;
        sh[1] = kr - cum;
        sh[2] = c[q];
      }
      cum += c[q];
    }
  }
  __syncthreads();
  const uint32_t B0 = sh[0], m = sh[2];
  uint32_t krem = sh[1];

  // Keys of bin B0 to the candidate list at (keys of lower quarters) + rank.
  const bool packed = m <= (uint32_t)kSelCand;
  if (packed) {
    const uint4 bc = reinterpret_cast<const uint4*>(hist)[B0];
    const uint32_t off = (sub > 0 ? bc.x : 0u) + (sub > 1 ? bc.y : 0u) + (sub > 2 ? bc.z : 0u);
#pragma unroll
    for (int q = 0; q < KPT; ++q)
      if (in[q] && bin[q] == B0) cand[off + rk[q]] = kk[q];
  } else {
#pragma unroll
    for (int q = 0; q < KPT; ++q) keys[q * kSelThreads + tid] = kk[q];
  }
  __syncthreads();

  // Last 20 bits: two 10-bit digits resolved by wave 0 alone, over the packed
  // candidates (or over the n keys in position order when the bin was too
  // large to pack; keys set to 0 by the recall never match its prefix).
  if (wave == 0) {
    uint32_t prefix = B0 << 20, kr = krem;
    const uint32_t* cs = packed ? cand : keys;
    const int lim = packed ? (int)m : n;
    prefix |= wave_digit(cs, lim, prefix, 0xFFF00000u, 10, kr, hist) << 10;
    prefix |= wave_digit(cs, lim, prefix, 0xFFFFFC00u, 0, kr, hist);
    if (lane == 0) {
      sh[0] = prefix;
      sh[1] = kr;
    }
  }
  __syncthreads();

  // T is the k-th largest key; every key above T is kept, and the first krem
  // keys equal to T in chunk order.  The ballot of one wave and slot covers the
  // 64 consecutive chunks q * 1024 + 64 * wave + lane, so the ballots are the
  // kept bitmaps, stored by lane 0 (the equal-to-T bitmap, cleared at the
  // start, only where it is not empty).
  const uint32_t T = sh[0];
  krem = sh[1];
  uint32_t* map_lds = hist;  // free from here on
  if (sa.map != nullptr) {
#pragma unroll
    for (int q = 0; q < KPT; ++q) map_lds[q * kSelThreads + tid] = mp[q];
  }
  uint64_t* gdst = reinterpret_cast<uint64_t*>(bm_gt) + wave;
  uint64_t* edst = reinterpret_cast<uint64_t*>(bm_eq) + wave;
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    const uint64_t g = __ballot(kk[q] > T);
    const uint64_t e = __ballot(kk[q] == T);
    if (lane == 0) {
      gdst[q * kSelWaves] = g;
      if (e != 0ull) edst[q * kSelWaves] = e;
    }
  }
  __syncthreads();

  // Emission in chunk order: thread v < 512 owns chunks 32v .. 32v+31.
  const bool emits = tid < kSelMaxN / 32;
  uint32_t g = 0, e = 0;
  if (emits) {
    const int valid = n - 32 * tid;  // chunk ids past n are padding
    const uint32_t live = valid >= 32 ? 0xFFFFFFFFu : valid > 0 ? (1u << valid) - 1u : 0u;
    g = bm_gt[tid] & live;
    e = bm_eq[tid] & live;
  }
  const uint32_t cnt = ((uint32_t)__popc(g) << 16) | (uint32_t)__popc(e);  // both <= 16384
  const uint32_t incl = wave_scan_incl(cnt);
  if (lane == 63) tot[wave] = incl;
  __syncthreads();
  if (emits) {
    const uint32_t wt = lane < kSelWaves ? tot[lane] : 0u;
    const uint32_t excl = lane_bcast(wave_scan_incl(lane < wave ? wt : 0u), 63) + incl - cnt;
    const uint32_t gb = excl >> 16, eb = excl & 0xFFFFu;
    uint32_t kept = g;
    for (uint32_t r = eb < krem ? krem - eb : 0u; e != 0u && r != 0u; --r) {
      kept |= e & (0u - e);  // lowest remaining chunk equal to T
      e &= e - 1u;
    }
    uint32_t pos = gb + min(eb, krem);
    while (kept != 0u) {
      const int i = 32 * tid + __builtin_ctz(kept);
      out[pos++] = sa.map != nullptr ? (int32_t)map_lds[i] : i;
      kept &= kept - 1u;
    }
  }
  finish_count(t, sa, b, k, out, sel_count, tid, kSelThreads);
}

// Ascending union of the Q per-query lists of each sequence via an LDS bitmap.
__global__ void __launch_bounds__(kThreads)
union_kernel(SeqTable t, const int32_t* __restrict__ per_query, int32_t k_pitch,
             int32_t* __restrict__ sel_idx, int32_t sel_pitch, int32_t* __restrict__ sel_count) {
  __shared__ uint32_t bm[LSA_MAX_UNION_CHUNKS / 32];
  __shared__ uint64_t wave_tot[kWaves];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int n = t.n[b], k = t.keep[b], Q = t.n_lookahead;
  const int nw = (n + 31) / 32;
  for (int w = tid; w < nw; w += kThreads) bm[w] = 0u;
  __syncthreads();
  // the ids of 8 queries at a time, all 8 loads in flight before their atomics
  const int32_t* pq = per_query + (int64_t)b * Q * k_pitch;
  for (int j0 = 0; j0 < Q; j0 += 8) {
    for (int r = tid; r < k; r += kThreads) {
      int c[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) c[u] = j0 + u < Q ? pq[(int64_t)(j0 + u) * k_pitch + r] : -1;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if ((unsigned)c[u] < (unsigned)n) atomicOr(&bm[c[u] >> 5], 1u << (c[u] & 31));
    }
  }
  __syncthreads();
  const int seg = (nw + kThreads - 1) / kThreads;
  const int w0 = min(tid * seg, nw), w1 = min(w0 + seg, nw);
  uint32_t cnt = 0;
  for (int w = w0; w < w1; ++w) cnt += __popc(bm[w]);
  const uint64_t base = block_exclusive_scan(cnt, wave_tot);
  int32_t* out = sel_idx + (int64_t)b * sel_pitch;
  uint32_t pos = (uint32_t)base;
  for (int w = w0; w < w1; ++w) {
    uint32_t bits = bm[w];
    while (bits) {
      const int bit = __ffs(bits) - 1;
      out[pos++] = w * 32 + bit;
      bits &= bits - 1;
    }
  }
  if (tid == kThreads - 1) sel_count[b] = (int32_t)pos;
}

// ---------------------------------------------------------------------------
// Two-level selection in one workgroup per sequence (up to 16384 history
// chunks): the recall (keys >= the key of +0.0, at most K_max, the largest
// first) and the Level-2 top-k2 of the native keys among the recalled chunks,
// each as one LDS radix pass of the kind above, then the window chunks.

// Shared arrays of one selection pass.
struct SelLds {
  uint32_t* hist;   // [4096 * kSelSub]
  uint32_t* cand;   // [kSelCand + 512]
  uint32_t* keys;   // [kSelMaxN]
  uint32_t* tot;    // [kSelWaves]
  uint32_t* bm_gt;  // [kSelMaxN / 32]
  uint32_t* bm_eq;  // [kSelMaxN / 32]
  uint32_t* sh;     // [4]
};

// The k largest nonzero keys of kk (key q * 1024 + tid in slot q), 1 <= k <=
// the number of nonzero keys: afterwards bm_gt marks the keys above the k-th
// largest key T and bm_eq the keys equal to T; returns how many of the keys
// equal to T are kept (those first in position order).
__device__ __forceinline__ uint32_t select_pass(const uint32_t (&kk)[kSelKPT], uint32_t k, const SelLds& S) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, sub = lane >> 4;
#pragma unroll
  for (int q = 0; q < kSelSub; ++q)
    reinterpret_cast<uint4*>(S.hist)[q * kSelThreads + tid] = make_uint4(0u, 0u, 0u, 0u);
  if (tid < kSelMaxN / 128) reinterpret_cast<uint4*>(S.bm_eq)[tid] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  uint32_t bin[kSelKPT], rk[kSelKPT];
#pragma unroll
  for (int q = 0; q < kSelKPT; ++q) {
    bin[q] = kk[q] >> 20;
    rk[q] = kk[q] != 0u ? atomicAdd(&S.hist[bin[q] * kSelSub + sub], 1u) : 0u;
  }
  __syncthreads();
  {
    const uint4* h4 = reinterpret_cast<const uint4*>(S.hist) + 4 * tid;
    uint32_t c[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 x = h4[q];
      c[q] = x.x + x.y + x.z + x.w;
    }
    const uint32_t mine = c[0] + c[1] + c[2] + c[3];
    const uint32_t incl = wave_scan_incl(mine);
    if (lane == 63) S.tot[wave] = incl;
    __syncthreads();
    const uint32_t wt = lane < kSelWaves ? S.tot[lane] : 0u;
    const uint32_t after = lane_bcast(wave_scan_incl(lane > wave ? wt : 0u), 63);
    uint32_t cum = after + lane_bcast(incl, 63) - incl;
#pragma unroll
    for (int q = 3; q >= 0; --q) {
      if (cum < k && cum + c[q] >= k) {
        S.sh[0] = 4u * tid + q;
        S.sh[1] = k - cum;
        S.sh[2] = c[q];
      }
      cum += c[q];
    }
  }
  __syncthreads();
  const uint32_t B0 = S.sh[0], m = S.sh[2];
  const bool packed = m <= (uint32_t)kSelCand;
  if (packed) {
    const uint4 bc = reinterpret_cast<const uint4*>(S.hist)[B0];
    const uint32_t off = (sub > 0 ? bc.x : 0u) + (sub > 1 ? bc.y : 0u) + (sub > 2 ? bc.z : 0u);
#pragma unroll
    for (int q = 0; q < kSelKPT; ++q)
      if (kk[q] != 0u && bin[q] == B0) S.cand[off + rk[q]] = kk[q];
  } else {
#pragma unroll
    for (int q = 0; q < kSelKPT; ++q) S.keys[q * kSelThreads + tid] = kk[q];
  }
  __syncthreads();
  if (wave == 0) {
    uint32_t prefix = B0 << 20, kr = S.sh[1];
    const uint32_t* cs = packed ? S.cand : S.keys;
    const int lim = packed ? (int)m : kSelMaxN;
    prefix |= wave_digit(cs, lim, prefix, 0xFFF00000u, 10, kr, S.hist) << 10;
    prefix |= wave_digit(cs, lim, prefix, 0xFFFFFC00u, 0, kr, S.hist);
    if (lane == 0) {
      S.sh[0] = prefix;
      S.sh[1] = kr;
    }
  }
  __syncthreads();
  const uint32_t T = S.sh[0], krem = S.sh[1];
  uint64_t* gdst = reinterpret_cast<uint64_t*>(S.bm_gt) + wave;
  uint64_t* edst = reinterpret_cast<uint64_t*>(S.bm_eq) + wave;
#pragma unroll
  for (int q = 0; q < kSelKPT; ++q) {
    const uint64_t g = __ballot(kk[q] > T);
    const uint64_t e = __ballot(kk[q] == T);
    if (lane == 0) {
      gdst[q * kSelWaves] = g;
      if (e != 0ull) edst[q * kSelWaves] = e;
    }
  }
  __syncthreads();
  return krem;
}

// For thread v < 512 (chunks 32v .. 32v+31 of n): the kept chunks of the last
// pass -- every chunk above T and the first krem equal to T -- as a bit word,
// and its exclusive prefix count in *before.
__device__ __forceinline__ uint32_t kept_word(const SelLds& S, int n, uint32_t krem, uint32_t* before) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool mine = tid < kSelMaxN / 32;
  uint32_t g = 0, e = 0;
  if (mine) {
    const int valid = n - 32 * tid;
    const uint32_t live = valid >= 32 ? 0xFFFFFFFFu : valid > 0 ? (1u << valid) - 1u : 0u;
    g = S.bm_gt[tid] & live;
    e = S.bm_eq[tid] & live;
  }
  const uint32_t cnt = ((uint32_t)__popc(g) << 16) | (uint32_t)__popc(e);
  const uint32_t incl = wave_scan_incl(cnt);
  if (lane == 63) S.tot[wave] = incl;
  __syncthreads();
  const uint32_t wt = lane < kSelWaves ? S.tot[lane] : 0u;
  const uint32_t excl = lane_bcast(wave_scan_incl(lane < wave ? wt : 0u), 63) + incl - cnt;
  const uint32_t gb = excl >> 16, eb = excl & 0xFFFFu;
  uint32_t kept = g;
  for (uint32_t r = eb < krem ? krem - eb : 0u; e != 0u && r != 0u; --r) {
    kept |= e & (0u - e);
    e &= e - 1u;
  }
  *before = gb + min(eb, krem);
  __syncthreads();  // S.tot is reused by the next pass
  return mine ? kept : 0u;
}

__global__ void __launch_bounds__(kSelThreads)
two_level_select_kernel(SeqTable t, TwoLevelSelArgs a) {
  __shared__ __align__(16) uint32_t hist[4096 * kSelSub];
  __shared__ uint32_t cand[kSelCand + 512];
  __shared__ uint32_t keys[kSelMaxN];
  __shared__ __align__(16) uint32_t tot[kSelWaves];
  __shared__ __align__(16) uint32_t bm_gt[kSelMaxN / 32];
  __shared__ __align__(16) uint32_t bm_eq[kSelMaxN / 32];
  __shared__ uint32_t rec[kSelMaxN / 32];
  __shared__ uint32_t sh[4];
  __shared__ uint32_t nonneg[kSelWaves];
  const SelLds S{hist, cand, keys, tot, bm_gt, bm_eq, sh};

  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // the table entries and arguments needed before the first loads, in one
  // round of kernel-argument loads (see seq_data)
  int nb = t.n[b];
  int64_t cb = t.chunk_off[b];
  const uint32_t* l1 = a.l1;
  const uint32_t* l2 = a.l2;
  asm volatile("" : "+s"(nb), "+s"(cb), "+s"(l1), "+s"(l2));
  const int n = min(nb, kSelMaxN);
  int32_t* out = a.out + b * a.pitch;

  // Level-1 keys; slots past n read 0 (buffer loads past the end)
  uint32_t kk[kSelKPT];
  {
    const __amdgpu_buffer_rsrc_t src = raw_buffer(l1 + cb, (uint32_t)n * 4u);
#pragma unroll
    for (int q = 0; q < kSelKPT; ++q)
      kk[q] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(src, tid * 4, q * kSelThreads * 4, 0);
  }
  // the native keys are loaded now too, and masked once the recall is known
  uint32_t nk[kSelKPT];
  {
    const __amdgpu_buffer_rsrc_t src = raw_buffer(l2 + cb, (uint32_t)n * 4u);
#pragma unroll
    for (int q = 0; q < kSelKPT; ++q)
      nk[q] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(src, tid * 4, q * kSelThreads * 4, 0);
  }
  uint32_t nn = 0;
#pragma unroll
  for (int q = 0; q < kSelKPT; ++q) nn += (uint32_t)__popcll(__ballot(kk[q] >= 0x80000000u));
  if (lane == 0) nonneg[wave] = nn;
  __syncthreads();
  const uint32_t recalled = lane_bcast(wave_scan_incl(lane < kSelWaves ? nonneg[lane] : 0u), 63);
  const uint32_t k1 = min((uint32_t)max(t.keep[b], 0), recalled);
  uint32_t k2 = 0;
  if (k1 > 0u) {  // uniform
    // Level 1: keys below the key of +0.0 (not recalled) leave the selection
#pragma unroll
    for (int q = 0; q < kSelKPT; ++q) kk[q] = kk[q] >= 0x80000000u ? kk[q] : 0u;
    const uint32_t krem1 = select_pass(kk, k1, S);
    uint32_t unused;
    const uint32_t rw = kept_word(S, n, krem1, &unused);
    if (tid < kSelMaxN / 32) rec[tid] = rw;
    __syncthreads();
    // Level 2 over the recalled chunks
#pragma unroll
    for (int q = 0; q < kSelKPT; ++q) {
      const int pos = q * kSelThreads + tid;
      nk[q] = pos < n && ((rec[pos >> 5] >> (pos & 31)) & 1u) ? nk[q] : 0u;
    }
    k2 = min((uint32_t)max(a.keep2[b], 1), k1);
    const uint32_t krem2 = select_pass(nk, k2, S);
    uint32_t pos;
    uint32_t kept = kept_word(S, n, krem2, &pos);
    while (kept != 0u) {
      out[pos++] = 32 * tid + __builtin_ctz(kept);
      kept &= kept - 1u;
    }
  }
  const int w0 = t.w0[b], nw = t.win[b];
  for (int i = tid; i < nw; i += kSelThreads) out[k2 + i] = w0 + i;
  if (tid == 0) a.count[b] = (int32_t)k2 + nw;
}

__global__ void zero_kernel(uint4* p, size_t n16, uint8_t* tail, size_t ntail) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    p[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0 && threadIdx.x < ntail) tail[threadIdx.x] = 0;
}

}  // namespace

namespace {

template <int MODE, bool RECALL>
hipError_t launch_topk_keys(const SeqTable& t, const uint32_t* scores, int32_t* out_idx, int64_t pitch_seq,
                            int64_t pitch_q, int32_t* sel_count, const SelectArgs& sa, hipStream_t s) {
  int n_max = 0;
  for (int b = 0; b < t.batch; ++b) n_max = max(n_max, t.n[b]);
  const dim3 grid(t.batch * t.n_lookahead);
  if (n_max <= 2 * kSelThreads)
    hipLaunchKernelGGL((topk_select_kernel<MODE, RECALL, 2>), grid, dim3(kSelThreads), 0, s, t, scores, out_idx,
                       pitch_seq, pitch_q, sel_count, sa);
  else if (n_max <= 4 * kSelThreads)
    hipLaunchKernelGGL((topk_select_kernel<MODE, RECALL, 4>), grid, dim3(kSelThreads), 0, s, t, scores, out_idx,
                       pitch_seq, pitch_q, sel_count, sa);
  else if (n_max <= 8 * kSelThreads)
    hipLaunchKernelGGL((topk_select_kernel<MODE, RECALL, 8>), grid, dim3(kSelThreads), 0, s, t, scores, out_idx,
                       pitch_seq, pitch_q, sel_count, sa);
  else if (n_max <= kSelMaxN)
    hipLaunchKernelGGL((topk_select_kernel<MODE, RECALL, kSelKPT>), grid, dim3(kSelThreads), 0, s, t, scores,
                       out_idx, pitch_seq, pitch_q, sel_count, sa);
  else
    hipLaunchKernelGGL((topk_kernel<MODE, RECALL>), grid, dim3(kThreads), 0, s, t, scores, out_idx, pitch_seq,
                       pitch_q, sel_count, sa);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_topk(const SeqTable& t, int32_t emb_dtype, bool keys_ready, const void* scores,
                       int32_t* out_idx, int64_t out_pitch_seq, int64_t out_pitch_query, int32_t* sel_count,
                       hipStream_t s, const SelectArgs& sa) {
  const uint32_t* sc = static_cast<const uint32_t*>(scores);
  if (sa.recall) {
    if (keys_ready)
      return launch_topk_keys<kKeysReady, true>(t, sc, out_idx, out_pitch_seq, out_pitch_query, sel_count, sa, s);
    return launch_topk_keys<kKeysFromF32, true>(t, sc, out_idx, out_pitch_seq, out_pitch_query, sel_count, sa, s);
  }
  if (keys_ready)
    return launch_topk_keys<kKeysReady, false>(t, sc, out_idx, out_pitch_seq, out_pitch_query, sel_count, sa, s);
  if (emb_dtype == LSA_I8)
    return launch_topk_keys<kKeysFromI32, false>(t, sc, out_idx, out_pitch_seq, out_pitch_query, sel_count, sa, s);
  return launch_topk_keys<kKeysFromF32, false>(t, sc, out_idx, out_pitch_seq, out_pitch_query, sel_count, sa, s);
}

hipError_t launch_two_level_select(const SeqTable& t, const TwoLevelSelArgs& a, hipStream_t s) {
  for (int b = 0; b < t.batch; ++b)
    if (t.n[b] > kSelMaxN) return hipErrorInvalidValue;
  hipLaunchKernelGGL(two_level_select_kernel, dim3(t.batch), dim3(kSelThreads), 0, s, t, a);
  return hipGetLastError();
}

hipError_t launch_union(const SeqTable& t, const int32_t* per_query, int32_t k_pitch,
                        int32_t* sel_idx, int32_t sel_pitch, int32_t* sel_count, hipStream_t s) {
  hipLaunchKernelGGL(union_kernel, dim3(t.batch), dim3(kThreads), 0, s, t, per_query, k_pitch, sel_idx,
                     sel_pitch, sel_count);
  return hipGetLastError();
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
  const size_t n16 = bytes / 16, ntail = bytes % 16;
  size_t blocks = (n16 + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<uint4*>(p), n16,
                     static_cast<uint8_t*>(p) + n16 * 16, ntail);
  return hipGetLastError();
}

}  // namespace lsa
