// Step 2 of the decode hot path: keep the k highest-scoring chunks (the Top-k
// of Sec. 2.1, Eq. 6, with the K_max recall bound of Sec. 2.5 as k) and,
// with several lookahead queries, the union of the per-query sets (the set
// union of Sec. 2.4, Eq. 13).
//
// One 1024-thread workgroup per (sequence, query).  Scores map to 32-bit keys
// whose unsigned order is the score order (fp32: -0.0 folded onto +0.0, sign
// bit set for positives, all bits flipped for negatives; int32: sign bit
// flipped).  A radix select finds the k-th largest key T and how many keys
// equal to T must be taken; the compaction then walks the keys in index order,
// keeping keys above T and keys equal to T while the tie quota lasts, so ties
// go to the lower chunk id and the output comes out ascending with no sort.
//
// topk_select_kernel (up to 16384 chunks): every key is loaded once into LDS
//   (16 per thread, all loads in flight together).  The first digit is the top
//   12 bits (4096-bin histogram); the keys of the threshold bin are then packed
//   into a candidate list, and the last 20 bits are resolved with 12- and 8-bit
//   digits over that list only (over all keys if the bin holds more than 4096).
//   The compaction scans each thread's contiguous 16-key segment.
// topk_kernel (longer contexts): 8-bit digits, with the keys staged in LDS when
//   they fit and re-read from memory in every pass otherwise.
#include "lsa_internal.h"

namespace lsa {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kLdsKeys = 16384;
constexpr int kSubHist = 4;

template <bool INT_KEYS>
__device__ __forceinline__ uint32_t order_key(uint32_t bits) {
  if constexpr (INT_KEYS) {
    return bits ^ 0x80000000u;
  } else {
    if (bits == 0x80000000u) bits = 0u;  // -0.0 ties +0.0
    return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
  }
}

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

template <bool INT_KEYS>
__global__ void __launch_bounds__(kThreads)
topk_kernel(SeqTable t, const uint32_t* __restrict__ scores, int32_t* __restrict__ out_idx,
            int64_t pitch_seq, int64_t pitch_q, int32_t* __restrict__ sel_count) {
  __shared__ uint32_t keys[kLdsKeys];
  __shared__ uint32_t hist[kSubHist][256];
  __shared__ uint64_t wave_tot[kWaves];
  __shared__ uint32_t sh_digit, sh_krem;

  const int Q = t.n_lookahead;
  const int b = blockIdx.x / Q, j = blockIdx.x % Q;
  const int n = t.n[b], k = t.keep[b];
  const int tid = threadIdx.x;
  const uint32_t* s = scores + (int64_t)Q * t.chunk_off[b] + (int64_t)j * n;
  int32_t* out = out_idx + b * pitch_seq + j * pitch_q;
  const bool staged = n <= kLdsKeys;

  if (staged)
    for (int i = tid; i < n; i += kThreads) keys[i] = order_key<INT_KEYS>(s[i]);

  uint32_t prefix = 0, pmask = 0, krem = (uint32_t)k;
  uint32_t* hflat = &hist[0][0];
  const int sub = (tid >> 6) & (kSubHist - 1);
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < kSubHist * 256; i += kThreads) hflat[i] = 0u;
    __syncthreads();
    for (int i = tid; i < n; i += kThreads) {
      const uint32_t key = staged ? keys[i] : order_key<INT_KEYS>(s[i]);
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
    const uint32_t key = order_key<INT_KEYS>(s[i]);
    gt += key > T;
    eq += key == T;
  }
  const uint64_t base = block_exclusive_scan(((uint64_t)gt << 32) | eq, wave_tot);
  uint32_t pgt = (uint32_t)(base >> 32), peq = (uint32_t)base;
  for (int i = i0; i < i1; ++i) {
    const uint32_t key = order_key<INT_KEYS>(s[i]);
    if (key > T) {
      const uint32_t pos = pgt + min(peq, krem);
      if (pos < (uint32_t)k) out[pos] = i;
      ++pgt;
    } else if (key == T) {
      if (peq < krem && pgt + peq < (uint32_t)k) out[pgt + peq] = i;
      ++peq;
    }
  }
  if (sel_count != nullptr && tid == 0) sel_count[b] = k;
}

// ---------------------------------------------------------------------------
// LDS-resident selection for up to 16384 chunks per (sequence, query).  The
// kernel runs once per step, so its code is kept compact (loops, not long
// unrolled straight-line code): instruction fetch, not arithmetic, is what a
// single-pass workgroup waits on.
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelMaxN = 16384;
constexpr int kSelKPT = kSelMaxN / kSelThreads;  // 16 keys per thread
constexpr int kSelCand = 4096;                   // threshold-bin keys packed for the last digits

// key i lives at LDS word i + i / 16, so the 16 keys of one thread's segment
// (read in the compaction) spread over the banks
__device__ __forceinline__ int kpos(int i) { return i + (i >> 4); }

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

// Inclusive prefix sum over the workgroup; *total receives the block sum.
__device__ __forceinline__ uint32_t sel_scan(uint32_t v, uint32_t* wave_tot, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t incl = wave_scan_incl(v);
  if (lane == 63) wave_tot[wave] = incl;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll 4
  for (int w = 0; w < kSelWaves; ++w) {
    const uint32_t x = wave_tot[w];
    before += (w < wave) ? x : 0u;
    tot += x;
  }
  *total = tot;
  __syncthreads();  // wave_tot is reused by the next scan
  return incl + before;
}

// Among 4096 bins (thread t owns bins 4t .. 4t+3), the bin holding the
// krem-th largest counted key, the keys to take from it and its size, written
// to LDS and read by every thread after the call.
__device__ __forceinline__ void sel_find_bin(const uint32_t* hist, uint32_t krem, uint32_t* wave_tot,
                                             uint32_t* sh) {
  const int tid = threadIdx.x;
  const uint4 c4 = reinterpret_cast<const uint4*>(hist)[tid];
  const uint32_t c[4] = {c4.x, c4.y, c4.z, c4.w};
  uint32_t total;
  const uint32_t incl = sel_scan(c4.x + c4.y + c4.z + c4.w, wave_tot, &total);
  uint32_t cum = total - incl;  // keys in bins above this thread's
  for (int q = 3; q >= 0; --q) {
    if (cum < krem && cum + c[q] >= krem) {
      sh[0] = 4u * tid + q;
      sh[1] = krem - cum;
      sh[2] = c[q];
    }
    cum += c[q];
  }
  __syncthreads();
}

template <bool INT_KEYS>
__global__ void __launch_bounds__(kSelThreads)
topk_select_kernel(SeqTable t, const uint32_t* __restrict__ scores, int32_t* __restrict__ out_idx,
                   int64_t pitch_seq, int64_t pitch_q, int32_t* __restrict__ sel_count) {
  __shared__ uint32_t keys[kSelMaxN + kSelMaxN / 16];
  __shared__ uint32_t hist[4096];
  __shared__ uint32_t cand[kSelCand];
  __shared__ uint32_t wave_tot[kSelWaves];
  __shared__ uint32_t sh[4];

  const int Q = t.n_lookahead;
  const int b = blockIdx.x / Q, j = blockIdx.x % Q;
  const int n = t.n[b], k = t.keep[b];
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t* s = scores + (int64_t)Q * t.chunk_off[b] + (int64_t)j * n;
  int32_t* out = out_idx + b * pitch_seq + j * pitch_q;

  reinterpret_cast<uint4*>(hist)[tid] = make_uint4(0u, 0u, 0u, 0u);
  if (tid == 0) sh[3] = 0u;
  __syncthreads();

  // Coalesced loads, all issued before use (indices clamped into range), then
  // keys to LDS and the histogram of their top 12 bits.  Keys past the end are
  // 0 (the smallest key): never above the threshold and, having the highest
  // chunk ids, never reached by the tie quota (which counts real keys only).
  {
    uint32_t raw[kSelKPT];
#pragma unroll
    for (int q = 0; q < kSelKPT; ++q) raw[q] = s[min(q * kSelThreads + tid, n - 1)];
#pragma unroll
    for (int q = 0; q < kSelKPT; ++q) {
      const int i = q * kSelThreads + tid;
      const uint32_t kk = i < n ? order_key<INT_KEYS>(raw[q]) : 0u;
      keys[kpos(i)] = kk;
      if (i < n) atomicAdd(&hist[kk >> 20], 1u);
    }
  }
  __syncthreads();

  sel_find_bin(hist, (uint32_t)k, wave_tot, sh);
  const uint32_t B0 = sh[0], m = sh[2];
  uint32_t krem = sh[1];
  uint32_t prefix = B0 << 20, pmask = 0xFFF00000u;

  // Remaining 20 bits: two more radix digits (12 and 8 bits) under prefix B0.
  // The keys of bin B0 are first packed into LDS (one atomic per wave and
  // iteration) when they fit, so those passes touch only them.
  const bool packed = m <= (uint32_t)kSelCand;
  if (packed) {
    __syncthreads();  // sh[] has been read by every thread
#pragma unroll 1
    for (int q = 0; q < kSelKPT; ++q) {
      const int i = q * kSelThreads + tid;
      const uint32_t kk = keys[kpos(i)];
      const bool pred = i < n && (kk >> 20) == B0;
      const uint64_t mask = __ballot(pred);
      if (mask == 0ull) continue;
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(&sh[3], (uint32_t)__popcll(mask));
      base = __shfl(base, 0);
      if (pred)
        cand[base + __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u))] = kk;
    }
  }
#pragma unroll 1
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 8 : 0;
    const uint32_t dmask = pass == 0 ? 0xFFFu : 0xFFu;
    reinterpret_cast<uint4*>(hist)[tid] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    if (packed) {
      for (int c = tid; c < (int)m; c += kSelThreads) {
        const uint32_t kk = cand[c];
        if ((kk & pmask) == prefix) atomicAdd(&hist[(kk >> shift) & dmask], 1u);
      }
    } else {
      for (int i = tid; i < n; i += kSelThreads) {
        const uint32_t kk = keys[kpos(i)];
        if ((kk & pmask) == prefix) atomicAdd(&hist[(kk >> shift) & dmask], 1u);
      }
    }
    __syncthreads();
    sel_find_bin(hist, krem, wave_tot, sh);
    prefix |= sh[0] << shift;
    pmask |= dmask << shift;
    krem = sh[1];
    __syncthreads();
  }

  // T is the k-th largest key; every key above T is kept, and the first krem
  // keys equal to T in chunk order.  Thread t walks its segment [16t, 16t+16).
  const uint32_t T = prefix;
  const int i0 = tid * kSelKPT;
  uint32_t gt = 0, eq = 0;
#pragma unroll 4
  for (int q = 0; q < kSelKPT; ++q) {
    const uint32_t kk = keys[kpos(i0 + q)];
    gt += kk > T;
    eq += kk == T;
  }
  uint32_t tot2;
  const uint32_t both = sel_scan((gt << 16) | eq, wave_tot, &tot2) - ((gt << 16) | eq);
  uint32_t pgt = both >> 16, peq = both & 0xFFFFu;
#pragma unroll 1
  for (int q = 0; q < kSelKPT; ++q) {
    const uint32_t kk = keys[kpos(i0 + q)];
    const bool g1 = kk > T, e1 = kk == T;
    const uint32_t pos = pgt + min(peq, krem);
    if ((g1 || (e1 && peq < krem)) && pos < (uint32_t)k) out[pos] = i0 + q;
    pgt += g1;
    peq += e1;
  }
  if (sel_count != nullptr && tid == 0) sel_count[b] = k;
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
  const int32_t* pq = per_query + (int64_t)b * Q * k_pitch;
  for (int i = tid; i < Q * k; i += kThreads) {
    const int c = pq[(int64_t)(i / k) * k_pitch + i % k];
    if ((unsigned)c < (unsigned)n) atomicOr(&bm[c >> 5], 1u << (c & 31));
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

__global__ void zero_kernel(uint4* p, size_t n16, uint8_t* tail, size_t ntail) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    p[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0 && threadIdx.x < ntail) tail[threadIdx.x] = 0;
}

}  // namespace

namespace {

template <bool INT_KEYS>
hipError_t launch_topk_keys(const SeqTable& t, const uint32_t* scores, int32_t* out_idx, int64_t pitch_seq,
                            int64_t pitch_q, int32_t* sel_count, hipStream_t s) {
  int n_max = 0;
  for (int b = 0; b < t.batch; ++b) n_max = max(n_max, t.n[b]);
  const dim3 grid(t.batch * t.n_lookahead);
  if (n_max <= kSelMaxN)
    hipLaunchKernelGGL((topk_select_kernel<INT_KEYS>), grid, dim3(kSelThreads), 0, s, t, scores, out_idx,
                       pitch_seq, pitch_q, sel_count);
  else
    hipLaunchKernelGGL((topk_kernel<INT_KEYS>), grid, dim3(kThreads), 0, s, t, scores, out_idx, pitch_seq,
                       pitch_q, sel_count);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_topk(const SeqTable& t, int32_t emb_dtype, const void* scores, int32_t* out_idx,
                       int64_t out_pitch_seq, int64_t out_pitch_query, int32_t* sel_count,
                       hipStream_t s) {
  const uint32_t* sc = static_cast<const uint32_t*>(scores);
  if (emb_dtype == LSA_I8) return launch_topk_keys<true>(t, sc, out_idx, out_pitch_seq, out_pitch_query, sel_count, s);
  return launch_topk_keys<false>(t, sc, out_idx, out_pitch_seq, out_pitch_query, sel_count, s);
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
