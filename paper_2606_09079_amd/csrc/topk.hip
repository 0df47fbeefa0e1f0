// Step 2 of the decode hot path: keep the k highest-scoring chunks (the Top-k
// of Sec. 2.1, Eq. corecomp, with the K_max recall bound of Sec. 2.5 as k) and,
// with several lookahead queries, the union of the per-query sets (the set
// union of Sec. 2.4, Eq. union).
//
// One 1024-thread workgroup per (sequence, query).  Scores map to 32-bit keys
// whose unsigned order is the score order (fp32: -0.0 folded onto +0.0, sign
// bit set for positives, all bits flipped for negatives; int32: sign bit
// flipped).  A 4-pass, 8-bit-digit radix select over keys staged in LDS finds
// the k-th largest key T and how many keys equal to T must be taken.  The
// final pass walks the scores in index order: keys above T are kept, and keys
// equal to T are kept while the tie quota lasts, so ties go to the lower chunk
// id and the output comes out ascending with no sort.  Histograms are split
// four ways by wave to cut LDS atomic contention on concentrated digits.
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

hipError_t launch_topk(const SeqTable& t, int32_t emb_dtype, const void* scores, int32_t* out_idx,
                       int64_t out_pitch_seq, int64_t out_pitch_query, int32_t* sel_count,
                       hipStream_t s) {
  const dim3 grid(t.batch * t.n_lookahead);
  if (emb_dtype == LSA_I8)
    hipLaunchKernelGGL(topk_kernel<true>, grid, dim3(kThreads), 0, s, t,
                       static_cast<const uint32_t*>(scores), out_idx, out_pitch_seq, out_pitch_query,
                       sel_count);
  else
    hipLaunchKernelGGL(topk_kernel<false>, grid, dim3(kThreads), 0, s, t,
                       static_cast<const uint32_t*>(scores), out_idx, out_pitch_seq, out_pitch_query,
                       sel_count);
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
