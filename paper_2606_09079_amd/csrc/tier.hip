// Host tier (Sec. 2.5): the full K/V cache lives in a pinned host mirror and
// only the recalled chunks are materialised, in a GPU reserve of chunk slots
// that attention then reads.
//
// tier_plan_kernel -- residency plan, one workgroup per sequence.  A kept
//   chunk that a slot already holds keeps that slot.  The other kept chunks
//   take, in ascending chunk order, the free slots in ascending slot order.  A
//   slot is free when no kept chunk holds it and the previous kept set does not
//   read it, so decode can keep reading the previous set while the new one is
//   copied in.  The kernel writes each kept chunk's slot, the (chunk, slot)
//   copies to make, and the new slot owners.
//   Per-sequence state is in LDS as bitmaps over chunk ids and slot ids:
//     kbit  kept chunks; the rank of a chunk among them (a word prefix count
//           plus a popcount) is its position in the ascending kept list
//     mbit  kept chunks that no slot holds (the copies to make)
//     pbit  protected slots (held by a kept chunk or read by the previous set)
// tier_fetch_kernel -- a few workgroups per sequence move the chunk-head
//   blocks of the copy list from the host mirror into their slots.  The reads
//   cross PCIe: the mirror is pinned host memory mapped into the GPU's address
//   space, so the copy list never has to go back to the host.
#include "lsa_internal.h"

namespace lsa {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kChunkWords = kMaxTierChunks / 32;
constexpr int kSlotWords = kMaxTierSlots / 32;
constexpr int kFetchWorkgroups = 32;  // default copy workgroups per launch (at least one per sequence)

// Exclusive prefix sum over the workgroup (one value per thread); *total
// receives the sum of all values.
__device__ __forceinline__ uint32_t block_scan(uint32_t v, uint32_t* wave_tot, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wave_tot[wave] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t x = wave_tot[w];
    before += w < wave ? x : 0u;
    all += x;
  }
  __syncthreads();  // wave_tot is reused by the next scan
  *total = all;
  return before + incl - v;
}

__device__ __forceinline__ bool test_bit(const uint32_t* bits, int i) { return (bits[i >> 5] >> (i & 31)) & 1u; }

__global__ void __launch_bounds__(kThreads)
tier_plan_kernel(SeqTable t, TierArgs a) {
  __shared__ uint32_t kbit[kChunkWords];
  __shared__ uint32_t kpref[kChunkWords];
  __shared__ uint32_t mbit[kChunkWords];
  __shared__ uint32_t pbit[kSlotWords];
  __shared__ uint32_t wave_tot[kWaves];

  const int b = blockIdx.x, tid = threadIdx.x;
  const int n = t.n[b];
  const int S = a.slots[b];
  const int nw = (n + 31) / 32, sw = (S + 31) / 32;
  const int m = min(max(a.kept_count[b], 0), a.pitch);
  const int mo = a.prev_slots != nullptr ? min(max(a.prev_count[b], 0), a.pitch) : 0;
  const int32_t* kept = a.kept + (int64_t)b * a.pitch;
  int32_t* owner = a.owner + a.slot_off[b];
  int32_t* slot_idx = a.slot_idx + (int64_t)b * a.pitch;
  int32_t* fetch = a.fetch + (int64_t)b * a.pitch * 2;

  for (int w = tid; w < nw; w += kThreads) kbit[w] = 0u;
  for (int w = tid; w < sw; w += kThreads) pbit[w] = 0u;
  __syncthreads();
  for (int i = tid; i < m; i += kThreads) {
    const int c = kept[i];
    if (c >= 0 && c < n) atomicOr(&kbit[c >> 5], 1u << (c & 31));
    slot_idx[i] = -1;  // stays -1 only for an id outside 0 .. n_b - 1
  }
  for (int i = tid; i < mo; i += kThreads) {
    const int s = a.prev_slots[(int64_t)b * a.pitch + i];
    if (s >= 0 && s < S) atomicOr(&pbit[s >> 5], 1u << (s & 31));
  }
  __syncthreads();

  // word prefix counts of kbit; thread tid owns words [w0, w1)
  const int wseg = (nw + kThreads - 1) / kThreads;
  const int w0 = min(tid * wseg, nw), w1 = min(w0 + wseg, nw);
  uint32_t cnt = 0;
  for (int w = w0; w < w1; ++w) cnt += __popc(kbit[w]);
  uint32_t n_kept;
  uint32_t run = block_scan(cnt, wave_tot, &n_kept);
  for (int w = w0; w < w1; ++w) {
    kpref[w] = run;
    mbit[w] = kbit[w];
    run += __popc(kbit[w]);
  }
  __syncthreads();

  // resident kept chunks keep their slot
  for (int s = tid; s < S; s += kThreads) {
    const int c = owner[s];
    if (c >= 0 && c < n && test_bit(kbit, c)) {
      const uint32_t below = kbit[c >> 5] & ((1u << (c & 31)) - 1u);
      slot_idx[kpref[c >> 5] + __popc(below)] = s;
      atomicAnd(&mbit[c >> 5], ~(1u << (c & 31)));
      atomicOr(&pbit[s >> 5], 1u << (s & 31));
    }
  }
  __syncthreads();

  // ranks of the chunks to copy (chunk order) and of the free slots (slot order)
  uint32_t miss = 0;
  for (int w = w0; w < w1; ++w) miss += __popc(mbit[w]);
  uint32_t n_miss;
  const uint32_t miss_before = block_scan(miss, wave_tot, &n_miss);
  const int sseg = (sw + kThreads - 1) / kThreads;
  const int v0 = min(tid * sseg, sw), v1 = min(v0 + sseg, sw);
  uint32_t nfree = 0;
  for (int w = v0; w < v1; ++w) {
    const uint32_t valid = (w == sw - 1 && (S & 31)) ? (1u << (S & 31)) - 1u : 0xFFFFFFFFu;
    nfree += __popc(~pbit[w] & valid);
  }
  uint32_t n_free;
  uint32_t r = block_scan(nfree, wave_tot, &n_free);
  if (n_free < n_miss) {  // reserve too small: owners untouched, no copies
    if (tid == 0) a.fetch_count[b] = -1;
    return;
  }
  // the first n_miss free slots, ascending, into the slot column of the copy list
  for (int w = v0; w < v1 && r < n_miss; ++w) {
    const uint32_t valid = (w == sw - 1 && (S & 31)) ? (1u << (S & 31)) - 1u : 0xFFFFFFFFu;
    uint32_t f = ~pbit[w] & valid;
    while (f != 0u && r < n_miss) {
      const int s = 32 * w + __builtin_ctz(f);
      f &= f - 1u;
      fetch[2 * r + 1] = s;
      ++r;
    }
  }
  __syncthreads();  // the slot column is read back by other waves of this workgroup

  uint32_t fi = miss_before;
  for (int w = w0; w < w1; ++w) {
    uint32_t mm = mbit[w];
    while (mm != 0u) {
      const int bit = __builtin_ctz(mm);
      mm &= mm - 1u;
      const int c = 32 * w + bit;
      const int s = fetch[2 * fi + 1];
      fetch[2 * fi] = c;
      owner[s] = c;
      slot_idx[kpref[w] + __popc(kbit[w] & ((1u << bit) - 1u))] = s;
      ++fi;
    }
  }
  if (tid == 0) a.fetch_count[b] = (int32_t)n_miss;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Copy block j of sequence blockIdx.y is (copy f, KV head g, K or V) with j =
// (f * Hkv + g) * 2 + kv; a few workgroups per sequence loop over the blocks,
// so that a copy that overlaps decode leaves the compute units to the
// attention (the PCIe link, not the number of workgroups, bounds the copy).
// 256 threads move one C x 128 bf16 block, 16 bytes per thread per round,
// every load of the block issued before its stores.
template <int C>
__global__ void __launch_bounds__(256)
tier_fetch_kernel(SeqTable t, TierFetchArgs a) {
  constexpr int kRounds = C * kHeadDim * 2 / 16 / 256;
  const int b = blockIdx.y;
  const int nf = min(max(a.fetch_count[b], 0), a.pitch);
  const int n_blocks = nf * a.n_kv_heads * 2;
  for (int j = blockIdx.x; j < n_blocks; j += gridDim.x) {
    const int kv = j & 1, g = (j >> 1) % a.n_kv_heads, f = (j >> 1) / a.n_kv_heads;
    const int32_t* fe = a.fetch + ((int64_t)b * a.pitch + f) * 2;
    const int c = min(max(fe[0], 0), t.n[b] - 1);
    const int s = min(max(fe[1], 0), a.slots[b] - 1);
    const u32x4* src = reinterpret_cast<const u32x4*>((kv ? a.host_v : a.host_k) +
                                                      (t.chunk_off[b] + c) * a.chunk_stride + g * a.head_stride);
    u32x4* dst = reinterpret_cast<u32x4*>((kv ? a.res_v : a.res_k) +
                                          ((int64_t)a.slot_off[b] + s) * a.res_slot_stride +
                                          (int64_t)g * C * kHeadDim);
    u32x4 v[kRounds];
#pragma unroll
    for (int r = 0; r < kRounds; ++r) v[r] = __builtin_nontemporal_load(src + r * 256 + threadIdx.x);
#pragma unroll
    for (int r = 0; r < kRounds; ++r) dst[r * 256 + threadIdx.x] = v[r];
  }
}

__global__ void __launch_bounds__(256) tier_reset_kernel(int32_t* owner, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) owner[i] = -1;
}

}  // namespace

hipError_t launch_tier_plan(const SeqTable& t, const TierArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(tier_plan_kernel, dim3(t.batch), dim3(kThreads), 0, s, t, a);
  return hipGetLastError();
}

hipError_t launch_tier_fetch(const SeqTable& t, const TierFetchArgs& a, int32_t chunk_size, hipStream_t s) {
  const int64_t blocks = (int64_t)a.pitch * a.n_kv_heads * 2;
  if (blocks == 0) return hipSuccess;
  const int wgs = a.workgroups > 0 ? a.workgroups : kFetchWorkgroups;
  const int64_t per_seq = std::min<int64_t>(blocks, std::max(1, wgs / t.batch));
  const dim3 grid((unsigned)per_seq, (unsigned)t.batch);
  if (chunk_size == 64)
    hipLaunchKernelGGL(tier_fetch_kernel<64>, grid, dim3(256), 0, s, t, a);
  else
    hipLaunchKernelGGL(tier_fetch_kernel<128>, grid, dim3(256), 0, s, t, a);
  return hipGetLastError();
}

hipError_t launch_tier_reset(int32_t* owner, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 1024);
  hipLaunchKernelGGL(tier_reset_kernel, dim3((unsigned)blocks), dim3(256), 0, s, owner, n);
  return hipGetLastError();
}

}  // namespace lsa
