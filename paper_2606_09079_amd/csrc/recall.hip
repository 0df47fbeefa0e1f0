// Recall path, step R1: the full Memory Indexer score (Sec. 2.1, Eq. 4, the
// argument of the sigmoid) of every compressed entry s of a sequence, for each
// of L indexer layers:
//   x_l[s] = sum_h w_l[h] * ReLU(q_l[h] . K_l[s])
// Layer l recalls s when sigmoid(x_l[s]) >= 1/2, that is x_l[s] >= 0 (Eq. 5),
// and the recalled set is the OR over the layers (Eq. 13), so the selection
// only needs r[s] = max_l x_l[s]: s is recalled exactly when r[s] >= 0, and the
// K_max bound (Sec. 2.5) keeps the entries with the largest r.
//
// The per-layer product [n_h x c] x [c x n_b] is a dense contraction, so it
// runs on v_mfma_f32_16x16x32_bf16 with the queries as the A operand (16 heads
// per block) and the index keys as the B operand (16 entries per wave).  After
// the c / 32 steps each lane holds the dot products of 4 heads with one entry,
// applies ReLU and its gates, and two xor shuffles finish the sum over heads.
//
// One workgroup of 4 waves covers 64 entries of one sequence.  It first copies
// the sequence's queries from HBM straight into LDS (global->LDS copies), laid
// out in MFMA operand order: each 1 KiB block is the A operand of one (layer,
// 16-head block, k-step), so every operand is one conflict-free 16-byte LDS
// read per lane.  Then it issues the loads of all its index keys, every layer.
// Vector loads complete in order, so the barrier after the copy waits only for
// the queries, and the products of layer l start as soon as layer l's keys are
// in while later layers' keys are still arriving.
#include "lsa_internal.h"

namespace lsa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = kRecallThreads;
constexpr int kWaves = kThreads / 64;

// s_waitcnt immediates (gfx9 encoding): at most n vector loads of this wave
// outstanding, or no LDS operation outstanding
constexpr int waitcnt_vm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }
constexpr int kWaitLds = 0xF | (0x3 << 14) | (0x7 << 4);

// The A operands of kBlocks MFMAs, one 1 KiB staged block each, read as one
// assembly block that ends with its own LDS wait (the compiler would otherwise
// make the first read wait for every vector load still in flight, since it
// cannot tell these reads from the global->LDS copies).
template <int N>
__device__ __forceinline__ void read_blocks(const uint4 (*blocks)[64], int first, int lane, bf16x8 (&out)[N]) {
  static_assert(N == 1 || N == 2 || N == 4, "1, 2 or 4 blocks");
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)&blocks[first][lane];
  uint4 v[N];
  if constexpr (N == 1) {
    asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=&v"(v[0]) : "v"(a) : "memory");
  } else if constexpr (N == 2) {
    asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %2 offset:1024\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(v[0]), "=&v"(v[1]) : "v"(a) : "memory");
  } else {
    asm volatile(
        "ds_read_b128 %0, %4\n\tds_read_b128 %1, %4 offset:1024\n\t"
        "ds_read_b128 %2, %4 offset:2048\n\tds_read_b128 %3, %4 offset:3072\n\ts_waitcnt lgkmcnt(0)"
        : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]) : "v"(a) : "memory");
  }
#pragma unroll
  for (int i = 0; i < N; ++i) out[i] = __builtin_bit_cast(bf16x8, v[i]);
}

// What the kernel writes: every layer's score x_l; the order key of max_l x_l
// per entry; or, in list mode, that key per listed entry.
enum RecallOut : int { kOutScores = 0, kOutKeys = 1, kOutListKeys = 2 };

template <int NH, int CD, int OUT>
__global__ void __launch_bounds__(kThreads)
recall_score_kernel(SeqTable t, RecallArgs r, void* __restrict__ out) {
  constexpr int kSteps = CD / 32;   // MFMA k-steps
  constexpr int kBlocks = NH / 16;  // 16-head blocks
  constexpr int kMaxStaged = kMaxIdxLayers * kBlocks * kSteps;
  // staged block (l, hb, st) at index (l * kSteps + st) * kBlocks + hb: the
  // kBlocks operands of one k-step are adjacent
  __shared__ uint4 sq[kMaxStaged][64];
  __shared__ float sw[kMaxIdxLayers * NH];

  const int L = r.n_layers;
  // keys mode with a native indexer: one more layer, scored but not max-ed
  const int NAT = (OUT == kOutKeys && r.nat_out != nullptr) ? 1 : 0;
  const int LT = L + NAT;
  const int wg = blockIdx.x;
  const SeqData sd = seq_data(t, t.score_wg_off, wg);
  const int b = sd.b;
  // entries of sequence b; in list mode t.n[b] is the list capacity and the
  // count is on the device
  const int n = OUT == kOutListKeys ? min(sd.n, max(r.list_count[b], 0)) : sd.n;
  if ((wg - sd.wg0) * kRecallRowsPerWg >= n) return;  // the whole workgroup: nothing to score
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int e0 = (wg - sd.wg0) * kRecallRowsPerWg + wave * 16;
  const int hi = lane >> 4;  // this lane's k-slice 8 hi .. 8 hi + 7 of every 32-wide step

  // queries -> LDS in operand order: lane i of block (l, hb, st) holds
  // q_l[16 hb + i % 16][32 st + 8 (i / 16) .. + 7]
  const int n_staged = LT * kBlocks * kSteps;
  const uint16_t* qb = r.q + (int64_t)b * L * NH * CD + (lane & 15) * CD + 8 * hi;
  const uint16_t* qn = NAT ? r.nat_q + (int64_t)b * NH * CD + (lane & 15) * CD + 8 * hi : qb;
  for (int blk = wave; blk < n_staged; blk += kWaves) {  // wave-uniform
    const int st = (blk / kBlocks) % kSteps, hb = blk % kBlocks, l = blk / (kBlocks * kSteps);
    const uint16_t* src = l < L ? qb + (l * NH + 16 * hb) * CD + 32 * st : qn + (16 * hb) * CD + 32 * st;
    __builtin_amdgcn_global_load_lds((const void*)src, (void __attribute__((address_space(3)))*)&sq[blk][0], 16, 0,
                                     0);
  }
  // LT * NH <= kThreads
  const float gate = tid < L * NH ? r.w[(int64_t)b * L * NH + tid]
                     : NAT ? r.nat_w[(int64_t)b * NH + min(tid - L * NH, NH - 1)]
                           : r.w[(int64_t)b * L * NH + L * NH - 1];

  // B operands: entry e0 + lane % 16 (clamped; its result is not stored), dims
  // 32 st + 8 hi .. + 7, every layer (layers past L re-read layer 0 and are
  // not used, so that the loads need no branches)
  constexpr int kKeyLoads = kMaxIdxLayers * kSteps;
  bf16x8 kb[kMaxIdxLayers][kSteps];
  {
    const int pos = min(e0 + (lane & 15), n - 1);
    // a list id is clamped into the key array (its score is then meaningless)
    const int ent = OUT == kOutListKeys
                        ? min(max(r.list[b * r.list_pitch + pos], 0), (int)(r.total - 1 - sd.chunk_off))
                        : pos;
    const uint16_t* kp = r.k + (sd.chunk_off + ent) * CD + 8 * hi;
    const uint16_t* kn = NAT ? r.nat_k + (sd.chunk_off + ent) * CD + 8 * hi : kp;
#pragma unroll
    for (int l = 0; l < kMaxIdxLayers; ++l) {
      const uint16_t* kl = l < L ? kp + l * r.layer_stride : l == L ? kn : kp;
#pragma unroll
      for (int st = 0; st < kSteps; ++st)
        kb[l][st] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(kl + 32 * st));
    }
  }

  // the copies and the gate are in once at most the key loads are outstanding
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(kKeyLoads));
  if (tid < LT * NH) sw[tid] = gate;
  __builtin_amdgcn_s_waitcnt(kWaitLds);
  __asm__ volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  __asm__ volatile("" ::: "memory");
  if (e0 >= n) return;

  float best = -INFINITY, native = 0.f;
#pragma unroll
  for (int l = 0; l < kMaxIdxLayers; ++l) {
    if (l >= LT) break;
    f32x4 acc[kBlocks];
#pragma unroll
    for (int hb = 0; hb < kBlocks; ++hb) acc[hb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      bf16x8 a[kBlocks];  // A operands: heads 16 hb + lane % 16, dims 32 st + 8 hi .. + 7
      read_blocks<kBlocks>(sq, (l * kSteps + st) * kBlocks, lane, a);
#pragma unroll
      for (int hb = 0; hb < kBlocks; ++hb)
        acc[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[hb], kb[l][st], acc[hb], 0, 0, 0);
    }
    // acc[hb][j] = q_l[16 hb + 4 hi + j] . K_l[e0 + lane % 16]
    float x = 0.f;
#pragma unroll
    for (int hb = 0; hb < kBlocks; ++hb)
#pragma unroll
      for (int j = 0; j < 4; ++j) x = fmaf(sw[l * NH + 16 * hb + 4 * hi + j], fmaxf(acc[hb][j], 0.f), x);
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    if constexpr (OUT == kOutScores) {
      if (lane < 16 && e0 + lane < n)
        static_cast<float*>(out)[l * r.total + sd.chunk_off + e0 + lane] = x;
    }
    if (l < L) best = fmaxf(best, x);
    else native = x;
  }
  if constexpr (OUT != kOutScores) {
    const int64_t base = OUT == kOutListKeys ? b * r.list_pitch : sd.chunk_off;
    if (lane < 16 && e0 + lane < n)
      static_cast<uint32_t*>(out)[base + e0 + lane] = order_key<kKeysFromF32>(__float_as_uint(best));
    if (NAT && lane < 16 && e0 + lane < n)
      r.nat_out[sd.chunk_off + e0 + lane] = order_key<kKeysFromF32>(__float_as_uint(native));
  }
}

template <int NH, int CD>
hipError_t launch_nh_cd(const SeqTable& t, const RecallArgs& r, void* out, bool keys, hipStream_t s) {
  const dim3 grid(t.score_wg_off[t.batch]);
  if (r.list != nullptr)
    hipLaunchKernelGGL((recall_score_kernel<NH, CD, kOutListKeys>), grid, dim3(kThreads), 0, s, t, r, out);
  else if (keys)
    hipLaunchKernelGGL((recall_score_kernel<NH, CD, kOutKeys>), grid, dim3(kThreads), 0, s, t, r, out);
  else
    hipLaunchKernelGGL((recall_score_kernel<NH, CD, kOutScores>), grid, dim3(kThreads), 0, s, t, r, out);
  return hipGetLastError();
}

template <int NH>
hipError_t launch_nh(const SeqTable& t, const RecallArgs& r, void* out, bool keys, hipStream_t s) {
  switch (r.key_dim) {
    case 64: return launch_nh_cd<NH, 64>(t, r, out, keys, s);
    case 128: return launch_nh_cd<NH, 128>(t, r, out, keys, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_recall_score(const SeqTable& t, const RecallArgs& r, void* out, bool keys, hipStream_t s) {
  if (t.score_wg_off[t.batch] == 0) return hipSuccess;
  switch (r.n_heads) {
    case 16: return launch_nh<16>(t, r, out, keys, s);
    case 32: return launch_nh<32>(t, r, out, keys, s);
    case 64: return launch_nh<64>(t, r, out, keys, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace lsa
