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
// One workgroup of 4 waves covers 64 entries of one sequence.  Its first act is
// to issue the loads of all its index keys (every layer), so that they are in
// flight while the queries and gates of the sequence are staged in LDS.
#include "lsa_internal.h"

namespace lsa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

template <int NH, int CD, bool KEYS>
__global__ void __launch_bounds__(kThreads)
recall_score_kernel(SeqTable t, RecallArgs r, void* __restrict__ out) {
  constexpr int kPitch = CD / 8 + 1;  // uint4 per staged query row; the pad slot spreads rows over the banks
  constexpr int kSteps = CD / 32;     // MFMA k-steps
  constexpr int kBlocks = NH / 16;    // 16-head blocks
  __shared__ uint4 sq[kMaxIdxLayers * NH * kPitch];
  __shared__ float sw[kMaxIdxLayers * NH];

  const int L = r.n_layers;
  const int wg = blockIdx.x;
  int b = 0;
  while (wg >= t.score_wg_off[b + 1]) ++b;
  const int n = t.n[b];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e0 = (wg - t.score_wg_off[b]) * kRecallRowsPerWg + wave * 16;
  const int hi = lane >> 4;  // this lane's k-slice 8 hi .. 8 hi + 7 of every 32-wide step

  // B operands: entry e0 + lane % 16 (clamped; its result is not stored), dims
  // 32 st + 8 hi .. + 7, every layer
  bf16x8 kb[kMaxIdxLayers][kSteps];
  {
    const int ent = min(e0 + (lane & 15), n - 1);
    const uint16_t* kp = r.k + (t.chunk_off[b] + ent) * CD + 8 * hi;
#pragma unroll
    for (int l = 0; l < kMaxIdxLayers; ++l)
#pragma unroll
      for (int st = 0; st < kSteps; ++st)
        kb[l][st] = l < L ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(kp + l * r.layer_stride + 32 * st))
                          : bf16x8{};
  }

  // queries [L][NH][CD] and gates [L][NH] of sequence b
  const uint4* qsrc = reinterpret_cast<const uint4*>(r.q) + (int64_t)b * L * NH * (CD / 8);
  for (int i = tid; i < L * NH * (CD / 8); i += kThreads) sq[(i / (CD / 8)) * kPitch + i % (CD / 8)] = qsrc[i];
  for (int i = tid; i < L * NH; i += kThreads) sw[i] = r.w[(int64_t)b * L * NH + i];
  __syncthreads();
  if (e0 >= n) return;

  float best = -INFINITY;
#pragma unroll
  for (int l = 0; l < kMaxIdxLayers; ++l) {
    if (l >= L) break;
    f32x4 acc[kBlocks];
#pragma unroll
    for (int hb = 0; hb < kBlocks; ++hb) acc[hb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < kSteps; ++st)
#pragma unroll
      for (int hb = 0; hb < kBlocks; ++hb) {
        // A operand: head 16 hb + lane % 16, dims 32 st + 8 hi .. + 7
        const uint4 a = sq[(l * NH + 16 * hb + (lane & 15)) * kPitch + 4 * st + hi];
        acc[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), kb[l][st], acc[hb], 0, 0, 0);
      }
    // acc[hb][j] = q_l[16 hb + 4 hi + j] . K_l[e0 + lane % 16]
    float x = 0.f;
#pragma unroll
    for (int hb = 0; hb < kBlocks; ++hb)
#pragma unroll
      for (int j = 0; j < 4; ++j) x = fmaf(sw[l * NH + 16 * hb + 4 * hi + j], fmaxf(acc[hb][j], 0.f), x);
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    if constexpr (!KEYS) {
      if (lane < 16 && e0 + lane < n)
        static_cast<float*>(out)[l * r.total + t.chunk_off[b] + e0 + lane] = x;
    }
    best = fmaxf(best, x);
  }
  if constexpr (KEYS) {
    if (lane < 16 && e0 + lane < n)
      static_cast<uint32_t*>(out)[t.chunk_off[b] + e0 + lane] = order_key<kKeysFromF32>(__float_as_uint(best));
  }
}

template <int NH, int CD>
hipError_t launch_nh_cd(const SeqTable& t, const RecallArgs& r, void* out, bool keys, hipStream_t s) {
  const dim3 grid(t.score_wg_off[t.batch]);
  if (keys)
    hipLaunchKernelGGL((recall_score_kernel<NH, CD, true>), grid, dim3(kThreads), 0, s, t, r, out);
  else
    hipLaunchKernelGGL((recall_score_kernel<NH, CD, false>), grid, dim3(kThreads), 0, s, t, r, out);
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
