// Step 1 of the decode hot path: the Memory Indexer score of every chunk
// (Sec. 2.1, Eq. 4 with one indexer head and unit gate, i.e. the dual-encoder
// dot product s_c = qe . E_c).
//
// HBM-streaming GEMV.  A chunk-embedding row of D elements is split into
// 16-byte pieces; L consecutive lanes read one row (one 16-byte load each), so a
// wavefront load instruction covers 1 KiB of contiguous embeddings.  Each
// workgroup owns a contiguous block of rows of one sequence, issues all of its
// row loads up front (2 per lane: many small workgroups beat fewer with more
// loads each) and then reuses the registers for every lookahead query of that
// sequence, so E is read exactly once.  Partial dot
// products are reduced across the L lanes of a row with xor shuffles.
//   F32 : fp32 FMA accumulation
//   BF16: bf16 widened to fp32 (exact), fp32 FMA accumulation
//   I8  : v_dot4 int8 -> int32, exact (|s| <= D * 127^2 < 2^31 for D <= 512)
// With bf16 embeddings and at least 4 lookahead queries the same product is a
// dense [n_b x D] x [D x Q] contraction and runs on MFMA (score_mfma_kernel).
#include "lsa_internal.h"

namespace lsa {
namespace {

constexpr int kThreads = 256;
constexpr int kPasses = 2;  // row loads per lane: small workgroups, many of them (measured fastest)

template <int DT> struct Elem;
template <> struct Elem<LSA_F32> { static constexpr int size = 4; };
template <> struct Elem<LSA_BF16> { static constexpr int size = 2; };
template <> struct Elem<LSA_I8> { static constexpr int size = 1; };

template <int DT, int D>
struct Geo {
  static constexpr int pieces = D * Elem<DT>::size / 16;          // 16-byte pieces per row
  static constexpr int lanes = pieces < 64 ? pieces : 64;          // lanes per row
  static constexpr int ppl = pieces / lanes;                       // pieces per lane
  static constexpr int rows_per_pass = kThreads / lanes;
  static constexpr int rows_per_wg = rows_per_pass * kPasses;
};

// Dot product of one 16-byte embedding piece with the matching query piece.
__device__ __forceinline__ float piece_dot_f32(uint4 e, uint4 q, float acc) {
  acc = fmaf(__uint_as_float(e.x), __uint_as_float(q.x), acc);
  acc = fmaf(__uint_as_float(e.y), __uint_as_float(q.y), acc);
  acc = fmaf(__uint_as_float(e.z), __uint_as_float(q.z), acc);
  acc = fmaf(__uint_as_float(e.w), __uint_as_float(q.w), acc);
  return acc;
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float piece_dot_bf16(uint4 e, uint4 q, float acc) {
  acc = fmaf(bf_lo(e.x), bf_lo(q.x), acc);
  acc = fmaf(bf_hi(e.x), bf_hi(q.x), acc);
  acc = fmaf(bf_lo(e.y), bf_lo(q.y), acc);
  acc = fmaf(bf_hi(e.y), bf_hi(q.y), acc);
  acc = fmaf(bf_lo(e.z), bf_lo(q.z), acc);
  acc = fmaf(bf_hi(e.z), bf_hi(q.z), acc);
  acc = fmaf(bf_lo(e.w), bf_lo(q.w), acc);
  acc = fmaf(bf_hi(e.w), bf_hi(q.w), acc);
  return acc;
}

__device__ __forceinline__ int piece_dot_i8(uint4 e, uint4 q, int acc) {
  acc = __builtin_amdgcn_sdot4((int)e.x, (int)q.x, acc, false);
  acc = __builtin_amdgcn_sdot4((int)e.y, (int)q.y, acc, false);
  acc = __builtin_amdgcn_sdot4((int)e.z, (int)q.z, acc, false);
  acc = __builtin_amdgcn_sdot4((int)e.w, (int)q.w, acc, false);
  return acc;
}

template <int DT, int D, bool KEYS>
__global__ void __launch_bounds__(kThreads)
score_kernel(SeqTable t, const uint8_t* __restrict__ qe, const uint8_t* __restrict__ E,
             uint32_t* __restrict__ scores) {
  using G = Geo<DT, D>;
  constexpr int es = Elem<DT>::size;
  const int wg = blockIdx.x;
  const SeqData sq = seq_data(t, t.score_wg_off, wg);
  const int b = sq.b, n = sq.n;
  const int Q = t.n_lookahead;
  const int row0 = (wg - sq.wg0) * G::rows_per_wg;
  const int sub = threadIdx.x % G::lanes;       // piece index within the row
  const int rw = threadIdx.x / G::lanes;        // row within a pass
  const uint8_t* Eb = E + sq.chunk_off * (int64_t)(D * es);

  uint4 e[kPasses][G::ppl];
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    const int r = row0 + p * G::rows_per_pass + rw;
#pragma unroll
    for (int pp = 0; pp < G::ppl; ++pp) {
      if (r < n)
        e[p][pp] = *reinterpret_cast<const uint4*>(Eb + (int64_t)r * (D * es) + (sub + pp * G::lanes) * 16);
      else
        e[p][pp] = make_uint4(0, 0, 0, 0);
    }
  }

  uint32_t* out_b = scores + (int64_t)Q * sq.chunk_off;
  for (int j = 0; j < Q; ++j) {
    const uint8_t* qj = qe + ((int64_t)b * Q + j) * (D * es);
    uint4 qv[G::ppl];
#pragma unroll
    for (int pp = 0; pp < G::ppl; ++pp)
      qv[pp] = *reinterpret_cast<const uint4*>(qj + (sub + pp * G::lanes) * 16);
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int r = row0 + p * G::rows_per_pass + rw;
      uint32_t bits;
      if constexpr (DT == LSA_I8) {
        int acc = 0;
#pragma unroll
        for (int pp = 0; pp < G::ppl; ++pp) acc = piece_dot_i8(e[p][pp], qv[pp], acc);
#pragma unroll
        for (int off = G::lanes / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
        bits = (uint32_t)acc;
      } else {
        float acc = 0.f;
#pragma unroll
        for (int pp = 0; pp < G::ppl; ++pp)
          acc = (DT == LSA_F32) ? piece_dot_f32(e[p][pp], qv[pp], acc) : piece_dot_bf16(e[p][pp], qv[pp], acc);
#pragma unroll
        for (int off = G::lanes / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
        bits = __float_as_uint(acc);
      }
      if constexpr (KEYS) bits = DT == LSA_I8 ? int_score_key((int32_t)bits) : order_key<kKeysFromF32>(bits);
      if (sub == 0 && r < n) out_b[(int64_t)j * n + r] = bits;
    }
  }
  zero_arrivals(t);
}

// Several lookahead queries with bf16 embeddings: the scores of a sequence are
// the product S^T = E qe^T of its [n_b x D] chunk embeddings with the [D x Q]
// query embeddings, a real dense contraction, so it runs on
// v_mfma_f32_16x16x32_bf16: each wave takes groups of 16 chunks (A operand: 16
// rows of E, 32 dims per step, loaded straight from HBM) against all Q <= 16
// queries (B operand, in registers), D / 32 steps per group.  E is still read
// exactly once.  A lane's four scores of a group are four consecutive chunks of
// one query and leave as one 16-byte store.
constexpr int kMfmaMinQueries = 4;
// 16-chunk groups per wave.  The groups share the wave's query operand, so the
// query embeddings are read from L2 once per 16 x groups chunks: 4 groups up
// to D = 256, 2 at D = 512 (4 groups of A operands would take 256 registers).
template <int D> constexpr int mfma_groups() { return D >= 512 ? 2 : 4; }
template <int D> constexpr int mfma_rows_per_wg() { return 4 * 16 * mfma_groups<D>(); }

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int D, bool KEYS>
__global__ void __launch_bounds__(kThreads)
score_mfma_kernel(SeqTable t, const uint16_t* __restrict__ qe, const uint16_t* __restrict__ E,
                  uint32_t* __restrict__ scores) {
  constexpr int kSteps = D / 32;
  const int wg = blockIdx.x;
  const SeqData sq = seq_data(t, t.score_wg_off, wg);
  const int b = sq.b, n = sq.n, Q = t.n_lookahead;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int kGroups = mfma_groups<D>();
  const int c0 = (wg - sq.wg0) * mfma_rows_per_wg<D>() + wave * 16 * kGroups;
  if (c0 >= n) return;
  // A operand rows: chunk c0 + 16 gi + lane % 16 (clamped; its scores are not stored)
  bf16x8 ea[kGroups][kSteps];
#pragma unroll
  for (int gi = 0; gi < kGroups; ++gi) {
    const int crow = min(c0 + 16 * gi + (lane & 15), n - 1);
    const uint16_t* er = E + (sq.chunk_off + crow) * (int64_t)D + 8 * (lane >> 4);
#pragma unroll
    for (int st = 0; st < kSteps; ++st)
      ea[gi][st] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(er + 32 * st));
  }
  // B operand: query lane % 16 (zero beyond Q), dims 32 st + 8 (lane / 16) .. + 7
  const int jq = lane & 15;
  bf16x8 qb[kSteps];
  const uint16_t* qp = qe + ((int64_t)b * Q + min(jq, Q - 1)) * D + 8 * (lane >> 4);
#pragma unroll
  for (int st = 0; st < kSteps; ++st)
    qb[st] = jq < Q ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(qp + 32 * st)) : bf16x8{};
  uint32_t* out = scores + (int64_t)Q * sq.chunk_off + (int64_t)jq * n;
#pragma unroll
  for (int gi = 0; gi < kGroups; ++gi) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < kSteps; ++st) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ea[gi][st], qb[st], acc, 0, 0, 0);
    // acc[r] = score of chunk c + r, c = c0 + 16 gi + 4 (lane / 16), for query lane % 16: four
    // consecutive scores of one query, one 16-byte store when they are aligned and all exist
    if (jq < Q) {
      uint32_t bits[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        bits[r] = __float_as_uint(acc[r]);
        if constexpr (KEYS) bits[r] = order_key<kKeysFromF32>(bits[r]);
      }
      const int c = c0 + 16 * gi + 4 * (lane >> 4);
      if (((reinterpret_cast<uintptr_t>(out + c) & 15u) == 0) && c + 4 <= n) {
        *reinterpret_cast<uint4*>(out + c) = make_uint4(bits[0], bits[1], bits[2], bits[3]);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (c + r < n) out[c + r] = bits[r];
      }
    }
  }
  zero_arrivals(t);  // wave 0 of workgroup 0 never returns early (c0 = 0)
}

template <int D>
hipError_t launch_mfma_d(const SeqTable& t, const void* qe, const void* E, void* scores, bool keys, hipStream_t s) {
  const int grid = t.score_wg_off[t.batch];
  const auto* q16 = static_cast<const uint16_t*>(qe);
  const auto* e16 = static_cast<const uint16_t*>(E);
  auto* out = static_cast<uint32_t*>(scores);
  if (keys)
    hipLaunchKernelGGL((score_mfma_kernel<D, true>), dim3(grid), dim3(kThreads), 0, s, t, q16, e16, out);
  else
    hipLaunchKernelGGL((score_mfma_kernel<D, false>), dim3(grid), dim3(kThreads), 0, s, t, q16, e16, out);
  return hipGetLastError();
}

bool use_mfma(int32_t emb_dtype, int32_t n_lookahead) {
  return emb_dtype == LSA_BF16 && n_lookahead >= kMfmaMinQueries;
}

template <int DT, int D>
hipError_t launch_dt_d(const SeqTable& t, const void* qe, const void* E, void* scores, bool keys, hipStream_t s) {
  const int grid = t.score_wg_off[t.batch];
  const auto* q8 = static_cast<const uint8_t*>(qe);
  const auto* e8 = static_cast<const uint8_t*>(E);
  auto* out = static_cast<uint32_t*>(scores);
  if (keys)
    hipLaunchKernelGGL((score_kernel<DT, D, true>), dim3(grid), dim3(kThreads), 0, s, t, q8, e8, out);
  else
    hipLaunchKernelGGL((score_kernel<DT, D, false>), dim3(grid), dim3(kThreads), 0, s, t, q8, e8, out);
  return hipGetLastError();
}

template <int DT>
hipError_t launch_dt(const SeqTable& t, int32_t D, const void* qe, const void* E, void* scores, bool keys,
                     hipStream_t s) {
  switch (D) {
    case 64: return launch_dt_d<DT, 64>(t, qe, E, scores, keys, s);
    case 128: return launch_dt_d<DT, 128>(t, qe, E, scores, keys, s);
    case 256: return launch_dt_d<DT, 256>(t, qe, E, scores, keys, s);
    case 512: return launch_dt_d<DT, 512>(t, qe, E, scores, keys, s);
    default: return hipErrorInvalidValue;
  }
}

template <int DT>
int rows_dt(int32_t D) {
  switch (D) {
    case 64: return Geo<DT, 64>::rows_per_wg;
    case 128: return Geo<DT, 128>::rows_per_wg;
    case 256: return Geo<DT, 256>::rows_per_wg;
    case 512: return Geo<DT, 512>::rows_per_wg;
    default: return 0;
  }
}

}  // namespace

int score_rows_per_wg(int32_t emb_dtype, int32_t emb_dim, int32_t n_lookahead) {
  if (use_mfma(emb_dtype, n_lookahead)) {
    switch (emb_dim) {
      case 64: return mfma_rows_per_wg<64>();
      case 128: return mfma_rows_per_wg<128>();
      case 256: return mfma_rows_per_wg<256>();
      case 512: return mfma_rows_per_wg<512>();
      default: return 0;
    }
  }
  switch (emb_dtype) {
    case LSA_F32: return rows_dt<LSA_F32>(emb_dim);
    case LSA_BF16: return rows_dt<LSA_BF16>(emb_dim);
    case LSA_I8: return rows_dt<LSA_I8>(emb_dim);
    default: return 0;
  }
}

hipError_t launch_score(const SeqTable& t, int32_t emb_dtype, int32_t emb_dim, const void* qe,
                        const void* E, void* scores, bool keys, hipStream_t s) {
  if (use_mfma(emb_dtype, t.n_lookahead)) {
    switch (emb_dim) {
      case 64: return launch_mfma_d<64>(t, qe, E, scores, keys, s);
      case 128: return launch_mfma_d<128>(t, qe, E, scores, keys, s);
      case 256: return launch_mfma_d<256>(t, qe, E, scores, keys, s);
      case 512: return launch_mfma_d<512>(t, qe, E, scores, keys, s);
      default: return hipErrorInvalidValue;
    }
  }
  switch (emb_dtype) {
    case LSA_F32: return launch_dt<LSA_F32>(t, emb_dim, qe, E, scores, keys, s);
    case LSA_BF16: return launch_dt<LSA_BF16>(t, emb_dim, qe, E, scores, keys, s);
    case LSA_I8: return launch_dt<LSA_I8>(t, emb_dim, qe, E, scores, keys, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace lsa
