// Step 3 of the decode hot path: decode attention softmax(scale q K^T) V over
// the tokens of the kept chunks only (Sec. 2.1, core attention over the
// selected entries), gathered by chunk id from the paged bf16 cache.
//
// Flash-decoding with split-K over the kept-chunk list.  Work unit = (sequence
// b, KV head g, split s); a split owns a contiguous range of the kept list.
// All G * Tq query rows that read KV head g are handled together, so each K/V
// byte is fetched from HBM once.
//
// Both products run on MFMA v_mfma_f32_16x16x32_bf16 with no data shuffles:
//  * QK computes S^T = K Q^T with 16 tokens as the M dimension and 16 query rows
//    as N.  The M rows of the two 16-token MFMAs of a 32-token tile are permuted
//    (tokens 8a+0..3 and 8a+4..7) so that after the product each lane holds the
//    8 consecutive tokens 8*(lane/16)..+7 of query row lane%16 -- exactly the
//    A-operand layout the PV MFMA wants for P.
//  * PV computes O = P V with the 32 tokens as K and 16 head dims per MFMA as N;
//    the V block is stored [dim][token], so every B operand is one 16-byte load.
//  * P is split into bf16 hi + lo parts (two MFMAs), keeping ~16 significant
//    bits of the probabilities; logits, the running max/sum and O stay fp32.
// Every operand load is a 16-byte global load; per instruction a wavefront
// reads 16 rows x 64 contiguous bytes.
//
// Rows <= 16 (one 16-row block): the 4 waves of a workgroup take alternate
// chunks of the split and merge their (m, l, O) states through LDS.  Rows > 16:
// each wave owns one 16-row block and walks every chunk of the split; the
// workgroup's waves read the same K/V lines back to back, so only the first
// read reaches HBM.
//
// Split partials (m, l, O) go to the workspace; the last workgroup of each
// (b, g, row group) -- detected with a device-scope counter, released and
// acquired with fences -- merges them in split order, so results are bitwise
// reproducible, and resets the counter to zero for the next call.
#include "lsa_internal.h"

namespace lsa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kThreads = kAttnWaves * 64;
constexpr int kOPad = 132;  // LDS row pitch (floats) of the wave merge

__device__ __forceinline__ bf16x8 load8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int C, bool ROW_SPLIT>
__global__ void __launch_bounds__(kThreads)
attn_kernel(SeqTable t, AttnArgs a) {
  __shared__ float sm_o[ROW_SPLIT ? 1 : kAttnWaves][16][kOPad];
  __shared__ float sm_m[kAttnWaves][16], sm_l[kAttnWaves][16];
  __shared__ int sh_last;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, kg = lane >> 4;

  // ---- which (sequence, kv head, row group, split) this workgroup owns
  const int wg = blockIdx.x;
  int b = 0;
  while (wg >= t.wg_off[b + 1]) ++b;
  const int ns = t.nsplit[b];
  const int RG = a.row_groups;
  const int local = wg - t.wg_off[b];
  const int g = local / (ns * RG);
  const int rg = (local / ns) % RG;
  const int s = local % ns;
  // sel_count and the chunk ids are clamped so that malformed device inputs
  // can only give wrong numbers, never an out-of-bounds access.
  const int cnt = min(max(a.sel_count[b], 0), a.sel_pitch);
  const int n_b = t.n[b];
  const int lo = (int)(((int64_t)s * cnt) / ns);
  const int hi = (int)(((int64_t)(s + 1) * cnt) / ns);
  const int G = a.group;

  // ---- query operand: row n16 of this wave's 16-row block
  const int rblock = ROW_SPLIT ? rg * kAttnWaves + wave : 0;
  const bool block_live = rblock * 16 < a.rows;
  bf16x8 qb[4];
  {
    const int row = rblock * 16 + n16;
    if (row < a.rows) {
      const int tq = row / G, h = g * G + row % G;
      const uint16_t* qp = a.q + (((int64_t)b * a.n_qtok + tq) * a.n_q_heads + h) * kHeadDim + 8 * kg;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) qb[jj] = load8(qp + 32 * jj);
    } else {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) qb[jj] = bf16x8{};
    }
  }

  f32x4 o[8];
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const int c_first = ROW_SPLIT ? lo : lo + wave;
  const int c_step = ROW_SPLIT ? 1 : kAttnWaves;
  const int32_t* sel = a.sel_idx + (int64_t)b * a.sel_pitch;
  const int tokA = 8 * (n16 >> 2) + (n16 & 3);  // token of this lane's A row in the first QK MFMA

  if (block_live) {
    for (int pos = c_first; pos < hi; pos += c_step) {
      const int c = min(max(__builtin_amdgcn_readfirstlane(sel[pos]), 0), n_b - 1);
      const int64_t gc = t.chunk_off[b] + c;
      const uint16_t* kb = a.k + gc * a.chunk_stride + g * a.head_stride;
      const uint16_t* vb = a.v + gc * a.chunk_stride + g * a.head_stride;
#pragma unroll
      for (int tt = 0; tt < C / 32; ++tt) {
        bf16x8 ka[2][4], vv[8];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            ka[hf][jj] = load8(kb + (32 * tt + tokA + 4 * hf) * kHeadDim + 8 * kg + 32 * jj);
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) vv[nb] = load8(vb + (16 * nb + n16) * C + 32 * tt + 8 * kg);

        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[0][jj], qb[jj], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[1][jj], qb[jj], s1, 0, 0, 0);
        }
        // lane holds logits of query row n16 for tokens 32tt + 8kg + 0..7
        float x[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          x[i] *= a.scale_log2e;
          mx = fmaxf(mx, x[i]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx);
        const float alpha = fast_exp2(m_run - m_new);
        float p[8], psum = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          p[i] = fast_exp2(x[i] - m_new);
          psum += p[i];
        }
        l_run = l_run * alpha + psum;
        m_run = m_new;
        if (__ballot(alpha != 1.f) != 0ull) {
          // O rows of this lane are 4kg..4kg+3; their alphas live in lanes 4kg+r
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float ar = __shfl(alpha, 4 * kg + r);
#pragma unroll
            for (int nb = 0; nb < 8; ++nb) o[nb][r] *= ar;
          }
        }
        bf16x8 ph, pl;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          ph[i] = (__bf16)p[i];
          pl[i] = (__bf16)(p[i] - (float)ph[i]);
        }
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
          o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, vv[nb], o[nb], 0, 0, 0);
          o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, vv[nb], o[nb], 0, 0, 0);
        }
      }
    }
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  // ---- write this workgroup's split partials
  const int rows_pad = a.rows_pad;
  const int64_t unit0 = (int64_t)t.wg_off[b] / RG + (int64_t)g * ns;  // split 0 of (b, g)
  const int64_t unit = unit0 + s;
  if constexpr (ROW_SPLIT) {
    if (block_live) {
      const int64_t rbase = unit * rows_pad + rblock * 16;
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int nb = 0; nb < 8; ++nb)
          a.part_o[(rbase + 4 * kg + r) * kHeadDim + 16 * nb + n16] = o[nb][r];
      if (kg == 0) {
        a.part_ml[(rbase + n16) * 2 + 0] = m_run;
        a.part_ml[(rbase + n16) * 2 + 1] = l_run;
      }
    }
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) sm_o[wave][4 * kg + r][16 * nb + n16] = o[nb][r];
    if (kg == 0) {
      sm_m[wave][n16] = m_run;
      sm_l[wave][n16] = l_run;
    }
    __syncthreads();
    for (int idx = tid; idx < a.rows * kHeadDim; idx += kThreads) {
      const int r = idx / kHeadDim, e = idx % kHeadDim;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kAttnWaves; ++w) M = fmaxf(M, sm_m[w][r]);
      float acc = 0.f, L = 0.f;
      if (M != -INFINITY) {
#pragma unroll
        for (int w = 0; w < kAttnWaves; ++w) {
          const float f = fast_exp2(sm_m[w][r] - M);
          acc += f * sm_o[w][r][e];
          L += f * sm_l[w][r];
        }
      }
      a.part_o[(unit * rows_pad + r) * kHeadDim + e] = acc;
      if (e == 0) {
        a.part_ml[(unit * rows_pad + r) * 2 + 0] = M;
        a.part_ml[(unit * rows_pad + r) * 2 + 1] = L;
      }
    }
  }

  // ---- the last split of (b, g, rg) to finish merges all splits in order
  __threadfence();
  __syncthreads();
  const int64_t cidx = ((int64_t)b * a.n_kv_heads + g) * RG + rg;
  if (tid == 0) {
    const uint32_t prev = atomicAdd(&a.counters[cidx], 1u);
    sh_last = (prev == (uint32_t)(ns - 1));
  }
  __syncthreads();
  if (!sh_last) return;
  __threadfence();
  if (tid == 0) atomicExch(&a.counters[cidx], 0u);

  const int row_begin = ROW_SPLIT ? rg * kAttnWaves * 16 : 0;
  const int row_end = ROW_SPLIT ? min(row_begin + kAttnWaves * 16, a.rows) : a.rows;
  for (int idx = tid; idx < (row_end - row_begin) * kHeadDim; idx += kThreads) {
    const int r = row_begin + idx / kHeadDim, e = idx % kHeadDim;
    float M = -INFINITY;
    for (int s2 = 0; s2 < ns; ++s2) M = fmaxf(M, a.part_ml[((unit0 + s2) * rows_pad + r) * 2]);
    float acc = 0.f, L = 0.f;
    for (int s2 = 0; s2 < ns; ++s2) {
      const float ms = a.part_ml[((unit0 + s2) * rows_pad + r) * 2];
      const float f = (ms == -INFINITY) ? 0.f : fast_exp2(ms - M);
      acc += f * a.part_o[((unit0 + s2) * rows_pad + r) * kHeadDim + e];
      L += f * a.part_ml[((unit0 + s2) * rows_pad + r) * 2 + 1];
    }
    const int tq = r / G, h = g * G + r % G;
    const int64_t orow = ((int64_t)b * a.n_qtok + tq) * a.n_q_heads + h;
    a.out[orow * kHeadDim + e] = acc / L;
    if (e == 0 && a.lse != nullptr) a.lse[orow] = (M + __log2f(L)) * kLn2;
  }
}

template <int C>
hipError_t launch_c(const SeqTable& t, const AttnArgs& a, hipStream_t s) {
  const dim3 grid(t.wg_off[t.batch]);
  if (a.rows > 16)
    hipLaunchKernelGGL((attn_kernel<C, true>), grid, dim3(kThreads), 0, s, t, a);
  else
    hipLaunchKernelGGL((attn_kernel<C, false>), grid, dim3(kThreads), 0, s, t, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const SeqTable& t, const AttnArgs& a, int32_t chunk_size, hipStream_t s) {
  if (chunk_size == 64) return launch_c<64>(t, a, s);
  if (chunk_size == 128) return launch_c<128>(t, a, s);
  return hipErrorInvalidValue;
}

}  // namespace lsa
