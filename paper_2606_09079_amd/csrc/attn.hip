// Step 3 of the decode hot path: decode attention softmax(scale q K^T) V over
// the tokens of the kept chunks only (Sec. 2.1, core attention over the
// selected entries), gathered by chunk id from the paged bf16 cache.
//
// Flash-decoding with split-K over the kept-chunk list, in two kernels:
//
// attn_split_kernel -- work unit = (sequence b, KV head g, split s).  The kept
//   list of (b, g) is cut into 32-token tiles and each split owns a contiguous,
//   equal share of them; the split count is sized so that the whole grid is one
//   resident round on MI355X (256 CUs x 2 workgroups).  All G * Tq query rows
//   that read KV head g are handled together, so every K/V byte is fetched from
//   HBM once.  Both products run on v_mfma_f32_16x16x32_bf16:
//   * QK computes S^T = K Q^T with 16 tokens as M and 16 query rows as N.  The
//     cache stores each (chunk, head) block in MFMA operand order, and the M
//     rows of the two 16-token MFMAs of a tile are tokens 8a+0..3 and 8a+4..7,
//     so after the product each lane holds the 8 consecutive tokens
//     8*(lane/16)..+7 of query row lane%16 -- the A-operand layout PV needs.
//   * PV computes O = P V with the tile's 32 tokens as K and 16 head dims per
//     MFMA as N.  P is split into bf16 hi + lo parts (two MFMAs), keeping ~16
//     significant bits; logits, the running max / sum and O stay fp32.
//   Every load instruction reads 1 KiB of contiguous cache with a nontemporal
//   (streaming) hint, and two tiles are in flight per wave (the next tile loads
//   while the current one computes).
//   Rows <= 16: the 4 waves of a workgroup take consecutive quarters of the
//   split's tiles and merge their (m, l, O) states through LDS.  Rows > 16:
//   each wave owns one 16-row block and walks all tiles of the split; the
//   workgroup's waves read the same cache lines back to back, so only the first
//   read reaches HBM.  Partials (m, l, O) go to the workspace.
//
// attn_combine_kernel -- one workgroup per output row (b, t, h) merges the
//   splits of its (b, g) in split order: weights exp2(m_s - M), then O as a
//   weighted sum of float4 slices, each thread holding a strided subset of the
//   splits so that all its loads are in flight at once.  Fixed order throughout,
//   so results are bitwise reproducible.
#include "lsa_internal.h"

namespace lsa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kThreads = kAttnWaves * 64;
constexpr int kOPad = 132;  // LDS row pitch (floats) of the wave merge
constexpr int kCombineGroups = kThreads / (kHeadDim / 4);  // split groups in the combine

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 load8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// K/V stream: every byte is read exactly once per step, so the loads are
// nontemporal (streaming) and do not displace other data in the caches.
__device__ __forceinline__ bf16x8 load8_stream(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// (sequence, kv head, row group, split) of attention workgroup wg
struct Unit {
  int b, g, rg, s, ns;
};

__device__ __forceinline__ Unit unit_of(const SeqTable& t, int RG, int wg) {
  Unit u;
  int b = 0;
  while (wg >= t.wg_off[b + 1]) ++b;
  const int ns = t.nsplit[b];
  const int local = wg - t.wg_off[b];
  u.b = b;
  u.ns = ns;
  u.g = local / (ns * RG);
  u.rg = (local / ns) % RG;
  u.s = local % ns;
  return u;
}

template <int C, bool ROW_SPLIT>
__global__ void __launch_bounds__(kThreads, 2)  // 2 waves per SIMD: <= 256 registers
attn_split_kernel(SeqTable t, AttnArgs a) {
  __shared__ float sm_o[ROW_SPLIT ? 1 : kAttnWaves][16][kOPad];
  __shared__ float sm_m[kAttnWaves][16], sm_l[kAttnWaves][16];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, kg = lane >> 4;
  const int RG = a.row_groups, G = a.group;
  const Unit u = unit_of(t, RG, blockIdx.x);
  const int b = u.b, g = u.g, s = u.s, ns = u.ns;

  // sel_count and the chunk ids are clamped so that malformed device inputs
  // can only give wrong numbers, never an out-of-bounds access.
  constexpr int TPC = C / 32;  // 32-token tiles per chunk
  const int cnt = min(max(a.sel_count[b], 0), a.sel_pitch);
  const int n_b = t.n[b];
  const int nTall = cnt * TPC;
  const int T0 = (int)(((int64_t)s * nTall) / ns), T1 = (int)(((int64_t)(s + 1) * nTall) / ns);
  int Tb = T0, Te = T1;
  if constexpr (!ROW_SPLIT) {
    Tb = T0 + (int)(((int64_t)wave * (T1 - T0)) / kAttnWaves);
    Te = T0 + (int)(((int64_t)(wave + 1) * (T1 - T0)) / kAttnWaves);
  }

  // ---- query operand: row n16 of this wave's 16-row block
  const int rblock = ROW_SPLIT ? u.rg * kAttnWaves + wave : 0;
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

  // Tiles Tb..Te-1 of the kept list; tile T is tile T % TPC of kept chunk T / TPC.
  // Chunk ids are fetched 64 at a time into a register (one per lane) and read
  // back with readlane, so no scalar load sits between consecutive tiles.
  const int nT = block_live && Te > Tb ? Te - Tb : 0;
  const int pos0 = Tb / TPC;
  const int npos = nT > 0 ? (Te - 1) / TPC - pos0 + 1 : 0;
  const int32_t* sel = a.sel_idx + (int64_t)b * a.sel_pitch + pos0;
  int sel_base = 0;
  int sel_lane = lane < npos ? sel[lane] : 0;
  const uint16_t* kbase = a.k + t.chunk_off[b] * a.chunk_stride + g * a.head_stride + lane * 8;
  const uint16_t* vbase = a.v + t.chunk_off[b] * a.chunk_stride + g * a.head_stride + lane * 8;

  // K and V tiles are 8 KiB each and contiguous in the MFMA-ordered block
  // layout: load instruction q of a tile reads bytes [1024 q, 1024 q + 1024).
  auto load_tile = [&](int i, bf16x8(&kt)[8], bf16x8(&vt)[8]) {
    const int T = Tb + i;
    const int j = T / TPC - pos0, tt = T % TPC;
    if (j - sel_base >= 64) {  // wave-uniform: next window of chunk ids
      sel_base = j & ~63;
      sel_lane = sel_base + lane < npos ? sel[sel_base + lane] : 0;
    }
    const int c = min(max(__builtin_amdgcn_readlane(sel_lane, j - sel_base), 0), n_b - 1);
    const int64_t off = (int64_t)c * a.chunk_stride + tt * (32 * kHeadDim);
    const uint16_t* kp = kbase + off;
    const uint16_t* vp = vbase + off;
#pragma unroll
    for (int q = 0; q < 8; ++q) kt[q] = load8_stream(kp + q * 512);
#pragma unroll
    for (int q = 0; q < 8; ++q) vt[q] = load8_stream(vp + q * 512);
  };

  auto compute_tile = [&](const bf16x8(&kt)[8], const bf16x8(&vt)[8]) {
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[jj], qb[jj], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[4 + jj], qb[jj], s1, 0, 0, 0);
    }
    // lane holds logits of query row n16 for tile tokens 8kg + 0..7
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
      o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, vt[nb], o[nb], 0, 0, 0);
      o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, vt[nb], o[nb], 0, 0, 0);
    }
  };

  // Two tile buffers: the loads of tile i+1 are in flight while tile i computes.
  bf16x8 ka[8], va[8], kb2[8], vb2[8];
  if (nT > 0) load_tile(0, ka, va);
  for (int i = 0; i < nT; i += 2) {
    if (i + 1 < nT) load_tile(i + 1, kb2, vb2);
    compute_tile(ka, va);
    if (i + 1 < nT) {
      if (i + 2 < nT) load_tile(i + 2, ka, va);
      compute_tile(kb2, vb2);
    }
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  // ---- this split's partials: rows of the (b, g) group, [unit][rows_pad]
  const int rows_pad = a.rows_pad;
  const int64_t unit = (int64_t)t.wg_off[b] / RG + (int64_t)g * ns + s;
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
}

__global__ void __launch_bounds__(kThreads)
attn_combine_kernel(SeqTable t, AttnArgs a) {
  __shared__ float sm_w[kMaxSplits];
  __shared__ float4 sm_red[kCombineGroups][kHeadDim / 4];
  __shared__ float sm_lw[kAttnWaves];
  __shared__ float sh_M;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = a.group;
  const int rows_per_b = a.n_qtok * a.n_q_heads;
  const int b = blockIdx.x / rows_per_b;
  const int rem = blockIdx.x - b * rows_per_b;
  const int tq = rem / a.n_q_heads, h = rem - tq * a.n_q_heads;
  const int g = h / G, r = tq * G + h % G;  // row within the (b, g) group
  const int ns = t.nsplit[b];
  const int64_t unit0 = (int64_t)t.wg_off[b] / a.row_groups + (int64_t)g * ns;
  const int rows_pad = a.rows_pad;

  // split weights exp2(m_s - M) in LDS and L = sum_s w_s l_s (one round of loads)
  float m_s = -INFINITY, l_s = 0.f;
  if (tid < ns) {
    const float2 ml = *reinterpret_cast<const float2*>(a.part_ml + ((unit0 + tid) * rows_pad + r) * 2);
    m_s = ml.x;
    l_s = ml.y;
  }
  float mw = m_s;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mw = fmaxf(mw, __shfl_xor(mw, off));
  if (lane == 0) sm_lw[wave] = mw;
  __syncthreads();
  if (tid == 0) {
    float M = sm_lw[0];
    for (int w = 1; w < kAttnWaves; ++w) M = fmaxf(M, sm_lw[w]);
    sh_M = M;
  }
  __syncthreads();
  const float M = sh_M;
  const float f = (tid < ns && m_s != -INFINITY) ? fast_exp2(m_s - M) : 0.f;
  if (tid < ns) sm_w[tid] = f;
  float lf = f * l_s;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) lf += __shfl_xor(lf, off);
  __syncthreads();  // sm_lw is reused
  if (lane == 0) sm_lw[wave] = lf;
  __syncthreads();
  float L = sm_lw[0];
  for (int w = 1; w < kAttnWaves; ++w) L += sm_lw[w];
  const float invL = 1.f / L;

  // O = sum_s w_s O_s: thread (group sg, slice e4) sums splits sg, sg + 8, ...
  const int sg = tid / (kHeadDim / 4), e4 = (tid % (kHeadDim / 4)) * 4;
  const float* src = a.part_o + (unit0 * rows_pad + r) * kHeadDim + e4;
  const int64_t sstride = (int64_t)rows_pad * kHeadDim;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8
  for (int s2 = sg; s2 < ns; s2 += kCombineGroups) {
    const float4 v = *reinterpret_cast<const float4*>(src + s2 * sstride);
    const float w = sm_w[s2];
    acc.x += w * v.x;
    acc.y += w * v.y;
    acc.z += w * v.z;
    acc.w += w * v.w;
  }
  sm_red[sg][e4 / 4] = acc;
  __syncthreads();
  const int64_t orow = ((int64_t)b * a.n_qtok + tq) * a.n_q_heads + h;
  if (tid < kHeadDim / 4) {
    float4 sum = sm_red[0][tid];
#pragma unroll
    for (int q = 1; q < kCombineGroups; ++q) {
      const float4 v = sm_red[q][tid];
      sum.x += v.x;
      sum.y += v.y;
      sum.z += v.z;
      sum.w += v.w;
    }
    sum.x *= invL;
    sum.y *= invL;
    sum.z *= invL;
    sum.w *= invL;
    *reinterpret_cast<float4*>(a.out + orow * kHeadDim + tid * 4) = sum;
  }
  if (tid == 0 && a.lse != nullptr) a.lse[orow] = (M + __log2f(L)) * kLn2;
}

template <int C>
hipError_t launch_c(const SeqTable& t, const AttnArgs& a, hipStream_t s) {
  const dim3 grid(t.wg_off[t.batch]);
  if (a.rows > 16)
    hipLaunchKernelGGL((attn_split_kernel<C, true>), grid, dim3(kThreads), 0, s, t, a);
  else
    hipLaunchKernelGGL((attn_split_kernel<C, false>), grid, dim3(kThreads), 0, s, t, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(t.batch * a.n_qtok * a.n_q_heads), dim3(kThreads), 0, s, t,
                     a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const SeqTable& t, const AttnArgs& a, int32_t chunk_size, hipStream_t s) {
  if (chunk_size == 64) return launch_c<64>(t, a, s);
  if (chunk_size == 128) return launch_c<128>(t, a, s);
  return hipErrorInvalidValue;
}

}  // namespace lsa
