// Step 3 of the decode hot path: decode attention softmax(scale q K^T) V over
// the tokens of the kept chunks only (Sec. 2.1, core attention over the
// selected entries), gathered by chunk id from the paged bf16 cache.
//
// Flash-decoding with split-K over the kept-chunk list.  The kept list of
// each (sequence b, KV head g) is cut into 32-token tiles, and each split owns
// a contiguous share of them, weighted by the XCD its workgroup runs on; the
// split count is sized so that the whole grid is one resident round on MI355X
// (one workgroup per CU for a few sequences, two for more).  All G * Tq
// query rows that read KV head g are handled by the same workgroup, so every
// K/V byte is fetched from HBM once.  Logits, the running max / sum and O stay
// fp32; the softmax weights P enter the PV product as bf16 hi + lo parts (two
// MFMAs per product), which keeps ~16 significant bits.
//
// attn_split_kernel (rows <= 16) on v_mfma_f32_16x16x32_bf16.  The 4 waves of
//   a workgroup take every fourth tile of the split (wave w: tiles w, w + 4,
//   ...), each streaming its own tiles straight into registers (1 KiB per load
//   instruction, nontemporal hint, two tiles in flight per wave), and merge
//   their (m, l, O) states through LDS.  Interleaved tiles keep the four waves
//   of a workgroup within a tile of each other where consecutive quarters left
//   them waiting for the slowest at the merge.
//   * QK computes S^T = K Q^T with 16 tokens as M and 16 query rows as N.  The
//     cache stores each (chunk, head) block in MFMA operand order, and the M
//     rows of the two 16-token MFMAs of a tile are tokens 8a+0..3 and 8a+4..7,
//     so after the product each lane holds the 8 consecutive tokens
//     8*(lane/16)..+7 of query row lane%16 -- the A-operand layout PV needs.
//   * PV computes O = P V with the tile's 32 tokens as K and 16 head dims per
//     MFMA as N.
// attn_rows_kernel (17..128 rows) on v_mfma_f32_32x32x16_bf16.  Every wave
//   owns 32 rows and needs every tile, so each tile is copied once per
//   workgroup from HBM into LDS (global->LDS copies into MFMA operand order,
//   three tiles ahead, five 16 KiB buffers).  QK computes S^T = K Q^T and PV
//   computes O^T = V^T P^T, so a lane's O registers all belong to its own row
//   and the softmax rescale needs no exchange; the QK products of tile j are
//   issued before the softmax and PV of tile j - 1, so VALU and MFMA overlap.
//
// attn_combine_kernel (more than 16 splits) -- one workgroup per output row
//   (b, t, h) merges the splits of its (b, g): weights exp2(m_s - M), O as the
//   weighted sum of the split outputs, divided by L = sum_s exp2(m_s - M) l_s.
//   Every wave computes M and L itself from all splits' (m, l), so the loads of
//   (m, l) and of the thread's O slices go out in one round and only the final
//   merge of the 8 split groups needs a barrier.
// attn_combine_few_kernel (at most 16 splits) -- the same merge with one thread
//   per (output row, float4 slice of O) walking every split itself.
// The summation order of both combines is fixed, so results are bitwise
// reproducible.  In the fused step with at most 16 splits and one workgroup
// per CU, the split kernel merges instead: its workgroups store their partials
// with device-scope (write-through) stores and count themselves in on a
// per-(b, g) counter that the scoring kernel zeroed; the last to arrive reads
// every partial with device-scope loads and runs the few-split merge, with no
// fence and no combine launch.
#include "lsa_internal.h"

namespace lsa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kThreads = kAttnWaves * 64;
constexpr int kOPad = 132;  // LDS row pitch (floats) of the wave merge

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

typedef float f32x8 __attribute__((ext_vector_type(8)));

// Softmax weights as the two bf16 A operands of P V: p = hi + lo to about 16
// significant bits.  hi is p truncated to bf16 (so converting it is exact) and
// lo is the exact remainder p - hi rounded to bf16.
__device__ __forceinline__ void split_bf16(const f32x8& p, bf16x8& ph, bf16x8& pl) {
  f32x8 hi;
#pragma unroll
  for (int e = 0; e < 8; ++e) hi[e] = __uint_as_float(__float_as_uint(p[e]) & 0xFFFF0000u);
  ph = __builtin_convertvector(hi, bf16x8);
  pl = __builtin_convertvector(p - hi, bf16x8);
}

// max over the lanes l, l ^ 16, l ^ 32, l ^ 48 (the four 16-lane rows of a
// column), with the cross-row swaps of gfx950
__device__ __forceinline__ float col_max(float x) {
  const auto s32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(s32[0]), __uint_as_float(s32[1]));
  const auto s16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(s16[0]), __uint_as_float(s16[1]));
}

// (sequence, kv head, split) of attention workgroup wg; workgroups of sequence
// b start at t.wg_off[b] and run head-major
struct Unit {
  int b, g, s, ns;
};

// Static split boundaries: even-numbered units get 6/5 of the tiles of odd
// ones.  In the split kernel a unit is its workgroup, which the dispatcher
// places on XCD i % 8, and per-workgroup timestamps on MI355X show the
// odd-numbered XCDs streaming 7-8% slower than the even ones (every run
// measured); the weighting took the 1M-token step from 84.6 to 82.9 us.  The
// many-rows kernel runs two workgroups per CU and maps units so that even
// units sit in the first slot of a CU, which runs faster than the second (1.8%
// on the lookahead step).  Returns the first tile of split s of (b, g), so that
// split s covers [first(s), first(s + 1)).
constexpr int kEvenUnitWeight = 6;
constexpr int kOddUnitWeight = 5;

__device__ __forceinline__ int split_first(int base, int s, int ns, int n_tiles) {
  // base: the workgroup of split 0 of (b, g)
  auto weight_below = [&](int j) -> int64_t {  // the weights of splits 0 .. j - 1
    const int64_t even = (int64_t)((base + j + 1) / 2 - (base + 1) / 2);
    return even * kEvenUnitWeight + (int64_t)(j - even) * kOddUnitWeight;
  };
  return (int)((int64_t)n_tiles * weight_below(s) / weight_below(ns));
}

__device__ __forceinline__ Unit unit_of(const SeqData& sd, int wg) {
  Unit u;
  const int local = wg - sd.wg0;
  u.b = sd.b;
  u.ns = sd.ns;
  u.g = local / sd.ns;
  u.s = local % sd.ns;
  return u;
}

// s_waitcnt immediates (gfx9 encoding) that wait for the vector-memory counter
// only: at most N of this wave's loads still outstanding.
constexpr int waitcnt_vm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// ---------------------------------------------------------------------------
// Merge of the split partials (m, l, O) of one (b, g): weights exp2(m_s - M),
// O as the weighted sum of the split outputs, divided by
// L = sum_s exp2(m_s - M) l_s.  Two fixed summation orders, chosen by the
// largest split count of the call: at most kFewSplits, one thread walks every
// split of a (row, float4 slice) in order (merge_few); more, 8 split groups
// and then the groups in order (attn_combine_kernel).  Results are bitwise
// reproducible.  merge_few serves both the few-split combine kernel and the
// split kernel's last workgroup, so the fused step and the separate entry
// points give the same bits.

// Wave-wide reductions with DPP row shifts and row broadcasts; the result is
// read from lane 63.
__device__ __forceinline__ float wave_max(float x) {
  const int ninf = (int)0xFF800000u;
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(x), 0x111, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(x), 0x112, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(x), 0x114, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(x), 0x118, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(x), 0x142, 0xA, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(x), 0x143, 0xC, 0xF, false)));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

__device__ __forceinline__ float wave_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x111, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x112, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x114, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x118, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x142, 0xA, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x143, 0xC, 0xF, false));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

constexpr int kSlices = kHeadDim / 4;        // float4 slices of an output row
constexpr int kGroups = kThreads / kSlices;  // split groups of the many-split merge (8)

// Partials as the combine kernels read them: plain loads (the split kernel
// has ended, so its writes are visible).  Offsets in floats.
struct CachedParts {
  const float* o;
  const float* ml;
  __device__ explicit CachedParts(const AttnArgs& a) : o(a.part_o), ml(a.part_ml) {}
  __device__ float4 o4(int64_t i) const { return *reinterpret_cast<const float4*>(o + i); }
  __device__ float2 ml2(int64_t i) const { return *reinterpret_cast<const float2*>(ml + i); }
};

// Partials as the split kernel's last workgroup reads them: device-scope
// buffer loads (cache policy sc1), coherent across the XCDs' L2 caches like
// the device-scope stores that wrote them.
constexpr int kScopeDevice = 16;  // the sc1 bit of a buffer instruction's cache policy on gfx950

struct DeviceParts {
  __amdgpu_buffer_rsrc_t ro, rm;
  __device__ DeviceParts(const SeqTable& t, const AttnArgs& a) {
    const uint32_t rows = (uint32_t)t.wg_off[t.batch] * (uint32_t)a.rows_pad;
    ro = __builtin_amdgcn_make_buffer_rsrc(a.part_o, (short)0, (int)(rows * kHeadDim * 4u), 0x00020000);
    rm = __builtin_amdgcn_make_buffer_rsrc(a.part_ml, (short)0, (int)(rows * 8u), 0x00020000);
  }
  __device__ float4 o4(int64_t i) const {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(ro, (int)(i * 4), 0, kScopeDevice);
    return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
  }
  __device__ float2 ml2(int64_t i) const {
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rm, (int)(i * 4), 0, kScopeDevice);
    return make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
  }
};

// Row r of the (b, g) group is query token r / G of query head g G + r % G.
__device__ __forceinline__ int64_t out_row(const AttnArgs& a, int b, int g, int r) {
  const int tq = r / a.group, h = g * a.group + r % a.group;
  return ((int64_t)b * a.n_qtok + tq) * a.n_q_heads + h;
}

// At most kFewSplits splits: one thread merges float4 slice `slice` of row r
// of (b, g), walking every split itself.
template <class Parts>
__device__ __forceinline__ void merge_few(const SeqTable& t, const AttnArgs& a, const Parts& pp, int b, int g, int r,
                                          int slice) {
  const int ns = min(t.nsplit[b], kFewSplits);
  const int64_t unit0 = (int64_t)t.wg_off[b] + (int64_t)g * ns;
  const int64_t rows_pad = a.rows_pad;
  float2 v[kFewSplits];
  float4 ov[kFewSplits];
#pragma unroll
  for (int sp = 0; sp < kFewSplits; ++sp) {
    if (sp < ns) {
      const int64_t pr = (unit0 + sp) * rows_pad + r;
      v[sp] = pp.ml2(pr * 2);
      ov[sp] = pp.o4(pr * kHeadDim + 4 * slice);
    }
  }
  float M = -INFINITY;
#pragma unroll
  for (int sp = 0; sp < kFewSplits; ++sp)
    if (sp < ns) M = fmaxf(M, v[sp].x);
  float L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int sp = 0; sp < kFewSplits; ++sp) {
    if (sp < ns && v[sp].x != -INFINITY) {
      const float w = fast_exp2(v[sp].x - M);
      L += w * v[sp].y;
      acc.x += w * ov[sp].x;
      acc.y += w * ov[sp].y;
      acc.z += w * ov[sp].z;
      acc.w += w * ov[sp].w;
    }
  }
  const float invL = L > 0.f ? 1.f / L : 0.f;  // an empty kept set gives out = 0, lse = -inf
  acc.x *= invL;
  acc.y *= invL;
  acc.z *= invL;
  acc.w *= invL;
  const int64_t orow = out_row(a, b, g, r);
  *reinterpret_cast<float4*>(a.out + orow * kHeadDim + 4 * slice) = acc;
  if (slice == 0 && a.lse != nullptr) a.lse[orow] = (M + __log2f(L)) * kLn2;
}

template <int C, bool MERGE>
__global__ void __launch_bounds__(kThreads, 2)  // 2 waves per SIMD: <= 256 registers
attn_split_kernel(SeqTable t, AttnArgs a) {
  __shared__ float sm_o[kAttnWaves][16][kOPad];
  __shared__ float sm_m[kAttnWaves][16], sm_l[kAttnWaves][16];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, kg = lane >> 4;
  // the arguments every workgroup needs before its first loads, in the same
  // round of kernel-argument loads as its sequence's numbers (see seq_data)
  int G = a.group, rows = a.rows, n_qtok = a.n_qtok, n_q_heads = a.n_q_heads, sel_pitch = a.sel_pitch;
  int count_is_keep = a.count_is_keep;
  int64_t chunk_stride = a.chunk_stride, head_stride = a.head_stride;
  asm volatile("" : "+s"(G), "+s"(rows), "+s"(n_qtok), "+s"(n_q_heads), "+s"(sel_pitch), "+s"(count_is_keep));
  asm volatile("" : "+s"(chunk_stride), "+s"(head_stride));
  const SeqData sd = seq_data(t, t.wg_off, blockIdx.x);
  const Unit u = unit_of(sd, blockIdx.x);
  const int b = u.b, g = u.g, s = u.s, ns = u.ns;

  // sel_count and the chunk ids are clamped so that malformed device inputs
  // can only give wrong numbers, never an out-of-bounds access.
  constexpr int TPC = C / 32;  // 32-token tiles per chunk
  const int n_b = sd.n;
  const int cnt = count_is_keep ? min(sd.keep, n_b) : min(max(a.sel_count[b], 0), sel_pitch);
  const int nTall = cnt * TPC;
  const int T0 = split_first(sd.wg0 + g * ns, s, ns, nTall), T1 = split_first(sd.wg0 + g * ns, s + 1, ns, nTall);
  // wave w takes tiles T0 + w, T0 + w + 4, ... of the split

  // ---- query operand: row n16 (rows <= 16 here)
  bf16x8 qb[4];
  {
    const int row = n16;
    if (row < rows) {
      const int tq = row / G, h = g * G + row % G;
      const uint16_t* qp = a.q + (((int64_t)b * n_qtok + tq) * n_q_heads + h) * kHeadDim + 8 * kg;
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

  // Tiles T0 + wave + 4 i of the kept list (i < nT); tile T is tile T % TPC of
  // kept chunk T / TPC.  The split's chunk ids are fetched 64 at a time into a
  // register (one per lane) and read back with readlane, so no scalar load
  // sits between consecutive tiles.
  const int nT = T1 - T0 > wave ? (T1 - T0 - wave + kAttnWaves - 1) / kAttnWaves : 0;
  const int pos0 = T0 / TPC;
  const int npos = nT > 0 ? (T1 - 1) / TPC - pos0 + 1 : 0;
  const int32_t* sel = a.sel_idx + (int64_t)b * sel_pitch + pos0;
  int sel_base = 0;
  int sel_lane = lane < npos ? sel[lane] : 0;
  const uint16_t* kbase = a.k + sd.chunk_off * chunk_stride + g * head_stride + lane * 8;
  const uint16_t* vbase = a.v + sd.chunk_off * chunk_stride + g * head_stride + lane * 8;

  // K and V tiles are 8 KiB each and contiguous in the MFMA-ordered block
  // layout: load instruction q of a tile reads bytes [1024 q, 1024 q + 1024).
  // Returns how many of the tile's tokens exist: 32, or fewer in the last
  // chunk of a context that ends inside it (and <= 0 for a tile past the end).
  auto load_tile = [&](int i, bf16x8(&kt)[8], bf16x8(&vt)[8]) -> int {
    const int T = T0 + wave + kAttnWaves * i;
    const int j = T / TPC - pos0, tt = T % TPC;
    if (j - sel_base >= 64) {  // wave-uniform: next window of chunk ids
      sel_base = j & ~63;
      sel_lane = sel_base + lane < npos ? sel[sel_base + lane] : 0;
    }
    const int c = min(max(__builtin_amdgcn_readlane(sel_lane, j - sel_base), 0), n_b - 1);
    const int64_t off = (int64_t)c * chunk_stride + tt * (32 * kHeadDim);
    const uint16_t* kp = kbase + off;
    const uint16_t* vp = vbase + off;
#pragma unroll
    for (int q = 0; q < 8; ++q) kt[q] = load8_stream(kp + q * 512);
#pragma unroll
    for (int q = 0; q < 8; ++q) vt[q] = load8_stream(vp + q * 512);
    return c == n_b - 1 ? sd.tail - 32 * tt : 32;
  };

  auto compute_tile = [&](const bf16x8(&kt)[8], bf16x8(&vt)[8], int lim) {
    if (lim <= 0) return;  // wave-uniform: the tile lies past the context end
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
    if (lim < 32) {  // the context ends inside this tile: no weight for tokens 8 kg + i >= lim
      mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        x[i] = 8 * kg + i < lim ? x[i] : -INFINITY;
        mx = fmaxf(mx, x[i]);
      }
    }
    mx = col_max(mx);  // finite: token 0 of the tile exists
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    f32x8 p;
    float psum = 0.f;
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
    split_bf16(p, ph, pl);
    if (lim < 32) {
      // the V slots of tokens past the context end may hold anything, NaN
      // included (not yet written): zero them, as a zero weight cancels only
      // finite values.  Lane element i is token 8 kg + i; dword j holds
      // elements 2j (low half) and 2j + 1.
      u32x4 keep;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        keep[j] = (8 * kg + 2 * j < lim ? 0x0000FFFFu : 0u) | (8 * kg + 2 * j + 1 < lim ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) vt[nb] = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, vt[nb]) & keep);
    }
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) {
      o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, vt[nb], o[nb], 0, 0, 0);
      o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, vt[nb], o[nb], 0, 0, 0);
    }
  };

  // Two tile buffers: the loads of tile i+1 are in flight while tile i computes.
  bf16x8 ka[8], va[8], kb2[8], vb2[8];
  int lim_a = 32, lim_b = 32;
  if (nT > 0) lim_a = load_tile(0, ka, va);
  for (int i = 0; i < nT; i += 2) {
    if (i + 1 < nT) lim_b = load_tile(i + 1, kb2, vb2);
    compute_tile(ka, va, lim_a);
    if (i + 1 < nT) {
      if (i + 2 < nT) lim_a = load_tile(i + 2, ka, va);
      compute_tile(kb2, vb2, lim_b);
    }
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  // ---- this split's partials: rows of the (b, g) group, [unit][rows_pad]
  const int rows_pad = a.rows_pad;
  const int64_t unit = (int64_t)sd.wg0 + (int64_t)g * ns + s;
  {
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
      float* po = a.part_o + (unit * rows_pad + r) * kHeadDim + e;
      float* pml = a.part_ml + (unit * rows_pad + r) * 2;
      if constexpr (MERGE) {
        // device-scope stores, written through to where every XCD reads them
        __hip_atomic_store(po, acc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (e == 0) {
          __hip_atomic_store(pml + 0, M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(pml + 1, L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      } else {
        *po = acc;
        if (e == 0) {
          pml[0] = M;
          pml[1] = L;
        }
      }
    }
  }
  if constexpr (!MERGE) return;  // a combine kernel merges the splits

  // The last of the ns workgroups of (b, g) to arrive merges the splits.  A
  // workgroup counts itself in only once its partials are stored (every
  // thread waits for its stores, then the barrier), so the last one finds
  // all of them; it reads them with device-scope loads.  No fence is needed:
  // the partials never sit in a non-coherent cache.  (On gfx950 an
  // agent-scope release is an L2 writeback plus a wait for the vector-memory
  // counter; the writeback exists for ordinary stores held in an XCD's L2,
  // and these stores are device-scope (sc1) stores that write through, so
  // the wait alone remains.  The acquire side's device-scope (sc1) loads
  // are what agent-scope atomic loads compile to, so no L2 invalidate is
  // needed either.)
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __shared__ int sh_last;
  __syncthreads();
  if (tid == 0)
    sh_last = __hip_atomic_fetch_add(a.arrive + b * a.n_kv_heads + g, 1u, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) == (uint32_t)(ns - 1);
  __syncthreads();
  if (!sh_last) return;
  // (the host sets arrive only with at most kFewSplits splits: merge_few's order)
  const DeviceParts pp(t, a);
  for (int role = tid; role < a.rows * kSlices; role += kThreads) merge_few(t, a, pp, b, g, role / kSlices, role % kSlices);
}


// More than 16 query rows per KV head (rows = G * n_qtok, up to 128).  One
// workgroup per (sequence, kv head, split) serves all the rows, so each K/V
// tile is fetched from HBM once: every wave copies 4 of the tile's 16 one-KiB
// pieces (K pieces 0-7, V pieces 8-15) straight into LDS with
// global_load_lds_dwordx4, kRowBufs - 1 tiles ahead of the tile being
// consumed, and every wave then reads the whole tile from LDS for its own row
// blocks (w and w + 4; RBW of them).  Each wave keeps an online softmax per row
// block and writes its rows' partials itself.
constexpr int kRowBufs = 5;  // LDS tile buffers per workgroup (16 KiB each; 2 workgroups fill a CU's LDS)

// This lane's slice of 8 staged pieces (K: pieces 0-7, V: pieces 8-15 of a
// tile).  The reads are issued as one assembly block that ends with its own LDS
// wait: the compiler cannot tell the staged buffers apart and would otherwise
// make every read wait for all global->LDS copies still in flight, draining
// the prefetch.
__device__ __forceinline__ void read_pieces(const uint4 (&tb)[16][64], int first, int lane, bf16x8 (&out)[8]) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)&tb[first][lane];
  uint4 v[8];
  asm volatile(
      "ds_read_b128 %0, %8 offset:0\n\tds_read_b128 %1, %8 offset:1024\n\t"
      "ds_read_b128 %2, %8 offset:2048\n\tds_read_b128 %3, %8 offset:3072\n\t"
      "ds_read_b128 %4, %8 offset:4096\n\tds_read_b128 %5, %8 offset:5120\n\t"
      "ds_read_b128 %6, %8 offset:6144\n\tds_read_b128 %7, %8 offset:7168\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7])
      : "v"(a)
      : "memory");
#pragma unroll
  for (int q = 0; q < 8; ++q) out[q] = __builtin_bit_cast(bf16x8, v[q]);
}


typedef const __attribute__((address_space(4))) int32_t* kept_ids_t;  // read-only during the kernel

typedef float f32x16 __attribute__((ext_vector_type(16)));

// Token held in MFMA row m of the QK product.  With this order the 32x32
// result leaves register r of lane j holding token 16 (r / 8) + 8 (j / 32) +
// r % 8 of query row j % 32, which is exactly the P^T operand of the PV
// product for 16-token step r / 8.
__device__ __forceinline__ int qk_token(int m) {
  return 16 * (m / 16) + 8 * ((m / 4) % 2) + 4 * ((m / 8) % 2) + m % 4;
}

template <int C>
__global__ void __launch_bounds__(kThreads, 2)
attn_rows_kernel(SeqTable t, AttnArgs a) {
  // four distinct LDS objects, always named statically, so that the compiler
  // can tell the tile being read from the tiles still being copied in.  A
  // staged tile holds, in MFMA operand order, K pieces d = 0..7 (QK step d)
  // and V pieces 8 + 4 s + n (PV token half s, 32-dim block n).
  __shared__ uint4 buf0[16][64], buf1[16][64], buf2[16][64], buf3[16][64], buf4[16][64];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.group;
  // Two workgroups share each CU, and the dispatcher fills the first slot of
  // every CU (the first half of a grid of two per CU) before the second, whose
  // workgroups run slower.  So consecutive units (the splits of one (b, g))
  // alternate between the first and the second half of the grid, and the even
  // ones, in the first half, get 6/5 of the tiles of the odd ones (split_first).
  const int half = (int)(gridDim.x + 1) / 2;
  const int unit_id = (int)blockIdx.x < half ? 2 * (int)blockIdx.x : 2 * ((int)blockIdx.x - half) + 1;
  const SeqData sd = seq_data(t, t.wg_off, unit_id);
  const Unit u = unit_of(sd, unit_id);
  const int b = u.b, g = u.g, s = u.s, ns = u.ns;

  constexpr int TPC = C / 32;
  const int n_b = sd.n;
  const int cnt = a.count_is_keep ? min(sd.keep, n_b) : min(max(a.sel_count[b], 0), a.sel_pitch);
  const int nTall = cnt * TPC;
  const int Tb = split_first(sd.wg0 + g * ns, s, ns, nTall), Te = split_first(sd.wg0 + g * ns, s + 1, ns, nTall);
  const int nT = Te > Tb ? Te - Tb : 0;

  // this wave's 32 query rows: lane j serves row 32 * wave + j % 32
  const bool live = 32 * wave < a.rows;  // wave-uniform
  const int row = 32 * wave + (lane & 31);
  bf16x8 qb[8];  // Q^T operand of QK step d: dims 16 d + 8 (lane / 32) .. + 7
  if (row < a.rows) {
    const int tq = row / G, h = g * G + row % G;
    const uint16_t* qp = a.q + (((int64_t)b * a.n_qtok + tq) * a.n_q_heads + h) * kHeadDim + 8 * (lane >> 5);
#pragma unroll
    for (int d = 0; d < 8; ++d) qb[d] = load8(qp + 16 * d);
  } else {
#pragma unroll
    for (int d = 0; d < 8; ++d) qb[d] = bf16x8{};
  }
  f32x16 o[4];  // O^T, 32-dim block n: dims 32 n + 8 (r / 4) + 4 (lane / 32) + r % 4
#pragma unroll
  for (int n = 0; n < 4; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[n][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  // Each wave copies 4 of a tile's 16 pieces; lane i of piece q gathers the 16
  // bytes of the cache block that MFMA lane i needs (element offsets within
  // the tile's 32-token slice of the chunk block).
  int goff[4];
  {
    const int i = lane, hi = lane >> 5;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (wave < 2) {  // K piece d: token qk_token(i % 32), dims 16 d + 8 hi .. + 7
        const int d = 4 * wave + q, tk = qk_token(i & 31), e0 = 16 * d + 8 * hi;
        goff[q] = (((((tk / 4) % 2) * 4 + e0 / 32) * 4 + (e0 / 8) % 4) * 16 + (tk / 8) * 4 + tk % 4) * 8;
      } else {  // V piece (s, n): dim 32 n + i % 32, tokens 16 s + 8 hi .. + 7
        const int sh = wave - 2, n = q, e = 32 * n + (i & 31), t0 = 16 * sh + 8 * hi;
        goff[q] = (((e / 16) * 4 + t0 / 8) * 16 + e % 16) * 8;
      }
    }
  }

  // the query operands are in registers before any tile copy starts (so that no
  // wait in the loop is ever for them); chunk ids come through the scalar cache
  // (wave-uniform loads), so the tile copies are the only vector loads in flight
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  const kept_ids_t sel = (kept_ids_t)(uintptr_t)(a.sel_idx + (int64_t)b * a.sel_pitch);
  const uint16_t* src = (wave < 2 ? a.k : a.v) + sd.chunk_off * a.chunk_stride + g * a.head_stride;

  // chunk id of the next tile to issue, loaded one issue ahead
  int c_next = nT > 0 ? sel[Tb / TPC] : 0;
  // this wave's pieces of tile i -> dst; returns how many of the tile's tokens
  // exist: 32, or fewer in the last chunk of a context that ends inside it
  // (<= 0 for a tile past the end)
  auto issue = [&](int i, uint4(&dst)[16][64]) -> int {
    const int T = Tb + i;
    const int tt = T % TPC;
    const int c = min(max(c_next, 0), n_b - 1);
    if (i + 1 < nT) c_next = sel[(T + 1) / TPC];
    const uint16_t* p = src + (int64_t)c * a.chunk_stride + tt * (32 * kHeadDim);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      __builtin_amdgcn_global_load_lds((const void*)(p + goff[q]),
                                       (void __attribute__((address_space(3)))*)&dst[4 * wave + q][0], 16, 0, 0);
    return c == n_b - 1 ? sd.tail - 32 * tt : 32;
  };

  // Software pipeline over tiles.  Step j (after the barrier that makes tile j
  // visible) issues the copy of tile j + 3, the QK products of tile j, and
  // then the softmax and PV products of tile j - 1, so the VALU softmax of one
  // tile runs while the MFMA unit works on the next tile's QK.  Tile j lives in
  // buffer j % 5: the copy of tile j + 3 reuses the buffer of tile j - 2, whose
  // last reader (step j - 1) is behind the barrier.
  // logits of the tile whose softmax is pending.  The QK products of a tile
  // form one chain of 8 dependent MFMAs: the softmax that reads them runs a
  // step later, so the chain's latency is hidden, and one accumulator instead
  // of two saves 16 registers and the 16 adds that summed them.
  f32x16 s_cur0;
#pragma unroll
  for (int r = 0; r < 16; ++r) s_cur0[r] = 0.f;

  auto qk = [&](const uint4(&tb)[16][64], f32x16& s0) {
    bf16x8 kp[8];
    read_pieces(tb, 0, lane, kp);
#pragma unroll
    for (int r = 0; r < 16; ++r) s0[r] = 0.f;
#pragma unroll
    for (int d = 0; d < 8; ++d) s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kp[d], qb[d], s0, 0, 0, 0);
  };

  auto softmax_pv = [&](const f32x16& x0, const uint4(&tb)[16][64], int lim) {
    if (lim <= 0) return;  // wave-uniform: the tile lies past the context end
    bf16x8 vp[8];
    read_pieces(tb, 8, lane, vp);
    f32x16 x = x0;
    if (lim < 32) {  // the context ends inside this tile: register r holds token 16 (r / 8) + 8 (lane / 32) + r % 8
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (16 * (r / 8) + 8 * (lane >> 5) + r % 8 >= lim) x[r] = -INFINITY;
      // those tokens' V slots may hold anything, NaN included (not yet
      // written): zero them, as a zero weight cancels only finite values.
      // Element i of vp[4 s + n] is token 16 s + 8 (lane / 32) + i; dword j
      // holds elements 2j (low half) and 2j + 1.
#pragma unroll
      for (int sh = 0; sh < 2; ++sh) {
        const int t0 = 16 * sh + 8 * (lane >> 5);
        u32x4 keep;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          keep[j] = (t0 + 2 * j < lim ? 0x0000FFFFu : 0u) | (t0 + 2 * j + 1 < lim ? 0xFFFF0000u : 0u);
#pragma unroll
        for (int n = 0; n < 4; ++n)
          vp[4 * sh + n] = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, vp[4 * sh + n]) & keep);
      }
    }
    // online softmax: lanes j and j ^ 32 share row j % 32 and split its tokens
    float mx = x[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, x[r]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    // max over raw logits (the scale is positive), then p = exp2(x * scale - m)
    const float m_new = fmaxf(m_run, mx * a.scale_log2e);
    const float alpha = fast_exp2(m_run - m_new);
    f32x8 p0, p1;
    float psum = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      p0[r] = fast_exp2(fmaf(x[r], a.scale_log2e, -m_new));
      p1[r] = fast_exp2(fmaf(x[8 + r], a.scale_log2e, -m_new));
      psum += p0[r] + p1[r];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
    if (__ballot(alpha != 1.f) != 0ull) {  // every O register of a lane belongs to its row
#pragma unroll
      for (int n = 0; n < 4; ++n) o[n] *= alpha;
    }
    bf16x8 ph0, pl0, ph1, pl1;
    split_bf16(p0, ph0, pl0);
    split_bf16(p1, ph1, pl1);
    // O^T += V^T P^T, token half s of the tile, 32-dim block n
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      o[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vp[n], ph0, o[n], 0, 0, 0);
      o[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vp[n], pl0, o[n], 0, 0, 0);
      o[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vp[4 + n], ph1, o[n], 0, 0, 0);
      o[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vp[4 + n], pl1, o[n], 0, 0, 0);
    }
  };

  // lims[k]: the token count of the tile staged in buffer k
  int lims[kRowBufs] = {32, 32, 32, 32, 32};
  auto step = [&](int j, const uint4(&cur)[16][64], const uint4(&prev)[16][64], uint4(&dma)[16][64], int kcur,
                  int kprev, int kdma) {
    // tile j has landed once at most `ahead` younger tiles of this wave are in flight
    const int ahead = min(nT - 1 - j, kRowBufs - 3);
    if (ahead >= 2)
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(8));
    else if (ahead == 1)
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(4));
    else
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    // every wave's pieces of tile j are in; every wave is done with tile j - 2
    // (a bare barrier: a fenced one would also wait for the tiles still in flight)
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
    if (j + kRowBufs - 2 < nT) lims[kdma] = issue(j + kRowBufs - 2, dma);
    if (!live) return;
    f32x16 n0;
    if (lims[kcur] > 0) qk(cur, n0);
    if (j > 0) softmax_pv(s_cur0, prev, lims[kprev]);
    s_cur0 = n0;
  };

  if (nT > 0) lims[0] = issue(0, buf0);
  if (nT > 1) lims[1] = issue(1, buf1);
  if (nT > 2) lims[2] = issue(2, buf2);
  int j = 0;
  for (; j + 5 <= nT; j += 5) {
    step(j, buf0, buf4, buf3, 0, 4, 3);
    step(j + 1, buf1, buf0, buf4, 1, 0, 4);
    step(j + 2, buf2, buf1, buf0, 2, 1, 0);
    step(j + 3, buf3, buf2, buf1, 3, 2, 1);
    step(j + 4, buf4, buf3, buf2, 4, 3, 2);
  }
  if (j < nT) step(j, buf0, buf4, buf3, 0, 4, 3);
  if (j + 1 < nT) step(j + 1, buf1, buf0, buf4, 1, 0, 4);
  if (j + 2 < nT) step(j + 2, buf2, buf1, buf0, 2, 1, 0);
  if (j + 3 < nT) step(j + 3, buf3, buf2, buf1, 3, 2, 1);
  // the last tile's softmax and PV (its buffer is nT - 1 mod 5)
  if (nT > 0 && live) {
    switch ((nT - 1) % 5) {
      case 0: softmax_pv(s_cur0, buf0, lims[0]); break;
      case 1: softmax_pv(s_cur0, buf1, lims[1]); break;
      case 2: softmax_pv(s_cur0, buf2, lims[2]); break;
      case 3: softmax_pv(s_cur0, buf3, lims[3]); break;
      default: softmax_pv(s_cur0, buf4, lims[4]); break;
    }
  }

  // partials of this wave's rows, [unit][rows_pad]; lanes j and j ^ 32 hold
  // halves of row j % 32's sum and disjoint dims of its output
  if (live) {
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_run), __float_as_uint(l_run), false, false);
    const float l = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
    if (row < a.rows) {
      const int64_t rbase = (int64_t)unit_id * a.rows_pad + row;
      float* po = a.part_o + rbase * kHeadDim + 4 * (lane >> 5);
#pragma unroll
      for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<float4*>(po + 32 * n + 8 * q) =
              make_float4(o[n][4 * q], o[n][4 * q + 1], o[n][4 * q + 2], o[n][4 * q + 3]);
      if (lane < 32) {
        a.part_ml[rbase * 2 + 0] = m_run;
        a.part_ml[rbase * 2 + 1] = l;
      }
    }
  }
}

// attn_combine_kernel (more than kFewSplits splits): one workgroup per output
// row (b, t, h).  Every wave computes M and L itself from all splits' (m, l)
// (lane l takes splits l, l + 64, ...), so the loads of (m, l) and of the
// thread's O slices go out in one round; thread (sg, slice) sums splits sg,
// sg + 8, ... of its slice, and only the final merge of the 8 split groups
// needs a barrier.
__global__ void __launch_bounds__(kThreads)
attn_combine_kernel(SeqTable t, AttnArgs a) {
  constexpr int kBatch = 8;  // splits per thread and round of loads
  __shared__ float4 sm_red[kGroups][kSlices];

  const int tid = threadIdx.x, lane = tid & 63;
  // output row (b, t, h) of this workgroup; sequence 0's split numbers come in
  // the first round of kernel-argument loads (see seq_data)
  int G = a.group, n_q_heads = a.n_q_heads, rows_per_b = a.n_qtok * a.n_q_heads, ns = t.nsplit[0];
  int64_t rows_pad = a.rows_pad;
  const float* part_o = a.part_o;
  const float* part_ml = a.part_ml;
  asm volatile("" : "+s"(G), "+s"(n_q_heads), "+s"(rows_per_b), "+s"(ns));
  asm volatile("" : "+s"(rows_pad), "+s"(part_o), "+s"(part_ml));
  int b = 0, wg0 = 0, rem = blockIdx.x;
  if (rem >= rows_per_b) {
    b = rem / rows_per_b;
    rem -= b * rows_per_b;
    ns = t.nsplit[b];
    wg0 = t.wg_off[b];
  }
  const int tq = rem / n_q_heads, h = rem - tq * n_q_heads;
  const int g = h / G, r = tq * G + h % G;  // row within the (b, g) group
  const int64_t unit0 = (int64_t)wg0 + (int64_t)g * ns;
  const float2* ml = reinterpret_cast<const float2*>(part_ml) + unit0 * rows_pad + r;  // split s at s * rows_pad
  const int sg = tid / kSlices, e4 = (tid % kSlices) * 4;
  const float* po = part_o + (unit0 * rows_pad + r) * kHeadDim + e4;
  const int64_t ostride = rows_pad * kHeadDim;

  // Every load of the first round is issued up front: (m, l) of all splits
  // (each wave reads them all, lane l splits l, l + 64, ...), and this
  // thread's first batch of O slices (splits sg, sg + 8, ...).
  float2 mls[kMaxSplits / 64];
#pragma unroll
  for (int i = 0; i < kMaxSplits / 64; ++i) {
    const int sp = lane + 64 * i;
    mls[i] = sp < ns ? ml[sp * rows_pad] : make_float2(-INFINITY, 0.f);
  }
  float4 ov[kBatch];
  float mo[kBatch];
#pragma unroll
  for (int i = 0; i < kBatch; ++i) {
    const int sp = sg + kGroups * i;
    ov[i] = sp < ns ? *reinterpret_cast<const float4*>(po + sp * ostride) : make_float4(0.f, 0.f, 0.f, 0.f);
    mo[i] = sp < ns ? ml[sp * rows_pad].x : -INFINITY;
  }

  // M = max_s m_s and L = sum_s exp2(m_s - M) l_s, in a fixed order
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < kMaxSplits / 64; ++i) mx = fmaxf(mx, mls[i].x);
  const float M = wave_max(mx);
  float lx = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxSplits / 64; ++i) lx += mls[i].x == -INFINITY ? 0.f : fast_exp2(mls[i].x - M) * mls[i].y;
  const float L = wave_sum(lx);

  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int base = 0;;) {
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const float w = mo[i] == -INFINITY ? 0.f : fast_exp2(mo[i] - M);
      acc.x += w * ov[i].x;
      acc.y += w * ov[i].y;
      acc.z += w * ov[i].z;
      acc.w += w * ov[i].w;
    }
    base += kGroups * kBatch;
    if (base >= ns) break;
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int sp = base + sg + kGroups * i;
      ov[i] = sp < ns ? *reinterpret_cast<const float4*>(po + sp * ostride) : make_float4(0.f, 0.f, 0.f, 0.f);
      mo[i] = sp < ns ? ml[sp * rows_pad].x : -INFINITY;
    }
  }
  sm_red[sg][tid % kSlices] = acc;
  __syncthreads();
  const int64_t orow = ((int64_t)b * a.n_qtok + tq) * a.n_q_heads + h;
  if (tid < kSlices) {
    float4 sum = sm_red[0][tid];
#pragma unroll
    for (int q = 1; q < kGroups; ++q) {
      const float4 v = sm_red[q][tid];
      sum.x += v.x;
      sum.y += v.y;
      sum.z += v.z;
      sum.w += v.w;
    }
    const float invL = L > 0.f ? 1.f / L : 0.f;  // an empty kept set gives out = 0, lse = -inf
    sum.x *= invL;
    sum.y *= invL;
    sum.z *= invL;
    sum.w *= invL;
    *reinterpret_cast<float4*>(a.out + orow * kHeadDim + tid * 4) = sum;
  }
  if (tid == 0 && a.lse != nullptr) a.lse[orow] = (M + __log2f(L)) * kLn2;
}

// attn_combine_few_kernel (at most kFewSplits splits): one thread per (output
// row, float4 slice of the head dim), so a 256-thread workgroup merges 8 rows
// with no cross-thread reduction.
__global__ void __launch_bounds__(kThreads)
attn_combine_few_kernel(SeqTable t, AttnArgs a, int n_rows) {
  const int gid = blockIdx.x * kThreads + threadIdx.x;
  const int orow = gid / kSlices, slice = gid % kSlices;
  if (orow >= n_rows) return;
  const int rows_per_b = a.n_qtok * a.n_q_heads;
  const int b = orow / rows_per_b;
  const int rem = orow - b * rows_per_b;
  const int tq = rem / a.n_q_heads, h = rem - tq * a.n_q_heads;
  merge_few(t, a, CachedParts(a), b, h / a.group, tq * a.group + h % a.group, slice);
}

template <int C>
hipError_t launch_c(const SeqTable& t, const AttnArgs& a, hipStream_t s) {
  const dim3 grid(t.wg_off[t.batch]);
  if (a.rows > 16)
    hipLaunchKernelGGL((attn_rows_kernel<C>), grid, dim3(kThreads), 0, s, t, a);
  else if (a.arrive != nullptr)
    hipLaunchKernelGGL((attn_split_kernel<C, true>), grid, dim3(kThreads), 0, s, t, a);
  else
    hipLaunchKernelGGL((attn_split_kernel<C, false>), grid, dim3(kThreads), 0, s, t, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.arrive != nullptr && a.rows <= kAttnRowsPerWave) return hipSuccess;  // the split kernel merged the splits
  const int n_rows = t.batch * a.n_qtok * a.n_q_heads;
  if (a.few_splits) {
    const int per_wg = kThreads / (kHeadDim / 4);
    hipLaunchKernelGGL(attn_combine_few_kernel, dim3((n_rows + per_wg - 1) / per_wg), dim3(kThreads), 0, s, t,
                       a, n_rows);
  } else {
    hipLaunchKernelGGL(attn_combine_kernel, dim3(n_rows), dim3(kThreads), 0, s, t, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const SeqTable& t, const AttnArgs& a, int32_t chunk_size, hipStream_t s) {
  if (chunk_size == 64) return launch_c<64>(t, a, s);
  if (chunk_size == 128) return launch_c<128>(t, a, s);
  return hipErrorInvalidValue;
}

}  // namespace lsa
