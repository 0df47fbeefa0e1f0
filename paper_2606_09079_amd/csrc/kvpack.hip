// Re-layout of a token-major K/V cache into the chunk-paged blocks that the
// attention kernels stream.
//
// The paper's serving stack keeps K/V token-major, row = token, [tokens][Hkv][d]
// with a ragged per-sequence offset (the paged cache of Sec. 2.1 and the KV
// layout of Sec. 2.5).  The attention here reads whole (chunk, KV head)
// blocks of C x 128 bf16 values in MFMA operand order instead, so that every
// 1 KiB it loads is one MFMA operand with no shuffle.  This kernel writes
// tokens [first_b, ctx_b) of every sequence into those blocks: the whole
// context once at prefill (first_b = 0), or the tokens decoded since the
// last call (one per step).
//
// One workgroup per (chunk in range, KV head).  The block's K and V token
// rows are loaded together (full 256-byte row segments per 16 lanes), then go
// through LDS in turn: written in token order, read back in block order and
// stored contiguously, 16 bytes per lane.  A K group holds 8
// consecutive dimensions of one token (one 16-byte LDS read); a V group holds
// one dimension of 8 consecutive tokens (eight 2-byte LDS reads, the
// transpose).  Tokens before the range are neither read nor written (a V
// group that straddles the range start is stored element by element); the
// positions past the context end in the last block are written as zeros, so
// a partial last chunk holds finite values only.  Global loads and stores
// are nontemporal: the data is touched once.
#include "lsa_internal.h"

namespace lsa {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kPackThreads = 256;
constexpr int kTilePitch = 136;  // bf16 elements per LDS row: 128 + 8 padding (272 B, 16-byte aligned)

// Token t and first dimension e0 of 16-byte group q of a K block (the K block
// layout of the attention's cache: lane groups of 4 tokens x 8 dimensions).
__device__ __forceinline__ void k_group(int q, int* t, int* e0) {
  const int n16 = q & 15, kg = (q >> 4) & 3, jj = (q >> 6) & 3, hf = (q >> 8) & 1, tt = q >> 9;
  *t = 32 * tt + 8 * (n16 >> 2) + 4 * hf + (n16 & 3);
  *e0 = 8 * (kg + 4 * jj);
}

// First token t0 and dimension e of group q of a V block (8 tokens of one
// dimension).
__device__ __forceinline__ void v_group(int q, int* t0, int* e) {
  const int n16 = q & 15, kq = (q >> 4) & 3, nb = (q >> 6) & 7, tt = q >> 9;
  *t0 = 32 * tt + 8 * kq;
  *e = 16 * nb + n16;
}

template <int C>
__global__ void __launch_bounds__(kPackThreads)
kv_pack_kernel(PackArgs a) {
  constexpr int kGroups = C * 16;                 // 16-byte groups per block
  constexpr int kPer = kGroups / kPackThreads;    // per thread: 4 (C = 64) or 8 (C = 128)
  __shared__ __attribute__((aligned(16))) uint16_t tile[C * kTilePitch];
  // the KV heads of one chunk are neighbours in the grid, so that the
  // workgroups in flight read whole token rows between them
  const int64_t u = blockIdx.x / a.n_kv_heads;
  const int g = (int)(blockIdx.x - u * a.n_kv_heads);
  // sequence of unit u: the count of later sequences starting at or before u
  // (starts are non-decreasing; all loaded at once, not one per step)
  int b = 0;
  if (a.batch > 1) {
#pragma unroll
    for (int j = 1; j < LSA_MAX_BATCH; ++j) b += (j < a.batch && a.unit_off[j] <= u) ? 1 : 0;
  }
  const int64_t c = a.first[b] / C + (u - a.unit_off[b]);  // chunk of sequence b
  const int lo = (int)(max(a.first[b], c * C) - c * C);
  const int hi = (int)(min(a.ctx[b], (c + 1) * C) - c * C);
  const int64_t row0 = a.tok_off[b] + c * C;  // source row of the block's token 0
  const int64_t dst = (a.chunk_off[b] + c) * a.chunk_stride + (int64_t)g * a.head_stride;
  const int64_t head = (int64_t)g * a.tok_head_stride;

  // every row segment of K and V in flight at once
  u32x4 xk[kPer], xv[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int p = threadIdx.x + r * kPackThreads, t = p >> 4, e0 = (p & 15) * 8;
    if (t >= lo && t < hi) {
      const int64_t off = (row0 + t) * a.tok_stride + head + e0;
      xk[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a.k_tok + off));
      xv[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a.v_tok + off));
    }
  }

  // K: a group is 8 dimensions of one token
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int p = threadIdx.x + r * kPackThreads, t = p >> 4, e0 = (p & 15) * 8;
    if (t >= lo && t < hi) *reinterpret_cast<u32x4*>(tile + t * kTilePitch + e0) = xk[r];
  }
  __syncthreads();
  u32x4* kout = reinterpret_cast<u32x4*>(a.k + dst);
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int q = threadIdx.x + r * kPackThreads;
    int t, e0;
    k_group(q, &t, &e0);
    if (t < lo) continue;
    u32x4 y = {0u, 0u, 0u, 0u};
    if (t < hi) y = *reinterpret_cast<const u32x4*>(tile + t * kTilePitch + e0);
    __builtin_nontemporal_store(y, kout + q);
  }
  __syncthreads();  // every read of K's tile is done

  // V: a group is one dimension of 8 consecutive tokens (the transpose)
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int p = threadIdx.x + r * kPackThreads, t = p >> 4, e0 = (p & 15) * 8;
    if (t >= lo && t < hi) *reinterpret_cast<u32x4*>(tile + t * kTilePitch + e0) = xv[r];
  }
  __syncthreads();
  uint16_t* vout = a.v + dst;
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int q = threadIdx.x + r * kPackThreads;
    int t0, e;
    v_group(q, &t0, &e);
    if (t0 + 8 <= lo) continue;
    uint16_t h[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = t0 + j < hi ? tile[(t0 + j) * kTilePitch + e] : (uint16_t)0;
    if (t0 >= lo) {
      u32x4 y;
      y.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
      y.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
      y.z = (uint32_t)h[4] | ((uint32_t)h[5] << 16);
      y.w = (uint32_t)h[6] | ((uint32_t)h[7] << 16);
      __builtin_nontemporal_store(y, reinterpret_cast<u32x4*>(vout) + q);
    } else {
      for (int j = 0; j < 8; ++j)
        if (t0 + j >= lo) vout[(int64_t)q * 8 + j] = h[j];
    }
  }
}

}  // namespace

hipError_t launch_kv_pack(const PackArgs& a, int64_t units, hipStream_t s) {
  if (units == 0) return hipSuccess;
  const dim3 grid((unsigned)(units * a.n_kv_heads));
  if (a.chunk == 64)
    hipLaunchKernelGGL(kv_pack_kernel<64>, grid, dim3(kPackThreads), 0, s, a);
  else
    hipLaunchKernelGGL(kv_pack_kernel<128>, grid, dim3(kPackThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace lsa
