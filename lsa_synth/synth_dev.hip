// Device side of the seeded input generator: fills a chunk-paged K or V cache
// in HBM with the same counter-based values that synth.c produces on the host.
//
// Test and benchmark infrastructure only; holds none of the method's
// arithmetic.  The value of the element at global token tau, KV head h and
// dimension e is table[draw(key, (tau * hkv + h) * d + e) >> 48], with draw the
// SplitMix64 counter generator (Steele, Lea, Flood, OOPSLA 2014).
//
// The block of global chunk c and KV head h starts at c*chunk_stride +
// h*head_stride and holds chunk*128 bf16 values in the MFMA operand order of
// the decode-attention library (head_dim 128, chunk a multiple of 32):
//   K (value_block == 0): token t, dim e at
//     ((((t/32*2 + t/4%2)*4 + e/32)*4 + e/8%4)*16 + t%32/8*4 + t%4)*8 + e%8
//   V (value_block == 1): token t, dim e at
//     (((t/32*8 + e/16)*4 + t%32/8)*16 + e%16)*8 + t%8
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ULL;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

__global__ void __launch_bounds__(256)
fill_kv(uint64_t key, const uint16_t* __restrict__ table, uint16_t* __restrict__ out,
        int64_t total_chunks, int32_t hkv, int32_t chunk, int32_t d,
        int64_t chunk_stride, int64_t head_stride, int32_t value_block) {
  const int64_t block_elems = (int64_t)chunk * d;
  const int64_t groups_per_block = block_elems / 8;
  const int64_t total = total_chunks * hkv * groups_per_block;
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < total;
       w += (int64_t)gridDim.x * blockDim.x) {
    const int64_t blk = w / groups_per_block;
    const int64_t inner0 = (w - blk * groups_per_block) * 8;
    const int64_t c = blk / hkv;
    const int32_t h = (int32_t)(blk - c * hkv);
    uint16_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t inner = inner0 + j;
      const int64_t w = inner % 8, n16 = (inner / 8) % 16, kg = (inner / 128) % 4;
      int64_t t, e;
      if (value_block) {
        const int64_t nb = (inner / 512) % 8, tt = inner / 4096;
        t = 32 * tt + 8 * kg + w;
        e = 16 * nb + n16;
      } else {
        const int64_t jj = (inner / 512) % 4, hf = (inner / 2048) % 2, tt = inner / 4096;
        t = 32 * tt + 8 * (n16 / 4) + 4 * hf + n16 % 4;
        e = 8 * (kg + 4 * jj) + w;
      }
      const int64_t tau = c * chunk + t;
      const uint64_t idx = (uint64_t)((tau * hkv + h) * d + e);
      v[j] = table[mix64(key + (idx + 1ULL) * kGamma) >> 48];
    }
    uint4 packed;
    packed.x = (uint32_t)v[0] | ((uint32_t)v[1] << 16);
    packed.y = (uint32_t)v[2] | ((uint32_t)v[3] << 16);
    packed.z = (uint32_t)v[4] | ((uint32_t)v[5] << 16);
    packed.w = (uint32_t)v[6] | ((uint32_t)v[7] << 16);
    *reinterpret_cast<uint4*>(out + c * chunk_stride + h * head_stride + inner0) = packed;
  }
}

// Token-major fill: row r of out holds the hkv x d values of global token
// tau_of_row[r] (the same values the paged fill puts in that token's
// positions), KV head h at r*tok_stride + h*head_stride; rows with a negative
// tau are left alone.
__global__ void __launch_bounds__(256)
fill_kv_tokens(uint64_t key, const uint16_t* __restrict__ table, uint16_t* __restrict__ out,
               const int64_t* __restrict__ tau_of_row, int64_t n_rows, int32_t hkv, int32_t d,
               int64_t tok_stride, int64_t head_stride) {
  const int64_t per_row = (int64_t)hkv * (d / 8);
  const int64_t total = n_rows * per_row;
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < total;
       w += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = w / per_row;
    const int64_t rem = w - r * per_row;
    const int32_t h = (int32_t)(rem / (d / 8));
    const int64_t e0 = (rem - (int64_t)h * (d / 8)) * 8;
    const int64_t tau = tau_of_row[r];
    if (tau < 0) continue;
    uint16_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint64_t idx = (uint64_t)((tau * hkv + h) * d + e0 + j);
      v[j] = table[mix64(key + (idx + 1ULL) * kGamma) >> 48];
    }
    uint4 packed;
    packed.x = (uint32_t)v[0] | ((uint32_t)v[1] << 16);
    packed.y = (uint32_t)v[2] | ((uint32_t)v[3] << 16);
    packed.z = (uint32_t)v[4] | ((uint32_t)v[5] << 16);
    packed.w = (uint32_t)v[6] | ((uint32_t)v[7] << 16);
    *reinterpret_cast<uint4*>(out + r * tok_stride + h * head_stride + e0) = packed;
  }
}

// Plain 16-byte copy, used only to calibrate hardware byte counters against a
// kernel whose traffic is known exactly (n16 * 16 bytes read and written).
__global__ void __launch_bounds__(256) copy16(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

// Plain streaming read, used only to measure the read-bandwidth ceiling of
// the device.  Workgroup g reads its own contiguous slice; per step a wave
// loads 4 x 1 KiB (nontemporal 16-byte loads), two steps in flight.  Each
// workgroup folds what it read into one word of `sink`, so the loads cannot be
// dropped.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kReadBlocks = 1024;
constexpr int64_t kReadStep16 = 1024;  // 16 KiB per workgroup step, in 16-byte units
__global__ void __launch_bounds__(256) read16(const u32x4* __restrict__ src, int64_t per_wg16, uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const u32x4* base = src + (int64_t)blockIdx.x * per_wg16 + w * 256 + lane;
  const int64_t steps = per_wg16 / kReadStep16;  // even: the host checks
  uint32_t acc = 0;
  for (int64_t i = 0; i < steps; i += 2) {
    u32x4 v[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = __builtin_nontemporal_load(base + i * kReadStep16 + q * 64);
#pragma unroll
    for (int q = 0; q < 4; ++q) v[4 + q] = __builtin_nontemporal_load(base + (i + 1) * kReadStep16 + q * 64);
#pragma unroll
    for (int q = 0; q < 8; ++q) acc ^= v[q].x ^ v[q].y ^ v[q].z ^ v[q].w;
  }
  acc |= __shfl_xor(acc, 1);
  if (threadIdx.x == 0) sink[blockIdx.x] = acc;
}

}  // namespace

// Returns 0 on success, 1 on a bad argument (bytes must be a positive
// multiple of 32 MiB), 2 on a HIP launch error.  `sink` must hold
// synth_read_sink_words() words.
extern "C" int synth_read_sink_words() { return kReadBlocks; }
extern "C" int synth_read_device(const void* src, int64_t bytes, uint32_t* sink, void* stream) {
  constexpr int64_t kUnit = (int64_t)kReadBlocks * 2 * kReadStep16 * 16;
  if (!src || !sink || bytes <= 0 || bytes % kUnit != 0 || (reinterpret_cast<uintptr_t>(src) & 15)) return 1;
  hipLaunchKernelGGL(read16, dim3(kReadBlocks), dim3(256), 0, (hipStream_t)stream, static_cast<const u32x4*>(src),
                     bytes / 16 / kReadBlocks, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" int synth_copy_device(const void* src, void* dst, int64_t bytes, void* stream) {
  if (!src || !dst || bytes <= 0 || bytes % 16 != 0) return 1;
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15) return 1;
  const int64_t n16 = bytes / 16;
  int64_t blocks = (n16 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(copy16, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     static_cast<const uint4*>(src), static_cast<uint4*>(dst), n16);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

// Golden-label logits: the same function as synth_golden_logits on the host,
// one element per thread iteration.
__global__ void __launch_bounds__(256)
fill_golden(uint64_t key_noise, uint64_t key_rel, uint64_t key_boost, const float* __restrict__ table,
            uint64_t start, int64_t total, int64_t n, int32_t b, float sigma, float beta, uint32_t rel_thr,
            uint32_t boost_thr, float* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t c = start + (uint64_t)i;
    const uint64_t d = mix64(key_noise + (c + 1ULL) * kGamma);
    const float z = __fadd_rn(table[d >> 48], (float)((d >> 32) & 0xFFFFu) * 0x1p-26f);
    float v = __fmul_rn(z, sigma);
    const int64_t s = i % n;
    const uint64_t rc = ((uint64_t)b << 32) | (uint64_t)s;
    const bool relevant = (uint32_t)(mix64(key_rel + (rc + 1ULL) * kGamma) >> 32) < rel_thr;
    if (relevant && (uint32_t)(mix64(key_boost + (c + 1ULL) * kGamma) >> 32) < boost_thr) v = __fadd_rn(v, beta);
    out[i] = v;
  }
}

extern "C" int synth_fill_golden_device(uint64_t key_noise, uint64_t key_rel, uint64_t key_boost, const float* table,
                                        uint64_t start, int64_t rows, int64_t n, int32_t b, float sigma, float beta,
                                        uint32_t rel_thr, uint32_t boost_thr, float* out, void* stream) {
  if (!table || !out || rows <= 0 || n <= 0) return 1;
  const int64_t total = rows * n;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_golden, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, key_noise, key_rel,
                     key_boost, table, start, total, n, b, sigma, beta, rel_thr, boost_thr, out);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

// Returns 0 on success, 1 on a bad argument, 2 on a HIP launch error.
extern "C" int synth_fill_kv_tokens_device(uint64_t key, const uint16_t* table, uint16_t* out,
                                           const int64_t* tau_of_row, int64_t n_rows, int32_t hkv, int32_t d,
                                           int64_t tok_stride, int64_t head_stride, void* stream) {
  if (!table || !out || !tau_of_row || n_rows <= 0 || hkv <= 0 || d != 128) return 1;
  if (tok_stride % 8 != 0 || head_stride % 8 != 0 || head_stride < d || tok_stride < (int64_t)hkv * head_stride)
    return 1;
  if ((reinterpret_cast<uintptr_t>(out) & 15) != 0) return 1;
  const int64_t total = n_rows * hkv * (d / 8);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_kv_tokens, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, key, table, out,
                     tau_of_row, n_rows, hkv, d, tok_stride, head_stride);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

// Returns 0 on success, 1 on a bad argument, 2 on a HIP launch error.
extern "C" int synth_fill_kv_device(uint64_t key, const uint16_t* table, uint16_t* out,
                                    int64_t total_chunks, int32_t hkv, int32_t chunk,
                                    int32_t d, int64_t chunk_stride, int64_t head_stride,
                                    int32_t value_block, void* stream) {
  if (!table || !out || total_chunks <= 0 || hkv <= 0 || chunk <= 0 || chunk % 32 != 0 || d != 128) return 1;
  if (((int64_t)chunk * d) % 8 != 0 || chunk_stride % 8 != 0 || head_stride % 8 != 0) return 1;
  if ((reinterpret_cast<uintptr_t>(out) & 15) != 0) return 1;
  const int64_t total = total_chunks * hkv * ((int64_t)chunk * d / 8);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_kv, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, key,
                     table, out, total_chunks, hkv, chunk, d, chunk_stride, head_stride,
                     value_block);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
