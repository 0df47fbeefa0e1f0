// Device side of the seeded input generator: fills a chunk-paged K or V cache
// in HBM with the same counter-based values that synth.c produces on the host.
//
// Test and benchmark infrastructure only; holds none of the method's
// arithmetic.  The value of the element at global token tau, KV head h and
// dimension e is table[draw(key, (tau * hkv + h) * d + e) >> 48], with draw the
// SplitMix64 counter generator (Steele, Lea, Flood, OOPSLA 2014).
//
// Physical layout of one (chunk, head) block of chunk*d elements:
//   inner_transposed == 0 : [token][dim]  (element t*d + e)
//   inner_transposed == 1 : [dim][token]  (element e*chunk + t)
// The block of global chunk c and head h starts at c*chunk_stride + h*head_stride.
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
        int64_t chunk_stride, int64_t head_stride, int32_t inner_transposed) {
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
      int64_t t, e;
      if (inner_transposed) { e = inner / chunk; t = inner - e * chunk; }
      else { t = inner / d; e = inner - t * d; }
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

}  // namespace

// Returns 0 on success, 1 on a bad argument, 2 on a HIP launch error.
extern "C" int synth_fill_kv_device(uint64_t key, const uint16_t* table, uint16_t* out,
                                    int64_t total_chunks, int32_t hkv, int32_t chunk,
                                    int32_t d, int64_t chunk_stride, int64_t head_stride,
                                    int32_t inner_transposed, void* stream) {
  if (!table || !out || total_chunks <= 0 || hkv <= 0 || chunk <= 0 || d <= 0) return 1;
  if (((int64_t)chunk * d) % 8 != 0 || chunk_stride % 8 != 0 || head_stride % 8 != 0) return 1;
  if ((reinterpret_cast<uintptr_t>(out) & 15) != 0) return 1;
  const int64_t total = total_chunks * hkv * ((int64_t)chunk * d / 8);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_kv, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, key,
                     table, out, total_chunks, hkv, chunk, d, chunk_stride, head_stride,
                     inner_transposed);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
