// Seeded synthetic-input generator, device side (gfx950).
//
// Holds no part of the verification method. Produces, bit for bit, the same
// bf16 values as synth_host.c (SplitMix64 output function of a counter,
// Irwin-Hall sum of eight 16-bit fields, one fp32 multiply, bf16
// round-to-nearest-even), so that a 30-130 GB synthetic model can be written
// straight into HBM while the host can regenerate any slice of it.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint16_t value(uint64_t key, uint64_t i, float scale) {
  const uint64_t g = 0x9E3779B97F4A7C15ULL;
  uint64_t a = mix64(key + (2 * i + 1) * g);
  uint64_t b = mix64(key + (2 * i + 2) * g);
  int32_t s = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    s += (int32_t)((a >> (16 * k)) & 0xFFFFu);
    s += (int32_t)((b >> (16 * k)) & 0xFFFFu);
  }
  // __fmul_rn: a single correctly rounded product, never contracted.
  return bf16_rne(__fmul_rn((float)(2 * s - 524280), scale));
}

__global__ void fill_linear_kernel(uint16_t* __restrict__ out, uint64_t key, uint64_t base,
                                   int64_t n, float scale) {
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += stride)
    out[t] = value(key, base + (uint64_t)t, scale);
}

__global__ void fill_const_kernel(uint16_t* __restrict__ out, uint16_t bits, int64_t n) {
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += stride)
    out[t] = bits;
}

// cache: [batch_cap][n_heads][capacity][head_dim] for one layer; sequence b
// gets positions [0, ctx_len[b]) filled, the same numbers as sy_fill_ctx.
__global__ void fill_ctx_kernel(uint16_t* __restrict__ cache, uint64_t key,
                                const int32_t* __restrict__ ctx_len, int32_t batch,
                                int32_t n_heads, int32_t capacity, int32_t head_dim, float scale) {
  int64_t rows = (int64_t)batch * n_heads * capacity;
  int64_t total = rows * head_dim;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
    int64_t r = t / head_dim;
    int32_t j = (int32_t)(t - r * head_dim);
    int32_t p = (int32_t)(r % capacity);
    int64_t bh = r / capacity;
    int32_t h = (int32_t)(bh % n_heads);
    int32_t b = (int32_t)(bh / n_heads);
    if (p >= ctx_len[b]) continue;
    uint64_t idx = ((((uint64_t)b * (uint64_t)n_heads + (uint64_t)h) << 20) | (uint64_t)p) *
                       (uint64_t)head_dim + (uint64_t)j;
    cache[t] = value(key, idx, scale);
  }
}

int grid_for(int64_t n) {
  int64_t g = (n + 255) / 256;
  if (g > 65536) g = 65536;
  if (g < 1) g = 1;
  return (int)g;
}

}  // namespace

extern "C" {

// All launches are asynchronous on `stream`; return 0 or the hipError_t code.
int sy_dev_fill_linear(void* out, uint64_t key, uint64_t base, int64_t n, float scale,
                       hipStream_t stream) {
  if (n <= 0) return 0;
  hipLaunchKernelGGL(fill_linear_kernel, dim3(grid_for(n)), dim3(256), 0, stream,
                     (uint16_t*)out, key, base, n, scale);
  return (int)hipGetLastError();
}

int sy_dev_fill_const(void* out, uint16_t bits, int64_t n, hipStream_t stream) {
  if (n <= 0) return 0;
  hipLaunchKernelGGL(fill_const_kernel, dim3(grid_for(n)), dim3(256), 0, stream,
                     (uint16_t*)out, bits, n);
  return (int)hipGetLastError();
}

int sy_dev_fill_ctx(void* cache_layer, uint64_t key, const int32_t* ctx_len_dev, int32_t batch,
                    int32_t n_heads, int32_t capacity, int32_t head_dim, float scale,
                    hipStream_t stream) {
  int64_t total = (int64_t)batch * n_heads * capacity * head_dim;
  if (total <= 0) return 0;
  hipLaunchKernelGGL(fill_ctx_kernel, dim3(grid_for(total)), dim3(256), 0, stream,
                     (uint16_t*)cache_layer, key, ctx_len_dev, batch, n_heads, capacity, head_dim,
                     scale);
  return (int)hipGetLastError();
}

}  // extern "C"
