// Row-wise kernels of the verification pass: embedding gather (with the row
// statistics the first pre-norm needs) and the per-row merge of the LM-head
// tiles (top-kappa, argmax, logsumexp).
#include "kernels.h"

namespace msd {
namespace {

// Fixed-order block sum (256 threads): butterfly inside each wave, then the
// four wave sums in wave order. Same result for the same inputs, always.
__device__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  float r = 0.0f;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) r += sh[w];
  return r;
}

// (mean, M2) of one row, two passes, fixed-order block sums.
__device__ void row_stats(const float* x, int d, float2* out, float* sh) {
  float s = 0.0f;
  for (int k = threadIdx.x; k < d; k += blockDim.x) s += x[k];
  const float mean = block_sum(s, sh) / (float)d;
  float v = 0.0f;
  for (int k = threadIdx.x; k < d; k += blockDim.x) {
    const float c = x[k] - mean;
    v += c * c;
  }
  const float m2 = block_sum(v, sh);
  if (threadIdx.x == 0) *out = make_float2(mean, m2);
}

__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  __shared__ float sh[8];
  const int m = blockIdx.x;
  // clear the split-K / merge counters of this pass
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.n_zero;
       i += (int64_t)gridDim.x * blockDim.x)
    a.zero_i32[i] = 0;
  int tok = a.tokens[m];
  if (tok < 0 || tok >= a.vocab) {
    if (threadIdx.x == 0) atomicOr(a.status, 4u);
    tok = 0;
  }
  const uint16_t* e = a.embed + (size_t)tok * a.d;
  const uint16_t* p = nullptr;
  if (a.pos_embed) {
    const int b = m / a.n_slots, slot = m - b * a.n_slots;
    int pos = a.len[b] + a.depth[slot];
    if (pos >= a.max_positions) pos = a.max_positions - 1;  // flagged by the cache check
    p = a.pos_embed + (size_t)pos * a.d;
  }
  float* x = a.x + (size_t)m * a.d;
  if (a.embed_frag) {
    // row tok of a fragment-major table: 8 consecutive columns per 16 bytes
    const size_t run = (size_t)(a.d >> 5) * 512;
    const uint16_t* grp = a.embed + (size_t)(tok >> 4) * run;
    for (int q = threadIdx.x; q < (a.d >> 3); q += blockDim.x) {
      const int ks = q >> 2, lane = (tok & 15) + 16 * (q & 3);
      const u32x4 w = *reinterpret_cast<const u32x4*>(grp + (size_t)ks * 512 + lane * 8);
      u32x4 pw = {0u, 0u, 0u, 0u};
      if (p) pw = *reinterpret_cast<const u32x4*>(p + q * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k = q * 8 + 2 * i;
        x[k] = bf_lo(w[i]) + bf_lo(pw[i]);
        x[k + 1] = bf_hi(w[i]) + bf_hi(pw[i]);
      }
    }
  } else {
    for (int q = threadIdx.x; q < (a.d >> 3); q += blockDim.x) {
      const u32x4 w = *reinterpret_cast<const u32x4*>(e + q * 8);
      u32x4 pw = {0u, 0u, 0u, 0u};
      if (p) pw = *reinterpret_cast<const u32x4*>(p + q * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[q * 8 + 2 * i] = bf_lo(w[i]) + bf_lo(pw[i]);
        x[q * 8 + 2 * i + 1] = bf_hi(w[i]) + bf_hi(pw[i]);
      }
    }
  }
  __syncthreads();
  row_stats(x, a.d, a.stats + m, sh);
}

__global__ __launch_bounds__(256) void row_stats_kernel(const float* x, int d, float2* stats) {
  __shared__ float sh[8];
  row_stats(x + (size_t)blockIdx.x * d, d, stats + blockIdx.x, sh);
}

// (max, sum exp) pair merge: the pair describes sum_i exp(v_i) = s * exp(m).
__device__ __forceinline__ float2 ms_merge(float2 a, float2 b) {
  if (b.x == -INFINITY) return a;
  if (a.x == -INFINITY) return b;
  if (a.x >= b.x) return make_float2(a.x, a.y + b.y * expf(b.x - a.x));
  return make_float2(b.x, b.y + a.y * expf(a.x - b.x));
}

// One workgroup per row: merge the per-tile (max, sum exp) pairs and top-kappa
// lists produced by the LM-head GEMM epilogue. KB bounds kappa at compile
// time so a tile's keys load together; tiles go four at a time.
template <int KB>
__global__ __launch_bounds__(256) void head_merge_kernel(HeadMergeArgs a) {
  extern __shared__ uint64_t lists[];  // [256][kappa]
  __shared__ float2 sh_ms[4];
  __shared__ uint64_t sh_key[4];
  const int m = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = a.kappa;
  uint64_t* mine = lists + (size_t)tid * K;
  for (int r = 0; r < K; ++r) mine[r] = 0ull;

  float2 acc = make_float2(-INFINITY, 0.0f);
  for (int t0 = tid; t0 < a.n_tiles; t0 += 4 * blockDim.x) {
    float2 ms[4];
    uint64_t keys[4][KB];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = t0 + u * blockDim.x;
      const int tc = t < a.n_tiles ? t : 0;
      ms[u] = a.tile_ms[(size_t)tc * a.M + m];
      const uint64_t* top = a.tile_top + ((size_t)tc * a.M + m) * K;
#pragma unroll
      for (int r = 0; r < KB; ++r) keys[u][r] = top[r < K ? r : 0];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (t0 + u * blockDim.x >= a.n_tiles) break;
      acc = ms_merge(acc, ms[u]);
#pragma unroll
      for (int r = 0; r < KB; ++r) {
        if (r >= K) break;
        const uint64_t key = keys[u][r];
        if (key <= mine[K - 1]) break;  // tile lists are sorted, descending
        int j = K - 1;
        while (j > 0 && mine[j - 1] < key) {
          mine[j] = mine[j - 1];
          --j;
        }
        mine[j] = key;
      }
    }
  }
  // fixed-order reduction of the (max, sum) pairs
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float2 other;
    other.x = __shfl_xor(acc.x, o);
    other.y = __shfl_xor(acc.y, o);
    acc = (lane & o) ? ms_merge(other, acc) : ms_merge(acc, other);
  }
  if (lane == 0) sh_ms[wave] = acc;
  __syncthreads();
  float2 tot = sh_ms[0];
  for (int w = 1; w < 4; ++w) tot = ms_merge(tot, sh_ms[w]);
  const float lse = tot.x + logf(tot.y);

  // kappa rounds of block-wide argmax over the heads of the per-thread lists
  int head = 0;
  for (int r = 0; r < K; ++r) {
    const uint64_t cand = head < K ? mine[head] : 0ull;
    const uint64_t wbest = wave_max_u64(cand);
    if (lane == 0) sh_key[wave] = wbest;
    __syncthreads();
    uint64_t best = sh_key[0];
    for (int w = 1; w < 4; ++w) best = sh_key[w] > best ? sh_key[w] : best;
    __syncthreads();
    if (cand == best && best != 0ull) ++head;
    if (tid == 0) {
      const int id = best ? key_id(best) : -1;
      const float v = best ? key_val(best) : -INFINITY;
      if (a.ids) a.ids[(size_t)m * K + r] = id;
      if (a.logp) a.logp[(size_t)m * K + r] = v - lse;
      if (r == 0 && a.argmax) a.argmax[m] = id;
    }
  }
  if (tid == 0 && a.lse) a.lse[m] = lse;
}

__global__ void zero_kernel(int32_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

}  // namespace

hipError_t launch_zero_i32(int32_t* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t g = (n + 255) / 256;
  if (g > 1024) g = 1024;
  hipLaunchKernelGGL(zero_kernel, dim3((int)g), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(embed_kernel, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_row_stats(const float* x, int M, int d, float2* stats, hipStream_t s) {
  hipLaunchKernelGGL(row_stats_kernel, dim3(M), dim3(256), 0, s, x, d, stats);
  return hipGetLastError();
}

hipError_t launch_head_merge(const HeadMergeArgs& a, hipStream_t s) {
  const size_t shmem = (size_t)256 * a.kappa * sizeof(uint64_t);
  if (a.kappa <= 1) hipLaunchKernelGGL(head_merge_kernel<1>, dim3(a.M), dim3(256), shmem, s, a);
  else if (a.kappa <= 8) hipLaunchKernelGGL(head_merge_kernel<8>, dim3(a.M), dim3(256), shmem, s, a);
  else hipLaunchKernelGGL(head_merge_kernel<32>, dim3(a.M), dim3(256), shmem, s, a);
  return hipGetLastError();
}

}  // namespace msd
