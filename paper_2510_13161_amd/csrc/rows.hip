// Row-wise kernels of the verification pass: the block rows (embedding gather
// or a given residual) as residual, 64-column statistics and activation
// image; the per-row merge of the LM-head tiles (top-kappa, argmax,
// logsumexp).
#include "kernels.h"

namespace msd {
namespace {

// Zero the image lanes of padding row m (K columns).
__device__ void zero_image_row(uint16_t* img, int K, int m, int MT) {
  const int mt = m >> 4, r16 = m & 15;
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (int i = threadIdx.x; i < (K >> 5) * 4; i += blockDim.x) {
    const int ks = i >> 2, g = i & 3;
    uint16_t* dst = img + img_offset(ks, mt, MT, 16 * g + r16);
    *reinterpret_cast<u32x4*>(dst) = z;
    *reinterpret_cast<u32x4*>(dst + 512) = z;
  }
}

// One workgroup per row (16 MT of them; rows past M only clear their image
// lanes). Thread tt owns columns [64 tt, 64 tt + 64) of the row: it gathers
// them (embedding row, plus the learned position row, or a given fp32 hidden
// row), stores the fp32 residual, the (mean, M2) of its 64 values (two
// passes in registers) and its two image k-steps (values times the gain of
// the next pre-norm, split into bf16 hi + lo).
__global__ __launch_bounds__(256) void rows_kernel(RowsArgs a) {
  const int m = blockIdx.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.n_zero;
       i += (int64_t)gridDim.x * blockDim.x)
    a.zero_i32[i] = 0;
  if (m >= a.M) {
    if (a.img.img) zero_image_row(a.img.img, a.d, m, a.MT);
    if (a.zero_img) zero_image_row(a.zero_img, a.zero_img_k, m, a.MT);
    return;
  }
  const int tt = threadIdx.x;
  if (tt >= (a.d >> 6)) return;
  float v[64];
  if (a.hidden) {
    const float4* src = reinterpret_cast<const float4*>(a.hidden + (size_t)m * a.d + 64 * tt);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float4 f = src[i];
      v[4 * i] = f.x;
      v[4 * i + 1] = f.y;
      v[4 * i + 2] = f.z;
      v[4 * i + 3] = f.w;
    }
  } else {
    int tok = a.tokens[m];
    if (tok < 0 || tok >= a.vocab) {
      if (tt == 0) atomicOr(a.status, 4u);
      tok = 0;
    }
    const uint16_t* p = nullptr;
    if (a.pos_embed) {
      const int b = m / a.n_slots, slot = m - b * a.n_slots;
      int pos = a.len[b] + a.depth[slot];
      if (pos >= a.max_positions) pos = a.max_positions - 1;  // flagged by the cache check
      p = a.pos_embed + (size_t)pos * a.d;
    }
    u32x4 w[8], pw[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int col = 64 * tt + 8 * c;
      if (a.embed_frag) {
        // row tok of a k-step-major fragment table (vocab / 16 groups per
        // k-step): 8 consecutive columns per 16 bytes
        const size_t ng = (size_t)(a.vocab >> 4);
        const int ks = col >> 5, lane = (tok & 15) + 16 * ((col >> 3) & 3);
        w[c] = *reinterpret_cast<const u32x4*>(a.embed + ((size_t)ks * ng + (size_t)(tok >> 4)) * 512 +
                                               lane * 8);
      } else {
        w[c] = *reinterpret_cast<const u32x4*>(a.embed + (size_t)tok * a.d + col);
      }
      pw[c] = p ? *reinterpret_cast<const u32x4*>(p + col) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[8 * c + 2 * i] = bf_lo(w[c][i]) + bf_lo(pw[c][i]);
        v[8 * c + 2 * i + 1] = bf_hi(w[c][i]) + bf_hi(pw[c][i]);
      }
  }
  if (a.x) {
    float4* dst = reinterpret_cast<float4*>(a.x + (size_t)m * a.d + 64 * tt);
#pragma unroll
    for (int i = 0; i < 16; ++i) dst[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
  }
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < 64; ++i) sum += v[i];
  const float mean = sum * (1.0f / 64.0f);
  float m2 = 0.0f;
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const float dv = v[i] - mean;
    m2 += dv * dv;
  }
  a.stats[(size_t)tt * a.M + m] = make_float2(mean, m2);
  if (a.img.img) {
    const int mt = m >> 4, r16 = m & 15;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float e8[8];
        const int c0 = 32 * h + 8 * g;
        u32x4 gw = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};  // bf16 ones
        if (a.img.gain) gw = *reinterpret_cast<const u32x4*>(a.img.gain + 64 * tt + c0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          e8[2 * i] = v[c0 + 2 * i] * bf_lo(gw[i]);
          e8[2 * i + 1] = v[c0 + 2 * i + 1] * bf_hi(gw[i]);
        }
        u32x4 hw, lw;
        split8_words(e8, hw, lw);
        uint16_t* dst = a.img.img + img_offset(2 * tt + h, mt, a.MT, 16 * g + r16);
        *reinterpret_cast<u32x4*>(dst) = hw;
        *reinterpret_cast<u32x4*>(dst + 512) = lw;
      }
  }
}

// (max, sum exp) pair merge: the pair describes sum_i exp(v_i) = s * exp(m).
__device__ __forceinline__ float2 ms_merge(float2 a, float2 b) {
  if (b.x == -INFINITY) return a;
  if (a.x == -INFINITY) return b;
  if (a.x >= b.x) return make_float2(a.x, a.y + b.y * expf(b.x - a.x));
  return make_float2(b.x, b.y + a.y * expf(a.x - b.x));
}

// kappa best keys of a wave: every lane holds a descending list v[0..KB);
// kappa rounds of shuffle argmax over the list heads (keys are unique). The
// result is the same in every lane.
template <int KB>
__device__ __forceinline__ void wave_topk(uint64_t (&v)[KB], int K, uint64_t (&out)[KB]) {
#pragma unroll
  for (int r = 0; r < KB; ++r) {
    out[r] = 0ull;
    if (r >= K) continue;
    const uint64_t best = wave_max_u64(v[0]);
    const bool pop = v[0] == best && best != 0ull;
#pragma unroll
    for (int x = 0; x < KB - 1; ++x) v[x] = pop ? v[x + 1] : v[x];
    if (pop) v[KB - 1] = 0ull;
    out[r] = best;
  }
}

// (max, sum) pairs of a wave, combined in a fixed butterfly order.
__device__ __forceinline__ float2 wave_ms(float2 acc) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float2 other;
    other.x = __shfl_xor(acc.x, o);
    other.y = __shfl_xor(acc.y, o);
    acc = (lane & o) ? ms_merge(other, acc) : ms_merge(acc, other);
  }
  return acc;
}

// Stage 1 of the per-row merge of the LM-head tiles: workgroup (row m,
// part p) takes 256 consecutive tiles, one per thread; each wave extracts
// its kappa best, wave 0 merges the 4 wave lists the same way and writes the
// part's (max, sum exp) and kappa best keys.
template <int KB>
__global__ __launch_bounds__(256) void head_part_kernel(HeadMergeArgs a) {
  __shared__ float2 sh_ms[4];
  __shared__ uint64_t sh_top[4][KB];
  const int m = blockIdx.x, p = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = a.kappa;
  const int t = p * 256 + tid;
  const bool live = t < a.n_tiles;
  const int tc = live ? t : 0;
  float2 acc = a.tile_ms[(size_t)tc * a.M + m];
  uint64_t v[KB];
  const uint64_t* top = a.tile_top + ((size_t)tc * a.M + m) * K;
#pragma unroll
  for (int r = 0; r < KB; ++r) v[r] = top[r < K ? r : 0];
#pragma unroll
  for (int r = 0; r < KB; ++r) v[r] = (live && r < K) ? v[r] : 0ull;
  if (!live) acc = make_float2(-INFINITY, 0.0f);
  acc = wave_ms(acc);
  uint64_t w[KB];
  wave_topk<KB>(v, K, w);
  if (lane == 0) {
    sh_ms[wave] = acc;
#pragma unroll
    for (int r = 0; r < KB; ++r) sh_top[wave][r] = w[r];
  }
  __syncthreads();
  if (wave != 0) return;
  // lanes 0..3 hold the four wave lists
#pragma unroll
  for (int r = 0; r < KB; ++r) v[r] = lane < 4 ? sh_top[lane][r] : 0ull;
  wave_topk<KB>(v, K, w);
  if (lane == 0) {
    float2 tot = sh_ms[0];
    for (int x = 1; x < 4; ++x) tot = ms_merge(tot, sh_ms[x]);
    const size_t q = (size_t)m * gridDim.y + p;
    a.part_ms[q] = tot;
#pragma unroll
    for (int r = 0; r < KB; ++r)
      if (r < K) a.part_top[q * K + r] = w[r];
  }
}

// Stage 2: one wave per row merges the parts' lists (lane = part) and
// (max, sum) pairs (in part order), and writes ids, log-probabilities,
// argmax and logsumexp.
template <int KB>
__global__ __launch_bounds__(64) void head_final_kernel(HeadMergeArgs a, int parts) {
  const int m = blockIdx.x, lane = threadIdx.x;
  const int K = a.kappa;
  const bool live = lane < parts;
  const size_t q = (size_t)m * parts + (live ? lane : 0);
  uint64_t v[KB];
#pragma unroll
  for (int r = 0; r < KB; ++r) v[r] = (live && r < K) ? a.part_top[q * K + (r < K ? r : 0)] : 0ull;
  uint64_t w[KB];
  wave_topk<KB>(v, K, w);
  if (lane != 0) return;
  float2 tot = a.part_ms[(size_t)m * parts];
  for (int x = 1; x < parts; ++x) tot = ms_merge(tot, a.part_ms[(size_t)m * parts + x]);
  const float lse = tot.x + logf(tot.y);
#pragma unroll
  for (int r = 0; r < KB; ++r) {
    const uint64_t k = w[r];
    const int id = k ? key_id(k) : -1;
    const float val = k ? key_val(k) : -INFINITY;
    if (r < K && a.ids) a.ids[(size_t)m * K + r] = id;
    if (r < K && a.logp) a.logp[(size_t)m * K + r] = val - lse;
    if (r == 0 && a.argmax) a.argmax[m] = id;
  }
  if (a.lse) a.lse[m] = lse;
}

}  // namespace

hipError_t launch_rows(const RowsArgs& a, hipStream_t s) {
  if (a.d % 64 || a.d > 64 * 256 || a.M < 1 || a.M > 16 * a.MT) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rows_kernel, dim3(16 * a.MT), dim3(256), 0, s, a);
  return hipGetLastError();
}

int head_parts(int n_tiles) { return (n_tiles + 255) / 256; }

hipError_t launch_head_merge(const HeadMergeArgs& a, hipStream_t s) {
  if (a.kappa < 1 || a.kappa > kMaxKappa) return hipErrorInvalidValue;
  const int parts = head_parts(a.n_tiles);
  if (parts > 64 || !a.part_ms || !a.part_top) return hipErrorInvalidValue;
  const dim3 g1(a.M, parts);
  if (a.kappa <= 1) {
    hipLaunchKernelGGL(head_part_kernel<1>, g1, dim3(256), 0, s, a);
    hipLaunchKernelGGL(head_final_kernel<1>, dim3(a.M), dim3(64), 0, s, a, parts);
  } else if (a.kappa <= 8) {
    hipLaunchKernelGGL(head_part_kernel<8>, g1, dim3(256), 0, s, a);
    hipLaunchKernelGGL(head_final_kernel<8>, dim3(a.M), dim3(64), 0, s, a, parts);
  } else {
    hipLaunchKernelGGL(head_part_kernel<32>, g1, dim3(256), 0, s, a);
    hipLaunchKernelGGL(head_final_kernel<32>, dim3(a.M), dim3(64), 0, s, a, parts);
  }
  return hipGetLastError();
}

}  // namespace msd
