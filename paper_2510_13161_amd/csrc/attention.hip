// Verify attention: every block row attends to the cached context of its
// sequence and to its ancestors-or-self inside the block (chain: causal; tree:
// the hypothesis-tree mask, one 64-bit ancestor mask per row, applied in
// registers). GQA: query head h reads kv head h / (H / H_kv).
//
// Work split: workgroup = (256-key chunk, kv head, sequence), wave = 64 keys
// of the chunk. The queries of one kv head (G heads x n_slots rows) are taken
// in 16-wide tiles. Per wave and query tile:
//   S^T[key][query] = K Q^T        MFMA 16x16x32, K from HBM (16-byte rows),
//                                  Q (fp32) as bf16 hi + lo parts;
//   softmax over the wave's keys   the D layout puts one query per lane
//                                  column, so row statistics need 2 shuffles;
//   O[query][d] = P V              P stays in registers as the MFMA A operand
//                                  (its k order = the S^T row order), V is
//                                  staged transposed in LDS once per wave.
// Waves merge in LDS (fixed order). When a sequence's keys span several
// chunks, every chunk stores its (max, sum, unnormalised output) and a second
// kernel merges the chunks of 16 queries per workgroup, in chunk order. All
// statistics in fp32.
#include "kernels.h"

namespace msd {
namespace {

constexpr int kVtStride = 64 + 8;  // bf16 per LDS row of V^T (64 keys + pad)

template <int HD>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  constexpr int KSTEPS = HD / 32;
  constexpr int DSUB = HD / 16;
  constexpr int OSTR = HD + 4;
  __shared__ __attribute__((aligned(16))) uint16_t vt[4][HD][kVtStride];
  __shared__ float wo[4][16][OSTR];
  __shared__ float wm[4][16], wl[4][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int b = blockIdx.z, kvh = blockIdx.y, c = blockIdx.x;
  const int L = a.len[b];
  const int ns = a.n_slots;
  const int T = L + ns;
  if (T > a.capacity) {
    if (c == 0 && kvh == 0 && tid == 0) atomicOr(a.status, 1u);
    return;
  }
  const int nch = (T + kAttnChunk - 1) / kAttnChunk;
  if (c >= nch) return;
  const int G = a.n_heads / a.n_kv_heads;
  const int Qn = G * ns;
  const int QT = (Qn + 15) >> 4;
  const size_t row0 = ((size_t)b * a.n_kv_heads + kvh) * a.capacity;
  const uint16_t* kbase = a.k_cache + row0 * HD;
  const uint16_t* vbase = a.v_cache + row0 * HD;
  const int key0 = c * kAttnChunk + wave * 64;

  // V^T of this wave's 64 keys (zero beyond the last key)
  for (int i = lane; i < 64 * (HD / 8); i += 64) {
    const int key = i / (HD / 8), d0 = (i - key * (HD / 8)) * 8;
    const int pos = key0 + key;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (pos < T) v = *reinterpret_cast<const u32x4*>(vbase + (size_t)pos * HD + d0);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      vt[wave][d0 + e][key] = (uint16_t)((e & 1) ? (v[e >> 1] >> 16) : (v[e >> 1] & 0xFFFFu));
  }
  // K rows of this wave as MFMA A fragments (row = key 16*j + l%16)
  bf16x8 kf[4][KSTEPS];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int pos = key0 + 16 * j + r16;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk)
      kf[j][kk] = pos < T ? load16(kbase + (size_t)pos * HD + kk * 32 + g * 8) : zero_bf16x8();
  }
  __syncthreads();

  for (int qt = 0; qt < QT; ++qt) {
    const int qv = qt * 16 + r16;
    const bool qok = qv < Qn;
    const int gq = qok ? qv / ns : 0;
    const int slot = qok ? qv - gq * ns : 0;
    const int h = kvh * G + gq;
    const float* qp = a.q + ((size_t)(b * ns + slot) * a.n_heads + h) * HD;
    bf16x8 qh[KSTEPS], ql[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      if (qok) {
        load_split8(qp + kk * 32 + g * 8, qh[kk], ql[kk]);
      } else {
        qh[kk] = zero_bf16x8();
        ql[kk] = zero_bf16x8();
      }
    }

    // q enters as bf16 hi + lo: two MFMAs per k-step against the bf16 keys
    floatx4 sc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KSTEPS; ++kk) {
        sc[j] = mfma16x16x32(kf[j][kk], qh[kk], sc[j]);
        sc[j] = mfma16x16x32(kf[j][kk], ql[kk], sc[j]);
      }
    }
    // lane holds S^T[key 16j + 4g + r][query r16]
    const uint64_t anc = a.topo.anc[slot];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int pos = key0 + 16 * j + 4 * g + r;
        const bool vis = qok && pos < T && (pos < L || ((anc >> (pos - L)) & 1ull));
        sc[j][r] = vis ? sc[j][r] * a.scale : -INFINITY;
        mx = fmaxf(mx, sc[j][r]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mref = mx == -INFINITY ? 0.0f : mx;
    float ls = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sc[j][r] = expf(sc[j][r] - mref);
        ls += sc[j][r];
      }
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 32);

    floatx4 o[DSUB];
#pragma unroll
    for (int ds = 0; ds < DSUB; ++ds) o[ds] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      // P as bf16 hi + lo (its k order is the S^T row order: keys 4g+r of the
      // two 16-key tiles), two MFMAs against the same V^T fragment
      u32x4 ph, pl;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p0 = sc[2 * kb + (i >> 1)][2 * (i & 1)];
        const float p1 = sc[2 * kb + (i >> 1)][2 * (i & 1) + 1];
        const uint16_t h0 = f2bf(p0), h1 = f2bf(p1);
        ph[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        pl[i] = pack_bf16x2(p0 - bf2f(h0), p1 - bf2f(h1));
      }
      const bf16x8 pah = __builtin_bit_cast(bf16x8, ph);
      const bf16x8 pal = __builtin_bit_cast(bf16x8, pl);
#pragma unroll
      for (int ds = 0; ds < DSUB; ++ds) {
        const uint16_t* vrow = &vt[wave][ds * 16 + r16][32 * kb];
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow + 4 * g);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + 16 + 4 * g);
        const u32x4 vw = {lo[0], lo[1], hi[0], hi[1]};
        const bf16x8 vb = __builtin_bit_cast(bf16x8, vw);
        o[ds] = mfma16x16x32(pah, vb, o[ds]);
        o[ds] = mfma16x16x32(pal, vb, o[ds]);
      }
    }
    if (g == 0) {
      wm[wave][r16] = mx;
      wl[wave][r16] = ls;
    }
#pragma unroll
    for (int ds = 0; ds < DSUB; ++ds)
#pragma unroll
      for (int r = 0; r < 4; ++r) wo[wave][4 * g + r][ds * 16 + r16] = o[ds][r];
    __syncthreads();

    // merge the four waves (fixed order) for 16 queries x HD
    for (int i = tid; i < 16 * HD; i += blockDim.x) {
      const int qq = i / HD, d = i - qq * HD;
      const int qg = qt * 16 + qq;
      if (qg >= Qn) continue;
      float M = -INFINITY;
      for (int w = 0; w < 4; ++w) M = fmaxf(M, wm[w][qq]);
      float S = 0.0f, O = 0.0f;
      if (M != -INFINITY) {
        for (int w = 0; w < 4; ++w) {
          if (wm[w][qq] == -INFINITY) continue;
          const float f = expf(wm[w][qq] - M);
          S += wl[w][qq] * f;
          O += wo[w][qq][d] * f;
        }
      }
      const int gg = qg / ns, sl = qg - gg * ns;
      if (nch == 1) {
        a.out[(size_t)(b * ns + sl) * a.n_heads * HD + (size_t)(kvh * G + gg) * HD + d] = O / S;
      } else {
        const size_t pidx = (((size_t)b * a.n_kv_heads + kvh) * a.max_chunks + c) * Qn + qg;
        a.part_o[pidx * HD + d] = O;
        if (d == 0) {
          a.part_ml[2 * pidx] = M;
          a.part_ml[2 * pidx + 1] = S;
        }
      }
    }
    __syncthreads();
  }
}

// Merge of the chunk partials of 16 queries of one (sequence, kv head):
// w_c = exp(m_c - M) / sum_c l_c exp(m_c - M), out = sum_c w_c O_c.
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  __shared__ float wgt[kMaxAttnChunks][16];
  const int tid = threadIdx.x;
  const int b = blockIdx.z, kvh = blockIdx.y, q0 = blockIdx.x * 16;
  const int ns = a.n_slots;
  const int T = a.len[b] + ns;
  if (T > a.capacity) return;
  const int nch = (T + kAttnChunk - 1) / kAttnChunk;
  if (nch == 1) return;  // the chunk kernel wrote the output directly
  const int G = a.n_heads / a.n_kv_heads;
  const int Qn = G * ns;
  const int nq = min(16, Qn - q0);
  if (nq <= 0) return;
  const size_t base = ((size_t)b * a.n_kv_heads + kvh) * a.max_chunks;
  for (int i = tid; i < nch * 16; i += blockDim.x) {
    const int c = i >> 4, q = i & 15;
    wgt[c][q] = q < nq ? a.part_ml[2 * ((base + c) * Qn + q0 + q)] : -INFINITY;
  }
  __syncthreads();
  if (tid < 16) {
    const int q = tid;
    float M = -INFINITY;
    for (int c = 0; c < nch; ++c) M = fmaxf(M, wgt[c][q]);
    float S = 0.0f;
    for (int c = 0; c < nch; ++c) {
      const float mc = wgt[c][q];
      const float f = (q < nq && mc != -INFINITY) ? expf(mc - M) : 0.0f;
      if (q < nq) S += a.part_ml[2 * ((base + c) * Qn + q0 + q) + 1] * f;
      wgt[c][q] = f;
    }
    const float inv = S > 0.0f ? 1.0f / S : 0.0f;
    for (int c = 0; c < nch; ++c) wgt[c][q] *= inv;
  }
  __syncthreads();
  // 16 queries x HD/4 float4 outputs
  for (int i = tid; i < 16 * (HD / 4); i += blockDim.x) {
    const int q = i / (HD / 4), d4 = i - q * (HD / 4);
    if (q >= nq) continue;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int c = 0; c < nch; ++c) {
      const float f = wgt[c][q];
      const float4 v = reinterpret_cast<const float4*>(a.part_o + ((base + c) * Qn + q0 + q) * HD)[d4];
      o.x += f * v.x;
      o.y += f * v.y;
      o.z += f * v.z;
      o.w += f * v.w;
    }
    const int qg = q0 + q, gg = qg / ns, sl = qg - gg * ns;
    float* dst = a.out + (size_t)(b * ns + sl) * a.n_heads * HD + (size_t)(kvh * G + gg) * HD;
    reinterpret_cast<float4*>(dst)[d4] = o;
  }
}

}  // namespace

hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t s) {
  if (a.max_chunks > kMaxAttnChunks) return hipErrorInvalidValue;
  const dim3 grid(a.max_chunks, a.n_kv_heads, a.batch);
  const int qn = a.n_heads / a.n_kv_heads * a.n_slots;
  const dim3 mgrid((qn + 15) / 16, a.n_kv_heads, a.batch);
  if (head_dim == 128) {
    hipLaunchKernelGGL(attn_kernel<128>, grid, dim3(256), 0, s, a);
    if (a.max_chunks > 1) hipLaunchKernelGGL(attn_merge_kernel<128>, mgrid, dim3(256), 0, s, a);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL(attn_kernel<64>, grid, dim3(256), 0, s, a);
    if (a.max_chunks > 1) hipLaunchKernelGGL(attn_merge_kernel<64>, mgrid, dim3(256), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace msd
