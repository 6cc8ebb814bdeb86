// Verify attention: every block row attends to the cached context of its
// sequence and to its ancestors-or-self inside the block (chain: causal; tree:
// the hypothesis-tree mask, one 64-bit ancestor mask per row, applied in
// registers). GQA: query head h reads kv head h / (H / H_kv).
//
// Flash-decoding split: each wave owns one span of keys (a multiple of 64,
// chosen per call so that the (sequence, kv head, span) items fill the chip)
// and walks it in 64-key blocks with an online softmax held in registers:
//   S^T[key][query] = K Q^T        MFMA 16x16x32; K rows straight from HBM,
//                                  Q (fp32) as bf16 hi + lo parts;
//   row statistics                 the D layout puts one query per lane
//                                  column, so a block max needs 2 shuffles;
//   O[query][d] += P V             P stays in registers as the MFMA A operand
//                                  (its k order = the S^T row order), V is
//                                  staged transposed in the wave's own LDS.
// Waves never synchronise with each other. A span writes its (max, sum,
// unnormalised output); a second kernel merges the spans of 16 queries per
// workgroup, in span order. All statistics in fp32.
#include "kernels.h"

namespace msd {
namespace {

constexpr int kVtStride = 64 + 8;  // bf16 per LDS row of V^T (64 keys + pad)
constexpr int kQG = 2;             // query tiles held in registers at a time

template <int HD>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  constexpr int KSTEPS = HD / 32;
  constexpr int DSUB = HD / 16;
  __shared__ __attribute__((aligned(16))) uint16_t vt_all[4][HD][kVtStride];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int b = blockIdx.z, kvh = blockIdx.y;
  const int sp = blockIdx.x * 4 + wave;  // this wave's span
  const int L = a.len[b];
  const int ns = a.n_slots;
  const int T = L + ns;
  if (T > a.capacity) {
    if (sp == 0 && kvh == 0 && lane == 0) atomicOr(a.status, 1u);
    return;
  }
  const int nsp = (T + a.span - 1) / a.span;
  if (sp >= nsp) return;
  uint16_t (*vt)[kVtStride] = vt_all[wave];
  const int G = a.n_heads / a.n_kv_heads;
  const int Qn = G * ns;
  const int QT = (Qn + 15) >> 4;
  const size_t row0 = ((size_t)b * a.n_kv_heads + kvh) * a.capacity;
  const uint16_t* kbase = a.k_cache + row0 * HD;
  const uint16_t* vbase = a.v_cache + row0 * HD;
  const int key_lo = sp * a.span, key_hi = min(T, key_lo + a.span);

  for (int qt0 = 0; qt0 < QT; qt0 += kQG) {
    // queries of up to kQG tiles: fragments, mask row, running statistics.
    // Loads are unconditional (rows clamped, values masked afterwards) so
    // that none waits behind a divergent branch.
    bf16x8 qh[kQG][KSTEPS], ql[kQG][KSTEPS];
    uint64_t anc[kQG];
    float run_m[kQG], run_l[kQG];
    floatx4 o[kQG][DSUB];
    u32x4 qraw[kQG][KSTEPS][2];
    float qmask[kQG];
#pragma unroll
    for (int q = 0; q < kQG; ++q) {
      const int qv = (qt0 + q) * 16 + r16;
      const bool qok = qv < Qn;
      const int gq = qok ? qv / ns : 0;
      const int slot = qok ? qv - gq * ns : 0;
      const float* qp = a.q + ((size_t)(b * ns + slot) * a.n_heads + kvh * G + gq) * HD + g * 8;
#pragma unroll
      for (int kk = 0; kk < KSTEPS; ++kk) {
        qraw[q][kk][0] = *reinterpret_cast<const u32x4*>(qp + kk * 32);
        qraw[q][kk][1] = *reinterpret_cast<const u32x4*>(qp + kk * 32 + 4);
      }
      qmask[q] = qok ? 1.0f : 0.0f;
      anc[q] = qok ? a.topo.anc[slot] : 0ull;
      run_m[q] = -INFINITY;
      run_l[q] = 0.0f;
#pragma unroll
      for (int ds = 0; ds < DSUB; ++ds) o[q][ds] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int q = 0; q < kQG; ++q)
#pragma unroll
      for (int kk = 0; kk < KSTEPS; ++kk) {
        float v[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          v[i] = __uint_as_float(qraw[q][kk][0][i]) * qmask[q];
          v[4 + i] = __uint_as_float(qraw[q][kk][1][i]) * qmask[q];
        }
        split_vals(v, qh[q][kk], ql[q][kk]);
      }

    for (int k0 = key_lo; k0 < key_hi; k0 += 64) {
      // the block's V rows (64 keys x HD/8 chunks of 16 bytes: lane l takes
      // key it*(512/HD) + l/(HD/8), chunk l%(HD/8)) and K fragments, all
      // issued before any use; rows past the last key are clamped to a valid
      // row and zeroed
      constexpr int VIT = HD / 8;         // 16-byte V chunks per lane
      constexpr int KPI = 512 / HD;       // keys per iteration
      u32x4 vraw[VIT];
#pragma unroll
      for (int it = 0; it < VIT; ++it) {
        const int key = it * KPI + lane / (HD / 8);
        const int pos = min(k0 + key, key_hi - 1);
        vraw[it] = *reinterpret_cast<const u32x4*>(vbase + (size_t)pos * HD + (lane % (HD / 8)) * 8);
      }
      bf16x8 kf[4][KSTEPS];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int pos = min(k0 + 16 * j + r16, key_hi - 1);
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) kf[j][kk] = load16(kbase + (size_t)pos * HD + kk * 32 + g * 8);
      }
#pragma unroll
      for (int it = 0; it < VIT; ++it) {
        const int key = it * KPI + lane / (HD / 8);
        const int d0 = (lane % (HD / 8)) * 8;
        const bool live = k0 + key < key_hi;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t w = vraw[it][e >> 1];
          vt[d0 + e][key] = live ? (uint16_t)((e & 1) ? (w >> 16) : (w & 0xFFFFu)) : (uint16_t)0;
        }
      }
      // (K rows past the last key are masked out of the scores below)

#pragma unroll
      for (int q = 0; q < kQG; ++q) {
        if ((qt0 + q) * 16 >= Qn) break;
        floatx4 sc[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kk = 0; kk < KSTEPS; ++kk) {
            sc[j] = mfma16x16x32(kf[j][kk], qh[q][kk], sc[j]);
            sc[j] = mfma16x16x32(kf[j][kk], ql[q][kk], sc[j]);
          }
        }
        // lane holds S^T[key 16j + 4g + r][query r16]: scale, mask, block max
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int pos = k0 + 16 * j + 4 * g + r;
            const bool vis = pos < key_hi && (pos < L || ((anc[q] >> (pos - L)) & 1ull));
            sc[j][r] = vis ? sc[j][r] * a.scale : -INFINITY;
            mx = fmaxf(mx, sc[j][r]);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(run_m[q], mx);
        const float mref = m_new == -INFINITY ? 0.0f : m_new;
        const float alpha = run_m[q] == -INFINITY ? 0.0f : expf(run_m[q] - mref);
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
        run_l[q] = run_l[q] * alpha + ls;
        run_m[q] = m_new;
        // rescale the output rows (D layout: rows 4g + r) by their alpha
        float ar[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) ar[r] = __shfl(alpha, 4 * g + r);
#pragma unroll
        for (int ds = 0; ds < DSUB; ++ds)
#pragma unroll
          for (int r = 0; r < 4; ++r) o[q][ds][r] *= ar[r];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          // P as bf16 hi + lo (k order: keys 4g+r of the two 16-key tiles)
          u32x4 ph, pl;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float p0 = sc[2 * kb + (i >> 1)][2 * (i & 1)];
            const float p1 = sc[2 * kb + (i >> 1)][2 * (i & 1) + 1];
            ph[i] = pack_bf16x2(p0, p1);
            pl[i] = pack_bf16x2(p0 - bf_lo(ph[i]), p1 - bf_hi(ph[i]));
          }
          const bf16x8 pah = __builtin_bit_cast(bf16x8, ph);
          const bf16x8 pal = __builtin_bit_cast(bf16x8, pl);
#pragma unroll
          for (int ds = 0; ds < DSUB; ++ds) {
            const uint16_t* vrow = &vt[ds * 16 + r16][32 * kb];
            const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow + 4 * g);
            const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + 16 + 4 * g);
            const u32x4 vw = {lo[0], lo[1], hi[0], hi[1]};
            const bf16x8 vb = __builtin_bit_cast(bf16x8, vw);
            o[q][ds] = mfma16x16x32(pah, vb, o[q][ds]);
            o[q][ds] = mfma16x16x32(pal, vb, o[q][ds]);
          }
        }
      }
    }

    // publish: the whole sequence in one span -> final output, else a partial
#pragma unroll
    for (int q = 0; q < kQG; ++q) {
      const int qtile = qt0 + q;
      if (qtile * 16 >= Qn) break;
      float lr[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) lr[r] = __shfl(run_l[q], 4 * g + r);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qg = qtile * 16 + 4 * g + r;
        if (qg >= Qn) continue;
        const int gg = qg / ns, sl = qg - gg * ns;
        if (nsp == 1) {
          float* dst = a.out + (size_t)(b * ns + sl) * a.n_heads * HD + (size_t)(kvh * G + gg) * HD;
          const float inv = lr[r] > 0.0f ? 1.0f / lr[r] : 0.0f;
#pragma unroll
          for (int ds = 0; ds < DSUB; ++ds) dst[ds * 16 + r16] = o[q][ds][r] * inv;
        } else {
          const size_t pidx = (((size_t)b * a.n_kv_heads + kvh) * a.max_spans + sp) * Qn + qg;
#pragma unroll
          for (int ds = 0; ds < DSUB; ++ds) a.part_o[pidx * HD + ds * 16 + r16] = o[q][ds][r];
        }
      }
      if (nsp > 1 && g == 0) {
        const int qg = qtile * 16 + r16;
        if (qg < Qn) {
          const size_t pidx = (((size_t)b * a.n_kv_heads + kvh) * a.max_spans + sp) * Qn + qg;
          a.part_ml[2 * pidx] = run_m[q];
          a.part_ml[2 * pidx + 1] = run_l[q];
        }
      }
    }
  }
}

// Merge of the span partials of 16 queries of one (sequence, kv head):
// w_c = exp(m_c - M) / sum_c l_c exp(m_c - M), out = sum_c w_c O_c.
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  __shared__ float wgt[kMaxAttnSpans][16];
  const int tid = threadIdx.x;
  const int b = blockIdx.z, kvh = blockIdx.y, q0 = blockIdx.x * 16;
  const int ns = a.n_slots;
  const int T = a.len[b] + ns;
  if (T > a.capacity) return;
  const int nch = (T + a.span - 1) / a.span;
  if (nch == 1) return;  // the span kernel wrote the output directly
  const int G = a.n_heads / a.n_kv_heads;
  const int Qn = G * ns;
  const int nq = min(16, Qn - q0);
  if (nq <= 0) return;
  const size_t base = ((size_t)b * a.n_kv_heads + kvh) * a.max_spans;
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
  if (a.max_spans > kMaxAttnSpans || a.span % 64) return hipErrorInvalidValue;
  const dim3 grid((a.max_spans + 3) / 4, a.n_kv_heads, a.batch);
  const int qn = a.n_heads / a.n_kv_heads * a.n_slots;
  const dim3 mgrid((qn + 15) / 16, a.n_kv_heads, a.batch);
  if (head_dim == 128) {
    hipLaunchKernelGGL(attn_kernel<128>, grid, dim3(256), 0, s, a);
    if (a.max_spans > 1) hipLaunchKernelGGL(attn_merge_kernel<128>, mgrid, dim3(256), 0, s, a);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL(attn_kernel<64>, grid, dim3(256), 0, s, a);
    if (a.max_spans > 1) hipLaunchKernelGGL(attn_merge_kernel<64>, mgrid, dim3(256), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace msd
