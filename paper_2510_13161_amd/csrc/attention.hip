// Verify attention: every block row attends to the cached context of its
// sequence and to its ancestors-or-self inside the block (chain: causal; tree:
// the hypothesis-tree mask, one 64-bit ancestor mask per row, applied in
// registers). GQA: query head h reads kv head h / (H / H_kv).
//
// Flash-decoding over 256-key chunks: a workgroup owns one (sequence, kv
// head, chunk) and each of its 4 waves one 64-key block of the chunk. A wave
// loads its block's K (as MFMA operands) and V (staged transposed in its own
// LDS) once, then serves every query tile of the kv head's group:
//   S^T[key][query] = K Q^T        MFMA 16x16x32; Q (fp32) as bf16 hi + lo;
//   block softmax statistics       one query per lane column: 2 shuffles;
//   O[query][d] = P V              P stays in registers as the MFMA operand.
// The 4 waves' (max, sum, output) are merged in LDS in wave order. A chunk
// that covers the whole sequence writes the normalised output straight into
// the output-projection's activation image; otherwise chunks publish their
// partials and the last chunk to arrive merges them in chunk order. All
// statistics in fp32; no floating-point atomics.
#include "kernels.h"

namespace msd {
namespace {

constexpr int kVtStride = 64 + 8;  // bf16 per LDS row of V^T (64 keys + pad)
constexpr int kQG = 2;             // query tiles per pass

// image write of 8 consecutive output dims [8 c8, 8 c8 + 8) of query qg
template <int HD>
__device__ __forceinline__ void write_out(const AttnArgs& a, int b, int kvh, int qg, int c8,
                                          const float (&o)[8]) {
  const int ns = a.n_slots, G = a.n_heads / a.n_kv_heads;
  const int gq = qg / ns, slot = qg - gq * ns;
  const int m = b * ns + slot, h = kvh * G + gq;
  const int col = h * HD + 8 * c8;
  const int ks = col >> 5, grp = (col >> 3) & 3;
  u32x4 hw, lw;
  split8_words(o, hw, lw);
  uint16_t* dst = a.out_img + img_offset(ks, m >> 4, a.MT, 16 * grp + (m & 15));
  *reinterpret_cast<u32x4*>(dst) = hw;
  *reinterpret_cast<u32x4*>(dst + 512) = lw;
}

template <int HD>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  constexpr int KSTEPS = HD / 32;
  constexpr int DSUB = HD / 16;
  constexpr int C8 = HD / 8;
  __shared__ __attribute__((aligned(16))) uint16_t vt_all[4][HD][kVtStride];
  __shared__ float ml_sh[4][kQG * 16][2];
  __shared__ __attribute__((aligned(16))) float o_sh[4][kQG * 16][HD + 4];
  __shared__ int s_last;

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
  uint16_t (*vt)[kVtStride] = vt_all[wave];
  const int G = a.n_heads / a.n_kv_heads;
  const int Qn = G * ns;
  const int QT = (Qn + 15) >> 4;
  const size_t row0 = ((size_t)b * a.n_kv_heads + kvh) * a.capacity;
  const uint16_t* kbase = a.k_cache + row0 * HD;
  const uint16_t* vbase = a.v_cache + row0 * HD;
  const int k0 = c * kAttnChunk + 64 * wave;
  const int key_hi = min(T, k0 + 64);  // keys [k0, key_hi) of this wave (maybe none)

  // this wave's K fragments and V^T, loaded once (rows clamped to a valid
  // key and masked afterwards, so no load waits behind a divergent branch)
  constexpr int VIT = HD / 8;    // 16-byte V chunks per lane
  constexpr int KPI = 512 / HD;  // keys per iteration
  u32x4 vraw[VIT];
#pragma unroll
  for (int it = 0; it < VIT; ++it) {
    const int key = it * KPI + lane / (HD / 8);
    const int pos = min(k0 + key, T - 1);
    vraw[it] = *reinterpret_cast<const u32x4*>(vbase + (size_t)pos * HD + (lane % (HD / 8)) * 8);
  }
  bf16x8 kf[4][KSTEPS];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int pos = min(k0 + 16 * j + r16, T - 1);
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
  __builtin_amdgcn_s_waitcnt(0xC07F);  // this wave's V^T is in LDS
  __builtin_amdgcn_wave_barrier();

  for (int qt0 = 0; qt0 < QT; qt0 += kQG) {
    bf16x8 qh[kQG][KSTEPS], ql[kQG][KSTEPS];
    uint64_t anc[kQG];
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

#pragma unroll
    for (int q = 0; q < kQG; ++q) {
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
          o[ds] = mfma16x16x32(pah, vb, o[ds]);
          o[ds] = mfma16x16x32(pal, vb, o[ds]);
        }
      }
      // publish to LDS: o D layout rows (queries) 4g + r, column (dim) 16 ds + r16
#pragma unroll
      for (int ds = 0; ds < DSUB; ++ds)
#pragma unroll
        for (int r = 0; r < 4; ++r) o_sh[wave][q * 16 + 4 * g + r][ds * 16 + r16] = o[ds][r];
      if (g == 0) {
        ml_sh[wave][q * 16 + r16][0] = mx;
        ml_sh[wave][q * 16 + r16][1] = ls;
      }
    }
    __syncthreads();
    // merge the 4 waves (wave order), then output or publish the chunk
    for (int i = tid; i < kQG * 16 * C8; i += blockDim.x) {
      const int ql = i / C8, c8 = i - ql * C8;
      const int qg = qt0 * 16 + ql;
      if (qg >= Qn) continue;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < 4; ++w) M = fmaxf(M, ml_sh[w][ql][0]);
      float S = 0.0f, o8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float mw = ml_sh[w][ql][0];
        const float f = mw == -INFINITY ? 0.0f : expf(mw - M);
        S += ml_sh[w][ql][1] * f;
        const float4 v0 = *reinterpret_cast<const float4*>(&o_sh[w][ql][8 * c8]);
        const float4 v1 = *reinterpret_cast<const float4*>(&o_sh[w][ql][8 * c8 + 4]);
        o8[0] += f * v0.x;
        o8[1] += f * v0.y;
        o8[2] += f * v0.z;
        o8[3] += f * v0.w;
        o8[4] += f * v1.x;
        o8[5] += f * v1.y;
        o8[6] += f * v1.z;
        o8[7] += f * v1.w;
      }
      if (nch == 1) {
        const float inv = S > 0.0f ? 1.0f / S : 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o8[e] *= inv;
        write_out<HD>(a, b, kvh, qg, c8, o8);
      } else {
        const size_t pidx = (((size_t)b * a.n_kv_heads + kvh) * a.max_chunks + c) * Qn + qg;
        float* po = a.part_o + pidx * HD + 8 * c8;
#pragma unroll
        for (int e = 0; e < 8; e += 2) store_coherent2(po + e, o8[e], o8[e + 1]);
        if (c8 == 0) store_coherent2(a.part_ml + 2 * pidx, M, S);
      }
    }
    __syncthreads();
  }
  if (nch == 1) return;

  // chunk hand-off: the last chunk of this (sequence, kv head) merges all
  drain_stores();
  __syncthreads();
  int32_t* ctr = a.counters + (size_t)b * a.n_kv_heads + kvh;
  if (tid == 0) s_last = counter_add(ctr, 1) == nch - 1;
  __syncthreads();
  if (!s_last) return;
  const size_t base = ((size_t)b * a.n_kv_heads + kvh) * a.max_chunks;
  for (int i = tid; i < Qn * C8; i += blockDim.x) {
    const int qg = i / C8, c8 = i - qg * C8;
    float M = -INFINITY, S = 0.0f, o8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nch; c0 += 4) {
      float pm[4], ps[4], pv[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int cc = c0 + u < nch ? c0 + u : c0;
        const size_t pidx = (base + cc) * Qn + qg;
        const float2 ml = load_coherent2(a.part_ml + 2 * pidx);
        pm[u] = ml.x;
        ps[u] = ml.y;
        const float* po = a.part_o + pidx * HD + 8 * c8;
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const float2 v = load_coherent2(po + e);
          pv[u][e] = v.x;
          pv[u][e + 1] = v.y;
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (c0 + u >= nch || pm[u] == -INFINITY) continue;
        const float Mn = fmaxf(M, pm[u]);
        const float fa = M == -INFINITY ? 0.0f : expf(M - Mn);
        const float fb = expf(pm[u] - Mn);
        S = S * fa + ps[u] * fb;
#pragma unroll
        for (int e = 0; e < 8; ++e) o8[e] = o8[e] * fa + pv[u][e] * fb;
        M = Mn;
      }
    }
    const float inv = S > 0.0f ? 1.0f / S : 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) o8[e] *= inv;
    write_out<HD>(a, b, kvh, qg, c8, o8);
  }
  if (tid == 0) counter_reset(ctr);
}

}  // namespace

hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t s) {
  if (a.max_chunks > kMaxAttnChunks || a.max_chunks < 1) return hipErrorInvalidValue;
  const dim3 grid(a.max_chunks, a.n_kv_heads, a.batch);
  if (head_dim == 128) hipLaunchKernelGGL(attn_kernel<128>, grid, dim3(256), 0, s, a);
  else if (head_dim == 64) hipLaunchKernelGGL(attn_kernel<64>, grid, dim3(256), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace msd
