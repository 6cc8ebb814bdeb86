// Verify attention: every block row attends to the cached context of its
// sequence and to its ancestors-or-self inside the block (chain: causal; tree:
// the hypothesis-tree mask, one 64-bit ancestor mask per row, applied in
// registers). GQA: query head h reads kv head h / (H / H_kv).
//
// Flash-decoding over 256-key chunks: a workgroup owns one (sequence, kv
// head, group of 16-query tiles of the head's GQA group, chunk) and each of
// its 4 waves one 64-key block. A wave loads its block's K as MFMA operands
// and V rows into its own LDS (16-byte writes, read back as P V operands with
// the gfx950 transposing LDS read) once, then for each query tile of the
// group in turn
//   S^T[key][query] = K Q^T        MFMA 16x16x32; Q as bf16 hi + lo operands
//                                  that the QKV epilogue wrote in MFMA order;
//   block softmax statistics       one query per lane column: 2 shuffles;
//   O[query][d] += P V             P stays in registers as the MFMA operand.
// Scores are kept in base-2 units (the 1/sqrt(hd) scale times log2 e), so
// every exponential is one hardware exp2.
// The 4 waves' (max, sum, output) are merged in LDS in wave order. A chunk
// that covers the whole sequence writes the normalised output straight into
// the output-projection's activation image; otherwise the chunks publish
// their partials with coherent stores and the last chunk of the (sequence,
// kv head, query tile) to arrive merges all of them in chunk order. All
// statistics in fp32; no floating-point atomics: bit-reproducible.
#include "kernels.h"

namespace msd {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

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

// the same for 4 consecutive dims [4 c4, 4 c4 + 4): half of an image lane
// (the same bf16 pairs as write_out, so the same bits)
template <int HD>
__device__ __forceinline__ void write_out4(const AttnArgs& a, int b, int kvh, int qg, int c4,
                                           const float (&o)[4]) {
  const int ns = a.n_slots, G = a.n_heads / a.n_kv_heads;
  const int gq = qg / ns, slot = qg - gq * ns;
  const int m = b * ns + slot, h = kvh * G + gq;
  const int col = h * HD + 4 * c4;
  const int ks = col >> 5, grp = (col >> 3) & 3;
  u32x2 hw, lw;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    hw[i] = pack_bf16x2(o[2 * i], o[2 * i + 1]);
    lw[i] = pack_bf16x2(o[2 * i] - bf_lo(hw[i]), o[2 * i + 1] - bf_hi(hw[i]));
  }
  uint16_t* dst = a.out_img + img_offset(ks, m >> 4, a.MT, 16 * grp + (m & 15)) + (col & 7);
  *reinterpret_cast<u32x2*>(dst) = hw;
  *reinterpret_cast<u32x2*>(dst + 512) = lw;
}

template <int HD>
struct AttnLds {
  static constexpr int kVS = HD + 4;  // bf16 per LDS row of V (one key), conflict-free strides
  static constexpr int kOS = HD + 4;  // floats per LDS row of a wave's output
  static constexpr int kVBytes = 64 * kVS * 2;
  static constexpr int kOBytes = 16 * kOS * 4;
  static constexpr int kRegion = kVBytes > kOBytes ? kVBytes : kOBytes;
};

// MULTI: the workgroup takes several query tiles in turn (K and V operands
// stay in registers across them); otherwise exactly one.
template <int HD, bool MULTI>
__global__ __launch_bounds__(256, 2) void attn_kernel(AttnArgs a) {
  using Lds = AttnLds<HD>;
  constexpr int KSTEPS = HD / 32;
  constexpr int DSUB = HD / 16;
  constexpr int C8 = HD / 8;
  constexpr int C4 = HD / 4;
  constexpr int VIT = HD / 8;    // 16-byte V chunks per lane per 64-key block
  constexpr int KPI = 512 / HD;  // keys per V chunk iteration
  __shared__ __attribute__((aligned(16))) unsigned char region_all[4][Lds::kRegion];
  __shared__ float ml_sh[4][16][2];
  __shared__ int last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int G = a.n_heads / a.n_kv_heads;
  const int ns = a.n_slots;
  const int Qn = G * ns;
  const int QT = (Qn + 15) >> 4;
  const int QG = (QT + a.q_per_wg - 1) / a.q_per_wg;  // query-tile groups per kv head
  const int b = blockIdx.z, kvh = blockIdx.y / QG, qgi = blockIdx.y - kvh * QG, c = blockIdx.x;
  const int qt0 = qgi * a.q_per_wg, qt1 = MULTI ? min(QT, qt0 + a.q_per_wg) : qt0 + 1;
  const int L = a.len[b];
  const int T = L + ns;
  if (T > a.capacity) {
    if (c == 0 && blockIdx.y == 0 && tid == 0) atomicOr(a.status, 1u);
    return;
  }
  const int nch = (T + kAttnChunk - 1) / kAttnChunk;
  if (c >= nch) return;
  uint16_t* vs = reinterpret_cast<uint16_t*>(region_all[wave]);  // [64 keys][kVS]
  float* os = reinterpret_cast<float*>(region_all[wave]);        // [16 queries][kOS]
  const size_t row0 = ((size_t)b * a.n_kv_heads + kvh) * a.capacity;
  const uint16_t* kbase = a.k_cache + row0 * HD;
  const uint16_t* vbase = a.v_cache + row0 * HD;
  const int k0 = c * kAttnChunk + 64 * wave;
  const int key_hi = min(T, k0 + 64);  // this wave's keys [k0, key_hi), maybe none

  // K fragments and V rows first (rows past the last key clamped to a valid
  // row; their scores are masked); they serve every query tile of the group
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

  // a query tile's split-bf16 operands, as the QKV epilogue wrote them,
  // straight into registers; padding queries (past G * n_slots) are zeroed by
  // selection, so whatever the workspace holds there never reaches a score
  bf16x8 qh[KSTEPS], ql[KSTEPS];
  auto load_q = [&](int qt) {
    const uint16_t* qtile =
        a.q_img + (((size_t)b * a.n_kv_heads + kvh) * QT + qt) * (size_t)KSTEPS * 1024 + lane * 8;
    const bool qok = qt * 16 + r16 < Qn;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      u32x4 h = *reinterpret_cast<const u32x4*>(qtile + (size_t)kk * 1024);
      u32x4 l = *reinterpret_cast<const u32x4*>(qtile + (size_t)kk * 1024 + 512);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        h[x] = qok ? h[x] : 0u;
        l[x] = qok ? l[x] : 0u;
      }
      qh[kk] = __builtin_bit_cast(bf16x8, h);
      ql[kk] = __builtin_bit_cast(bf16x8, l);
    }
  };
  load_q(qt0);
  // V rows into the wave's LDS as they are (16-byte writes), read back as
  // P V operands: lane l takes dim 16 ds + l%16 of keys 32 kb + 4 g + e and
  // 32 kb + 16 + 4 g + e (e < 4), the k order of P below
#pragma unroll
  for (int it = 0; it < VIT; ++it) {
    const int key = it * KPI + lane / (HD / 8);
    *reinterpret_cast<u32x4*>(vs + key * Lds::kVS + (lane % (HD / 8)) * 8) = vraw[it];
  }
  wave_lds_sync();
  // transposing LDS reads: in each 16-lane group, lane i receives element
  // i % 4 of the 8-byte chunks addressed by lanes i / 4 + 4 k (k < 4), so
  // lane s of group g points at key 32 kb + 4 g + s / 4 (+ 16), dims
  // 16 ds + 4 (s % 4) .. +4, and gets dim 16 ds + s of keys 4 g + k
  bf16x8 vb[2][DSUB];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int ds = 0; ds < DSUB; ++ds) {
      const uint16_t* p0 = vs + (32 * kb + 4 * g + (r16 >> 2)) * Lds::kVS + 16 * ds + 4 * (r16 & 3);
      const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p0);
      const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + 16 * Lds::kVS));
      vb[kb][ds] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }

  const float scale2 = a.scale * kLog2e;
  const size_t pbase = ((size_t)b * a.n_kv_heads + kvh) * a.max_chunks;
  // this (sequence, kv head)'s chunk outputs: [max_chunks][Qn][HD] floats
  const __amdgpu_buffer_rsrc_t pco =
      coherent_region(a.part_o + pbase * Qn * HD, (uint32_t)((size_t)a.max_chunks * Qn * HD * 4));
  for (int qt = qt0; qt < qt1; ++qt) {
    if (MULTI && qt != qt0) load_q(qt);
    const int qv = qt * 16 + r16;
    const uint64_t anc = qv < Qn ? a.topo.anc[qv % ns] : 0ull;
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
    // lane holds S^T[key 16j + 4g + r][query r16]: scale (base 2), mask, softmax
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int pos = k0 + 16 * j + 4 * g + r;
        const bool vis = pos < key_hi && (pos < L || ((anc >> (pos - L)) & 1ull));
        sc[j][r] = vis ? sc[j][r] * scale2 : -INFINITY;
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
        sc[j][r] = exp2_hw(sc[j][r] - mref);
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
      for (int x = 0; x < 4; ++x) {
        const float p0 = sc[2 * kb + (x >> 1)][2 * (x & 1)];
        const float p1 = sc[2 * kb + (x >> 1)][2 * (x & 1) + 1];
        ph[x] = pack_bf16x2(p0, p1);
        pl[x] = pack_bf16x2(p0 - bf_lo(ph[x]), p1 - bf_hi(ph[x]));
      }
      const bf16x8 pah = __builtin_bit_cast(bf16x8, ph);
      const bf16x8 pal = __builtin_bit_cast(bf16x8, pl);
#pragma unroll
      for (int ds = 0; ds < DSUB; ++ds) {
        o[ds] = mfma16x16x32(pah, vb[kb][ds], o[ds]);
        o[ds] = mfma16x16x32(pal, vb[kb][ds], o[ds]);
      }
    }

    // publish the wave's (max, sum, output) to its LDS region: every wave's
    // V reads, and the previous tile's merge, are done once all have passed
    // this barrier
    __syncthreads();
#pragma unroll
    for (int ds = 0; ds < DSUB; ++ds)
#pragma unroll
      for (int r = 0; r < 4; ++r) os[(4 * g + r) * Lds::kOS + ds * 16 + r16] = o[ds][r];
    if (g == 0) {
      ml_sh[wave][r16][0] = mx;
      ml_sh[wave][r16][1] = ls;
    }
    __syncthreads();
    // merge the 4 waves (wave order), then output or publish the chunk
    if (nch == 1) {
      for (int x = tid; x < 16 * C8; x += blockDim.x) {
        const int qloc = x / C8, c8 = x - qloc * C8;
        const int qg = qt * 16 + qloc;
        if (qg >= Qn) continue;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < 4; ++w) M = fmaxf(M, ml_sh[w][qloc][0]);
        float S = 0.0f, o8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float mw = ml_sh[w][qloc][0];
          const float f = mw == -INFINITY ? 0.0f : exp2_hw(mw - M);
          S += ml_sh[w][qloc][1] * f;
          const float* src = reinterpret_cast<const float*>(region_all[w]) + qloc * Lds::kOS + 8 * c8;
          const float4 v0 = *reinterpret_cast<const float4*>(src);
          const float4 v1 = *reinterpret_cast<const float4*>(src + 4);
          o8[0] += f * v0.x;
          o8[1] += f * v0.y;
          o8[2] += f * v0.z;
          o8[3] += f * v0.w;
          o8[4] += f * v1.x;
          o8[5] += f * v1.y;
          o8[6] += f * v1.z;
          o8[7] += f * v1.w;
        }
        const float inv = S > 0.0f ? 1.0f / S : 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o8[e] *= inv;
        write_out<HD>(a, b, kvh, qg, c8, o8);
      }
    } else {
      // 4 dims a thread, so that each 16-byte store of a wave covers one
      // contiguous 1 KB of the chunk's [Qn][HD] partial: whole lines
      for (int x = tid; x < 16 * C4; x += blockDim.x) {
        const int qloc = x / C4, c4 = x - qloc * C4;
        const int qg = qt * 16 + qloc;
        if (qg >= Qn) continue;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < 4; ++w) M = fmaxf(M, ml_sh[w][qloc][0]);
        float S = 0.0f;
        floatx4 o4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float mw = ml_sh[w][qloc][0];
          const float f = mw == -INFINITY ? 0.0f : exp2_hw(mw - M);
          S += ml_sh[w][qloc][1] * f;
          const float4 v0 = *reinterpret_cast<const float4*>(
              reinterpret_cast<const float*>(region_all[w]) + qloc * Lds::kOS + 4 * c4);
          o4[0] += f * v0.x;
          o4[1] += f * v0.y;
          o4[2] += f * v0.z;
          o4[3] += f * v0.w;
        }
        const size_t pidx = (pbase + c) * Qn + qg;
        store_coherent4(pco, (uint32_t)((((size_t)c * Qn + qg) * HD + 4 * c4) * 4), o4);
        if (c4 == 0) store_coherent2(a.part_ml + 2 * pidx, M, S);
      }
    }
  }
  if (nch == 1) return;

  // hand-off, once per workgroup: the last chunk of the (sequence, kv head,
  // tile group) to arrive merges every tile of the group in chunk order
  drain_stores();
  __syncthreads();
  int32_t* ctr = a.counters + ((size_t)b * a.n_kv_heads + kvh) * QG + qgi;
  if (tid == 0) last = counter_add(ctr, 1) == nch - 1;
  __syncthreads();
  if (!last) return;
  constexpr int MB = 8;  // chunk partials in flight per merge round
  for (int x = tid; x < (qt1 - qt0) * 16 * C4; x += blockDim.x) {
    const int qloc = x / C4, c4 = x - qloc * C4;
    const int qg = qt0 * 16 + qloc;
    if (qg >= Qn) continue;
    float M = -INFINITY, S = 0.0f, o4[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nch; c0 += MB) {
      float2 ml[MB];
      floatx4 v[MB];
#pragma unroll
      for (int u = 0; u < MB; ++u) {
        const int cc = c0 + u < nch ? c0 + u : c0;
        const size_t pidx = (pbase + cc) * Qn + qg;
        ml[u] = load_coherent2(a.part_ml + 2 * pidx);
        v[u] = load_coherent4(pco, (uint32_t)((((size_t)cc * Qn + qg) * HD + 4 * c4) * 4));
      }
#pragma unroll
      for (int u = 0; u < MB; ++u) {
        if (c0 + u >= nch || ml[u].x == -INFINITY) continue;
        const float Mn = fmaxf(M, ml[u].x);
        const float fa = M == -INFINITY ? 0.0f : exp2_hw(M - Mn);
        const float fb = exp2_hw(ml[u].x - Mn);
        S = S * fa + ml[u].y * fb;
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = o4[e] * fa + v[u][e] * fb;
        M = Mn;
      }
    }
    const float inv = S > 0.0f ? 1.0f / S : 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) o4[e] *= inv;
    write_out4<HD>(a, b, kvh, qg, c4, o4);
  }
  if (tid == 0) counter_reset(ctr);
}

}  // namespace

hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t s) {
  if (a.max_chunks > kMaxAttnChunks || a.max_chunks < 1) return hipErrorInvalidValue;
  if (a.max_chunks > 1 && !a.counters) return hipErrorInvalidValue;
  const int qt = (a.n_heads / a.n_kv_heads * a.n_slots + 15) / 16;
  if (a.q_per_wg < 1) return hipErrorInvalidValue;
  const dim3 grid(a.max_chunks, a.n_kv_heads * ((qt + a.q_per_wg - 1) / a.q_per_wg), a.batch);
  const bool multi = a.q_per_wg > 1 && qt > 1;
  if (head_dim == 128) {
    if (multi) hipLaunchKernelGGL((attn_kernel<128, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((attn_kernel<128, false>), grid, dim3(256), 0, s, a);
  } else if (head_dim == 64) {
    if (multi) hipLaunchKernelGGL((attn_kernel<64, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((attn_kernel<64, false>), grid, dim3(256), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace msd
