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
//
// Long contexts (grids of one-span chunks larger than the chip holds at
// once): attn_stream_kernel, where a workgroup walks several 256-key spans
// with an online softmax and streams its next block while it computes; the
// merges above run once per chunk of spans.
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

// Publish a wave's (max, sum, output) of one query tile to its LDS region: o[ds][r]
// holds query 4 g + r, dim 16 ds + lane % 16; the statistics are replicated
// over g. The first barrier orders the region's earlier use (V rows, the
// previous tile's merge) before the writes.
template <int HD>
__device__ __forceinline__ void publish_tile(unsigned char (*region_all)[AttnLds<HD>::kRegion],
                                             float (*ml_sh)[16][2], const floatx4* o, float mx, float ls) {
  using Lds = AttnLds<HD>;
  constexpr int DSUB = HD / 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  float* os = reinterpret_cast<float*>(region_all[wave]);
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
}

// Merge the 4 published waves of query tile qt in wave order; a chunk that
// covers the whole sequence writes the normalised output into the image,
// any other publishes its partial (4 dims a thread, so that each 16-byte
// store of a wave covers one contiguous 1 KB of the chunk's [Qn][HD]
// partial: whole lines).
template <int HD>
__device__ __forceinline__ void merge_waves(const AttnArgs& a, unsigned char (*region_all)[AttnLds<HD>::kRegion],
                                            float (*ml_sh)[16][2], int b, int kvh, int qt, int Qn, int nch,
                                            int c, size_t pbase, __amdgpu_buffer_rsrc_t pco) {
  using Lds = AttnLds<HD>;
  constexpr int C8 = HD / 8;
  constexpr int C4 = HD / 4;
  const int tid = threadIdx.x;
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

// The chunk hand-off, once per workgroup after its partials are stored: the
// last chunk of the (sequence, kv head, tile group) to arrive merges tiles
// [qt0, qt1) over all nch chunks in chunk order and writes the normalised
// output; it leaves the counter zero.
template <int HD>
__device__ __forceinline__ void merge_chunks(const AttnArgs& a, int* last, int32_t* ctr, int b, int kvh,
                                             int qt0, int qt1, int Qn, int nch, size_t pbase,
                                             __amdgpu_buffer_rsrc_t pco) {
  constexpr int C4 = HD / 4;
  const int tid = threadIdx.x;
  drain_stores();
  __syncthreads();
  if (tid == 0) *last = counter_add(ctr, 1) == nch - 1;
  __syncthreads();
  if (!*last) return;
  constexpr int MB = 8;  // chunk partials in flight per item and merge round
  constexpr int IT = 2;  // items of a thread whose loads are in flight together
  const int n_items = (qt1 - qt0) * 16 * C4;
  for (int x0 = tid; x0 < n_items; x0 += IT * blockDim.x) {
    int qg[IT], c4[IT];
    bool ok[IT];
    float M[IT], S[IT], o4[IT][4];
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const int x = x0 + i * blockDim.x;
      const int qloc = x / C4;
      c4[i] = x - qloc * C4;
      qg[i] = qt0 * 16 + qloc;
      ok[i] = x < n_items && qg[i] < Qn;
      if (!ok[i]) qg[i] = 0, c4[i] = 0;  // loads stay in bounds; results unused
      M[i] = -INFINITY;
      S[i] = 0.0f;
#pragma unroll
      for (int e = 0; e < 4; ++e) o4[i][e] = 0.0f;
    }
    for (int c0 = 0; c0 < nch; c0 += MB) {
      float2 ml[IT][MB];
      floatx4 v[IT][MB];
#pragma unroll
      for (int i = 0; i < IT; ++i)
#pragma unroll
        for (int u = 0; u < MB; ++u) {
          const int cc = c0 + u < nch ? c0 + u : c0;
          const size_t pidx = (pbase + cc) * Qn + qg[i];
          ml[i][u] = load_coherent2(a.part_ml + 2 * pidx);
          v[i][u] = load_coherent4(pco, (uint32_t)((((size_t)cc * Qn + qg[i]) * HD + 4 * c4[i]) * 4));
        }
#pragma unroll
      for (int i = 0; i < IT; ++i)
#pragma unroll
        for (int u = 0; u < MB; ++u) {
          if (c0 + u >= nch || ml[i][u].x == -INFINITY) continue;
          const float Mn = fmaxf(M[i], ml[i][u].x);
          const float fa = M[i] == -INFINITY ? 0.0f : exp2_hw(M[i] - Mn);
          const float fb = exp2_hw(ml[i][u].x - Mn);
          S[i] = S[i] * fa + ml[i][u].y * fb;
#pragma unroll
          for (int e = 0; e < 4; ++e) o4[i][e] = o4[i][e] * fa + v[i][u][e] * fb;
          M[i] = Mn;
        }
    }
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      if (!ok[i]) continue;
      const float inv = S[i] > 0.0f ? 1.0f / S[i] : 0.0f;
      float out[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) out[e] = o4[i][e] * inv;
      write_out4<HD>(a, b, kvh, qg[i], c4[i], out);
    }
  }
  if (tid == 0) counter_reset(ctr);
}

// Workgroup coordinates from a one-dimensional grid ordered kv head first:
// the hardware hands consecutive workgroups to the 8 XCDs in turn, so with
// a kv-head count that is a multiple of 8 every workgroup of one kv head
// (its chunks, query-tile groups and sequences) runs on the same XCD and its
// repeated reads of that head's K and V are served by one L2.
struct AttnWg {
  int b, kvh, qgi, c;
};
__device__ __forceinline__ AttnWg attn_wg(const AttnArgs& a, int chunks, int QG) {
  int id = blockIdx.x;
  AttnWg w;
  w.kvh = id % a.n_kv_heads;
  id /= a.n_kv_heads;
  w.c = id % chunks;
  id /= chunks;
  w.qgi = id % QG;
  w.b = id / QG;
  return w;
}

// MULTI: the workgroup takes several query tiles in turn (K and V operands
// stay in registers across them); otherwise exactly one.
template <int HD, bool MULTI>
__global__ __launch_bounds__(256, 2) void attn_kernel(AttnArgs a) {
  using Lds = AttnLds<HD>;
  constexpr int KSTEPS = HD / 32;
  constexpr int DSUB = HD / 16;
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
  const AttnWg wg = attn_wg(a, a.max_chunks, QG);
  const int b = wg.b, kvh = wg.kvh, qgi = wg.qgi, c = wg.c;
  const int qt0 = qgi * a.q_per_wg, qt1 = MULTI ? min(QT, qt0 + a.q_per_wg) : qt0 + 1;
  const int L = a.len[b];
  const int T = L + ns;
  if (T > a.capacity) {
    if (c == 0 && kvh == 0 && qgi == 0 && tid == 0) atomicOr(a.status, 1u);
    return;
  }
  const int nch = (T + kAttnChunk - 1) / kAttnChunk;
  if (c >= nch) return;
  uint16_t* vs = reinterpret_cast<uint16_t*>(region_all[wave]);  // [64 keys][kVS]
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
    // lane holds S^T[key 16j + 4g + r][query r16]: scale (base 2), mask (a
    // block wholly inside the cached context is visible to every query: a
    // branch the whole wave takes; otherwise without branches), softmax
    float mx = -INFINITY;
    if (k0 + 64 <= L) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          sc[j][r] *= scale2;
          mx = fmaxf(mx, sc[j][r]);
        }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pos = k0 + 16 * j + 4 * g + r;
          const bool anc_bit = (anc >> ((pos - L) & 63)) & 1ull;
          const bool vis = (pos < key_hi) & ((pos < L) | anc_bit);
          sc[j][r] = vis ? sc[j][r] * scale2 : -INFINITY;
          mx = fmaxf(mx, sc[j][r]);
        }
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

    // every wave's V reads, and the previous tile's merge, are done once all
    // have passed publish_tile's first barrier
    publish_tile<HD>(region_all, ml_sh, o, mx, ls);
    merge_waves<HD>(a, region_all, ml_sh, b, kvh, qt, Qn, nch, c, pbase, pco);
  }
  if (nch == 1 || a.defer) return;
  merge_chunks<HD>(a, &last, a.counters + ((size_t)b * a.n_kv_heads + kvh) * QG + qgi, b, kvh, qt0, qt1, Qn,
                   nch, pbase, pco);
}

// Long contexts: a workgroup owns a chunk of nb consecutive 256-key spans and
// takes them in turn, each wave its 64-key block of every span. Per query tile
// of the group a wave keeps a running (max, sum, output), rescaled at each
// block (the online softmax), and it issues the loads of its next block
// before the arithmetic of the current one, so that its K and V stream while
// it computes. The group's query tiles sit in LDS, shared by the 4 waves.
// The 4-wave merge, the chunk hand-off and the final merge are those of the
// kernel above, once per chunk of nb spans instead of once per span.
template <int HD, int QPW>
__global__ __launch_bounds__(256, 1) void attn_stream_kernel(AttnArgs a) {
  using Lds = AttnLds<HD>;
  constexpr int KSTEPS = HD / 32;
  constexpr int DSUB = HD / 16;
  constexpr int VIT = HD / 8;
  constexpr int KPI = 512 / HD;
  __shared__ __attribute__((aligned(16))) unsigned char region_all[4][Lds::kRegion];
  __shared__ __attribute__((aligned(16))) uint16_t q_sh[QPW * KSTEPS * 1024];
  __shared__ float ml_sh[4][16][2];
  __shared__ int last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int G = a.n_heads / a.n_kv_heads;
  const int ns = a.n_slots;
  const int Qn = G * ns;
  const int QT = (Qn + 15) >> 4;
  const int QG = (QT + QPW - 1) / QPW;
  const AttnWg wg = attn_wg(a, (a.max_chunks + a.nb - 1) / a.nb, QG);
  const int b = wg.b, kvh = wg.kvh, qgi = wg.qgi, c = wg.c;
  const int qt0 = qgi * QPW, ntile = min(QPW, QT - qt0);
  const int L = a.len[b];
  const int T = L + ns;
  if (T > a.capacity) {
    if (c == 0 && kvh == 0 && qgi == 0 && tid == 0) atomicOr(a.status, 1u);
    return;
  }
  const int nch = (T + a.nb * kAttnChunk - 1) / (a.nb * kAttnChunk);
  if (c >= nch) return;
  const int sp0 = c * a.nb;                                              // first 256-key span
  const int nsp = min(a.nb, (T + kAttnChunk - 1) / kAttnChunk - sp0);  // spans with keys, >= 1
  uint16_t* vs = reinterpret_cast<uint16_t*>(region_all[wave]);  // [64 keys][kVS]
  const size_t row0 = ((size_t)b * a.n_kv_heads + kvh) * a.capacity;
  const uint16_t* kbase = a.k_cache + row0 * HD;
  const uint16_t* vbase = a.v_cache + row0 * HD;

  // one 64-key block: V rows and K fragments (rows past the last key clamped
  // to a valid row; their scores are masked)
  u32x4 vraw[VIT];
  bf16x8 kf[4][KSTEPS];
  auto load_block = [&](int k0) {
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int pos = min(k0 + it * KPI + lane / (HD / 8), T - 1);
      vraw[it] = *reinterpret_cast<const u32x4*>(vbase + (size_t)pos * HD + (lane % (HD / 8)) * 8);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int pos = min(k0 + 16 * j + r16, T - 1);
#pragma unroll
      for (int kk = 0; kk < KSTEPS; ++kk) kf[j][kk] = load16(kbase + (size_t)pos * HD + kk * 32 + g * 8);
    }
  };
  load_block(sp0 * kAttnChunk + 64 * wave);
  {
    // the group's query tiles (the QKV epilogue's split-bf16 operand image,
    // tiles of one kv head contiguous) into LDS
    const u32x4* src = reinterpret_cast<const u32x4*>(
        a.q_img + (((size_t)b * a.n_kv_heads + kvh) * QT + qt0) * (size_t)KSTEPS * 1024);
    u32x4* dst = reinterpret_cast<u32x4*>(q_sh);
    // 16-byte piece i is lane (i % 64) of a 512-element part: query row
    // (i % 16) of its tile; padding queries (past G * n_slots) and tiles past
    // the group's last are zero, so whatever the workspace holds there never
    // reaches a score
    for (int i = tid; i < QPW * KSTEPS * 128; i += blockDim.x) {
      const int t = i / (KSTEPS * 128);
      const bool ok = t < ntile && (qt0 + t) * 16 + (i & 15) < Qn;
      dst[i] = ok ? src[i] : u32x4{0u, 0u, 0u, 0u};
    }
  }
  uint64_t anc[QPW];
#pragma unroll
  for (int t = 0; t < QPW; ++t) {
    const int qv = (qt0 + t) * 16 + r16;
    anc[t] = t < ntile && qv < Qn ? a.topo.anc[qv % ns] : 0ull;
  }
  __syncthreads();

  const float scale2 = a.scale * kLog2e;
  float mrun[QPW], lrun[QPW];
  floatx4 o[QPW][DSUB];
#pragma unroll
  for (int t = 0; t < QPW; ++t) {
    mrun[t] = -INFINITY;
    lrun[t] = 0.0f;
#pragma unroll
    for (int ds = 0; ds < DSUB; ++ds) o[t][ds] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  for (int sp = 0; sp < nsp; ++sp) {
    const int k0 = (sp0 + sp) * kAttnChunk + 64 * wave;
    const int key_hi = min(T, k0 + 64);  // this wave's keys [k0, key_hi), maybe none
    // V rows into the wave's LDS (its previous block's reads are done: one
    // wave's LDS accesses complete in order)
    wave_lds_sync();
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int key = it * KPI + lane / (HD / 8);
      *reinterpret_cast<u32x4*>(vs + key * Lds::kVS + (lane % (HD / 8)) * 8) = vraw[it];
    }
    bf16x8 kc[4][KSTEPS];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int kk = 0; kk < KSTEPS; ++kk) kc[j][kk] = kf[j][kk];
    wave_lds_sync();
    if (sp + 1 < nsp) load_block(k0 + kAttnChunk);
    __builtin_amdgcn_sched_barrier(0);

    // the tiles phase by phase, so that one tile's latencies (LDS reads,
    // lane exchanges) overlap the others' arithmetic: scores of every tile
    floatx4 sc[QPW][4];
#pragma unroll
    for (int t = 0; t < QPW; ++t) {
      bf16x8 qh[KSTEPS], ql[KSTEPS];
#pragma unroll
      for (int kk = 0; kk < KSTEPS; ++kk) {
        qh[kk] = *reinterpret_cast<const bf16x8*>(q_sh + (t * KSTEPS + kk) * 1024 + lane * 8);
        ql[kk] = *reinterpret_cast<const bf16x8*>(q_sh + (t * KSTEPS + kk) * 1024 + 512 + lane * 8);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sc[t][j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) {
          sc[t][j] = mfma16x16x32(kc[j][kk], qh[kk], sc[t][j]);
          sc[t][j] = mfma16x16x32(kc[j][kk], ql[kk], sc[t][j]);
        }
      }
    }
    // lane holds S^T[key 16j + 4g + r][query r16]: scale (base 2), mask (a
    // block wholly inside the cached context is visible to every query: a
    // branch the whole wave takes), block max, running statistics of query
    // r16, P as bf16 hi + lo
    const bool open = k0 + 64 <= L;
    u32x4 ph[QPW][2], pl[QPW][2];
#pragma unroll
    for (int t = 0; t < QPW; ++t) {
      float mx = -INFINITY;
      if (open) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            sc[t][j][r] *= scale2;
            mx = fmaxf(mx, sc[t][j][r]);
          }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int pos = k0 + 16 * j + 4 * g + r;
            const bool anc_bit = (anc[t] >> ((pos - L) & 63)) & 1ull;
            const bool vis = (pos < key_hi) & ((pos < L) | anc_bit);
            sc[t][j][r] = vis ? sc[t][j][r] * scale2 : -INFINITY;
            mx = fmaxf(mx, sc[t][j][r]);
          }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      // The reference of the running sums moves up only when a block max
      // exceeds it by more than 2^8 (or on the first visible block): the
      // sums and P are exact for any reference at or above the true max
      // minus 8, and the rescale of the output, the costly part, is skipped
      // for most blocks. The decision is the wave's, so the branch is too.
      if (__builtin_amdgcn_read_exec() & __ballot(mx > mrun[t] + 8.0f)) {
        const float mnew = fmaxf(mrun[t], mx);
        const float alpha = mrun[t] == -INFINITY ? 0.0f : exp2_hw(mrun[t] - mnew);
        lrun[t] *= alpha;
        mrun[t] = mnew;
        // o[t][ds][r] belongs to query 4 g + r, whose factor lane 4 g + r holds
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float ar = __shfl(alpha, 4 * g + r);
#pragma unroll
          for (int ds = 0; ds < DSUB; ++ds) o[t][ds][r] *= ar;
        }
      }
      const float mref = mrun[t] == -INFINITY ? 0.0f : mrun[t];
      float ls = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          sc[t][j][r] = exp2_hw(sc[t][j][r] - mref);
          ls += sc[t][j][r];
        }
      ls += __shfl_xor(ls, 16);
      ls += __shfl_xor(ls, 32);
      lrun[t] += ls;
      // P in the k order of the V operand: keys 4 g + r of the two 16-key tiles
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const float p0 = sc[t][2 * kb + (x >> 1)][2 * (x & 1)];
          const float p1 = sc[t][2 * kb + (x >> 1)][2 * (x & 1) + 1];
          ph[t][kb][x] = pack_bf16x2(p0, p1);
          pl[t][kb][x] = pack_bf16x2(p0 - bf_lo(ph[t][kb][x]), p1 - bf_hi(ph[t][kb][x]));
        }
    }
    // O += P V: each V operand read once (the transposing LDS read of the
    // kernel above: dim 16 ds + lane % 16 of keys 32 kb + 4 g + e and
    // 32 kb + 16 + 4 g + e) for every tile
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int ds = 0; ds < DSUB; ++ds) {
        const uint16_t* p0 = vs + (32 * kb + 4 * g + (r16 >> 2)) * Lds::kVS + 16 * ds + 4 * (r16 & 3);
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p0);
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + 16 * Lds::kVS));
        const bf16x8 vb = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
        for (int t = 0; t < QPW; ++t) {
          o[t][ds] = mfma16x16x32(__builtin_bit_cast(bf16x8, ph[t][kb]), vb, o[t][ds]);
          o[t][ds] = mfma16x16x32(__builtin_bit_cast(bf16x8, pl[t][kb]), vb, o[t][ds]);
        }
      }
  }

  const size_t pbase = ((size_t)b * a.n_kv_heads + kvh) * a.max_chunks;
  const __amdgpu_buffer_rsrc_t pco =
      coherent_region(a.part_o + pbase * Qn * HD, (uint32_t)((size_t)a.max_chunks * Qn * HD * 4));
#pragma unroll
  for (int t = 0; t < QPW; ++t) {
    if (t >= ntile) break;
    publish_tile<HD>(region_all, ml_sh, o[t], mrun[t], lrun[t]);
    merge_waves<HD>(a, region_all, ml_sh, b, kvh, qt0 + t, Qn, nch, c, pbase, pco);
  }
  if (nch == 1 || a.defer) return;
  merge_chunks<HD>(a, &last, a.counters + ((size_t)b * a.n_kv_heads + kvh) * QG + qgi, b, kvh, qt0,
                   qt0 + ntile, Qn, nch, pbase, pco);
}

// Long contexts, fed through an LDS ring (head dim 128): a workgroup owns
// a chunk of nb consecutive 256-key spans of one (sequence, kv head) and a
// group of up to 4 query tiles, two compute waves per tile (one per 32-key
// half of every block, so that each SIMD holds two and one's softmax overlaps
// the other's MFMAs; the two halves are merged once at the end). Two loader waves
// copy the chunk's 64-key blocks of K and of V straight from HBM into a ring
// of R LDS slots with global-to-LDS loads, P blocks ahead of the compute
// waves, each waiting on its own load counter; one barrier per block passes
// the slots on (the protocol of the LDS-shared GEMM kernel). Every compute
// wave then reads its half-block's K operands and transposed V operands from
// LDS and keeps its running (max, sum, output) in registers with the online
// softmax of attn_stream_kernel, so a compute unit keeps P blocks (96 KB) in
// flight without registers for them and no wave waits for its own loads. Rows are stored XOR-swizzled by 16-byte unit (K: unit ^ key%16;
// V: unit ^ 2 (key%8)) so that the K operand reads (16 keys, one unit each)
// and the transposing V reads (8 keys, two half-units each per 32 lanes)
// touch every LDS bank once. The chunk's partials are merged as in the
// kernels above (last arrival or the merge kernel).
template <int NQ>
__global__ __launch_bounds__(64 * (2 * NQ + 2)) void attn_ring_kernel(AttnArgs a) {
  constexpr int HD = 128;
  constexpr int KSTEPS = HD / 32;
  constexpr int DSUB = HD / 16;
  constexpr int C4 = HD / 4;
  constexpr int UNITS = HD / 8;             // 16-byte units of a key row
  constexpr int LOADS = 64 * UNITS / 64;    // 1 KB global-to-LDS loads per block of K (or V)
  constexpr int P = 3;                      // blocks in flight ahead of the one computed
  constexpr int R = P + 1;                  // ring slots: refilled one barrier after their last read
  constexpr int ORS = HD + 4;               // floats per row of a wave's output staging
  static_assert((P - 1) * LOADS <= 63, "a loader waits on at most 63 outstanding loads");
  static_assert(R * 2 * 64 * HD * 2 >= 2 * NQ * 16 * ORS * 4, "the output staging reuses the ring");
  __shared__ __attribute__((aligned(16))) uint16_t ring[R][2][64 * HD];
  __shared__ float2 ml_sh[NQ][2][16];
  __shared__ int last;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int G = a.n_heads / a.n_kv_heads;
  const int ns = a.n_slots;
  const int Qn = G * ns;
  const int QT = (Qn + 15) >> 4;
  const int QG = (QT + NQ - 1) / NQ;
  const AttnWg wg = attn_wg(a, (a.max_chunks + a.nb - 1) / a.nb, QG);
  const int b = wg.b, kvh = wg.kvh, qgi = wg.qgi, c = wg.c;
  const int qt0 = qgi * NQ, ntile = min(NQ, QT - qt0);
  const int L = a.len[b];
  const int T = L + ns;
  if (T > a.capacity) {
    if (c == 0 && kvh == 0 && qgi == 0 && tid == 0) atomicOr(a.status, 1u);
    return;
  }
  const int ck = a.nb * kAttnChunk;  // keys per chunk
  const int nch = (T + ck - 1) / ck;
  if (c >= nch) return;
  const int kbeg = c * ck;
  const int nblk = (min(T, kbeg + ck) - kbeg + 63) >> 6;
  const size_t row0 = ((size_t)b * a.n_kv_heads + kvh) * a.capacity;

  floatx4 o[DSUB];
  float mrun = -INFINITY, lrun = 0.0f;
#pragma unroll
  for (int ds = 0; ds < DSUB; ++ds) o[ds] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (wave >= 2 * NQ) {
    // the loaders: wave 2 NQ the K blocks, wave 2 NQ + 1 the V blocks; block i
    // goes to slot i % R, issued after barrier i - P (which the compute waves
    // pass only once done with block i - P - 1, the slot's previous content)
    // and complete before barrier i
    const int isv = wave - 2 * NQ;
    const uint16_t* src = (isv ? a.v_cache : a.k_cache) + row0 * HD;
    auto fetch = [&](int i, int slot) {
      const int k0 = kbeg + 64 * i;
#pragma unroll
      for (int x = 0; x < LOADS; ++x) {
        const int U = x * 64 + lane;  // 16-byte unit of the slot
        const int key = U / UNITS, p = U - key * UNITS;
        const int u = isv ? p ^ ((key & 7) << 1) : p ^ (key & 15);
        const int pos = min(k0 + key, T - 1);  // rows past the last key: a valid row, masked
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(src + (size_t)pos * HD + u * 8),
                                         (__attribute__((address_space(3))) void*)&ring[slot][isv][x * 512], 16, 0,
                                         0);
      }
    };
#pragma unroll
    for (int p = 0; p < P; ++p)
      if (p < nblk) fetch(p, p);
    int slot_in = P % R;
    for (int i = 0; i < nblk; ++i) {
      if (i + P <= nblk) wait_vmcnt<(P - 1) * LOADS>();
      else wait_vmcnt<0>();
      lds_barrier();
      if (i + P < nblk) {
        fetch(i + P, slot_in);
        slot_in = slot_in + 1 == R ? 0 : slot_in + 1;
      }
    }
  } else {
    const int hk = wave & 1;  // keys 32 hk .. 32 hk + 31 of every block
    const int qt = qt0 + (wave >> 1);
    const bool has = (wave >> 1) < ntile;  // a wave past the group's last tile only passes the barriers
    const int qv = qt * 16 + r16;
    const uint64_t anc = has && qv < Qn ? a.topo.anc[qv % ns] : 0ull;
    bf16x8 qh[KSTEPS], ql[KSTEPS];
    {
      const uint16_t* qtile =
          a.q_img + (((size_t)b * a.n_kv_heads + kvh) * QT + (has ? qt : 0)) * (size_t)KSTEPS * 1024 + lane * 8;
      const bool qok = has && qv < Qn;
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
    }
    const float scale2 = a.scale * kLog2e;
    int slot = 0;
    for (int i = 0; i < nblk; ++i) {
      lds_barrier();
      if (has) {
        const uint16_t* ks = ring[slot][0];
        const uint16_t* vsl = ring[slot][1];
        const int k0 = kbeg + 64 * i;
        const int key_hi = min(T, k0 + 64);
        // S^T[key][query] = K Q^T over the wave's half: lane holds key
        // 16 (2 hk + j) + 4 g + r, query r16
        floatx4 sc[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          sc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kk = 0; kk < KSTEPS; ++kk) {
            const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks + (16 * (2 * hk + j) + r16) * HD +
                                                               (((4 * kk + g) ^ r16) << 3));
            sc[j] = mfma16x16x32(kf, qh[kk], sc[j]);
            sc[j] = mfma16x16x32(kf, ql[kk], sc[j]);
          }
        }
        float mx = -INFINITY;
        if (k0 + 64 <= L) {
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              sc[j][r] *= scale2;
              mx = fmaxf(mx, sc[j][r]);
            }
        } else {
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int pos = k0 + 16 * (2 * hk + j) + 4 * g + r;
              const bool anc_bit = (anc >> ((pos - L) & 63)) & 1ull;
              const bool vis = (pos < key_hi) & ((pos < L) | anc_bit);
              sc[j][r] = vis ? sc[j][r] * scale2 : -INFINITY;
              mx = fmaxf(mx, sc[j][r]);
            }
        }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        // the reference of the running sums moves up only when a block max
        // exceeds it by more than 2^8 (as in attn_stream_kernel)
        if (__builtin_amdgcn_read_exec() & __ballot(mx > mrun + 8.0f)) {
          const float mnew = fmaxf(mrun, mx);
          const float alpha = mrun == -INFINITY ? 0.0f : exp2_hw(mrun - mnew);
          lrun *= alpha;
          mrun = mnew;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float ar = __shfl(alpha, 4 * g + r);
#pragma unroll
            for (int ds = 0; ds < DSUB; ++ds) o[ds][r] *= ar;
          }
        }
        const float mref = mrun == -INFINITY ? 0.0f : mrun;
        float ls = 0.0f;
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            sc[j][r] = exp2_hw(sc[j][r] - mref);
            ls += sc[j][r];
          }
        ls += __shfl_xor(ls, 16);
        ls += __shfl_xor(ls, 32);
        lrun += ls;
        // O += P V, P as bf16 hi + lo in the k order of the V operand (keys
        // 4 g + r of the half's two 16-key tiles); V by the transposing LDS
        // read: lane r16 of group g addresses key 32 hk + 4 g + r16 / 4 (and
        // + 16), dims 16 ds + 4 (r16 % 4) .. + 4
        {
          u32x4 ph, pl;
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            const float p0 = sc[x >> 1][2 * (x & 1)];
            const float p1 = sc[x >> 1][2 * (x & 1) + 1];
            ph[x] = pack_bf16x2(p0, p1);
            pl[x] = pack_bf16x2(p0 - bf_lo(ph[x]), p1 - bf_hi(ph[x]));
          }
          const bf16x8 pah = __builtin_bit_cast(bf16x8, ph);
          const bf16x8 pal = __builtin_bit_cast(bf16x8, pl);
          const int kr = 32 * hk + 4 * g + (r16 >> 2);
#pragma unroll
          for (int ds = 0; ds < DSUB; ++ds) {
            const int u = 2 * ds + ((r16 & 3) >> 1);
            const uint16_t* p0 = vsl + kr * HD + ((u ^ ((kr & 7) << 1)) << 3) + 4 * (r16 & 1);
            const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p0);
            const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + 16 * HD));
            const bf16x8 vb = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
            o[ds] = mfma16x16x32(pah, vb, o[ds]);
            o[ds] = mfma16x16x32(pal, vb, o[ds]);
          }
        }
      }
      slot = slot + 1 == R ? 0 : slot + 1;
    }
  }

  // every wave is past its last ring access: the ring becomes the output
  // staging. Each compute wave stages its half's (max, sum, output); then the
  // two waves of a tile merge the halves (each half of the tile's items) and
  // write the tile's output or partial.
  __syncthreads();
  const size_t pbase = ((size_t)b * a.n_kv_heads + kvh) * a.max_chunks;
  const __amdgpu_buffer_rsrc_t pco =
      coherent_region(a.part_o + pbase * Qn * HD, (uint32_t)((size_t)a.max_chunks * Qn * HD * 4));
  float* stage = reinterpret_cast<float*>(&ring[0][0][0]);
  const int tl = wave >> 1, hk = wave & 1;
  if (wave < 2 * ntile) {
    float* os = stage + wave * 16 * ORS;
#pragma unroll
    for (int ds = 0; ds < DSUB; ++ds)
#pragma unroll
      for (int r = 0; r < 4; ++r) os[(4 * g + r) * ORS + ds * 16 + r16] = o[ds][r];
    if (g == 0) ml_sh[tl][hk][r16] = make_float2(mrun, lrun);
  }
  __syncthreads();
  if (wave < 2 * ntile) {
    const float* o0 = stage + 2 * tl * 16 * ORS;
    const float* o1 = o0 + 16 * ORS;
    const int qt = qt0 + tl;
    for (int x = hk * 8 * C4 + lane; x < (hk + 1) * 8 * C4; x += 64) {
      const int qloc = x / C4, c4 = x - qloc * C4;
      const int qg = qt * 16 + qloc;
      if (qg >= Qn) continue;
      const float2 m0 = ml_sh[tl][0][qloc], m1 = ml_sh[tl][1][qloc];
      const float M = fmaxf(m0.x, m1.x);
      const float f0 = m0.x == -INFINITY ? 0.0f : exp2_hw(m0.x - M);
      const float f1 = m1.x == -INFINITY ? 0.0f : exp2_hw(m1.x - M);
      const float4 v0 = *reinterpret_cast<const float4*>(o0 + qloc * ORS + 4 * c4);
      const float4 v1 = *reinterpret_cast<const float4*>(o1 + qloc * ORS + 4 * c4);
      const float4 v = make_float4(v0.x * f0 + v1.x * f1, v0.y * f0 + v1.y * f1, v0.z * f0 + v1.z * f1,
                                   v0.w * f0 + v1.w * f1);
      const float2 ml = make_float2(M, m0.y * f0 + m1.y * f1);
      if (nch == 1) {
        const float inv = ml.y > 0.0f ? 1.0f / ml.y : 0.0f;
        const float out[4] = {v.x * inv, v.y * inv, v.z * inv, v.w * inv};
        write_out4<HD>(a, b, kvh, qg, c4, out);
      } else {
        store_coherent4(pco, (uint32_t)((((size_t)c * Qn + qg) * HD + 4 * c4) * 4),
                        floatx4{v.x, v.y, v.z, v.w});
        if (c4 == 0) store_coherent2(a.part_ml + 2 * ((pbase + c) * Qn + qg), ml.x, ml.y);
      }
    }
  }
  if (nch == 1 || a.defer) return;
  merge_chunks<HD>(a, &last, a.counters + ((size_t)b * a.n_kv_heads + kvh) * QG + qgi, b, kvh, qt0,
                   qt0 + ntile, Qn, nch, pbase, pco);
}

// The chunk merge as a kernel of its own (AttnArgs::defer): one thread per
// (sequence, kv head, query, 4 output dims) of every sequence with more than
// one chunk, the running merge of merge_chunks in chunk order (the same
// arithmetic, so the same bits), output written into the image. The kernel
// boundary orders the chunks' partials before these loads, so the chunk
// workgroups need no drain, counter or last-arrival pass.
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int C4 = HD / 4;
  constexpr int MB = 8;
  const int G = a.n_heads / a.n_kv_heads, ns = a.n_slots, Qn = G * ns;
  const int b = blockIdx.z, kvh = blockIdx.y;
  const int x = blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= Qn * C4) return;
  const int T = a.len[b] + ns;
  if (T > a.capacity) return;  // flagged by the attention kernel
  const int nch = (T + a.nb * kAttnChunk - 1) / (a.nb * kAttnChunk);
  if (nch <= 1) return;        // written by its only chunk
  const int qg = x / C4, c4 = x - qg * C4;
  const size_t pbase = ((size_t)b * a.n_kv_heads + kvh) * a.max_chunks;
  float M = -INFINITY, S = 0.0f, o4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int c0 = 0; c0 < nch; c0 += MB) {
    float2 ml[MB];
    floatx4 v[MB];
#pragma unroll
    for (int u = 0; u < MB; ++u) {
      const int cc = c0 + u < nch ? c0 + u : c0;
      const size_t pidx = (pbase + cc) * Qn + qg;
      ml[u] = *reinterpret_cast<const float2*>(a.part_ml + 2 * pidx);
      v[u] = *reinterpret_cast<const floatx4*>(a.part_o + pidx * HD + 4 * c4);
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
  float out[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = o4[e] * inv;
  write_out4<HD>(a, b, kvh, qg, c4, out);
}

}  // namespace

hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t s) {
  if (a.max_chunks > kMaxAttnChunks || a.max_chunks < 1) return hipErrorInvalidValue;
  if (a.max_chunks > 1 && !a.counters) return hipErrorInvalidValue;
  if (head_dim != 128 && head_dim != 64) return hipErrorInvalidValue;
  const int qt = (a.n_heads / a.n_kv_heads * a.n_slots + 15) / 16;
  if (a.q_per_wg < 1 || a.nb < 1) return hipErrorInvalidValue;
  const int qg = (qt + a.q_per_wg - 1) / a.q_per_wg;
  if (a.ring) {
    // the ring-fed kernel: head dim 128, up to 4 query tiles a workgroup
    if (head_dim != 128 || a.q_per_wg > 4) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((a.max_chunks + a.nb - 1) / a.nb) * a.n_kv_heads * qg * a.batch);
    switch (a.q_per_wg) {
      case 1: hipLaunchKernelGGL((attn_ring_kernel<1>), grid, dim3(64 * 4), 0, s, a); break;
      case 2: hipLaunchKernelGGL((attn_ring_kernel<2>), grid, dim3(64 * 6), 0, s, a); break;
      case 3: hipLaunchKernelGGL((attn_ring_kernel<3>), grid, dim3(64 * 8), 0, s, a); break;
      default: hipLaunchKernelGGL((attn_ring_kernel<4>), grid, dim3(64 * 10), 0, s, a); break;
    }
    return hipGetLastError();
  }
  if (a.nb > 1) {
    // the streaming kernel: up to 3 query tiles a workgroup, chunks of nb spans
    if (a.q_per_wg > 3) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((a.max_chunks + a.nb - 1) / a.nb) * a.n_kv_heads * qg * a.batch);
    const int qpw = a.q_per_wg;
    if (head_dim == 128) {
      if (qpw == 1) hipLaunchKernelGGL((attn_stream_kernel<128, 1>), grid, dim3(256), 0, s, a);
      else if (qpw == 2) hipLaunchKernelGGL((attn_stream_kernel<128, 2>), grid, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((attn_stream_kernel<128, 3>), grid, dim3(256), 0, s, a);
    } else {
      if (qpw == 1) hipLaunchKernelGGL((attn_stream_kernel<64, 1>), grid, dim3(256), 0, s, a);
      else if (qpw == 2) hipLaunchKernelGGL((attn_stream_kernel<64, 2>), grid, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((attn_stream_kernel<64, 3>), grid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
  }
  const dim3 grid((unsigned)a.max_chunks * a.n_kv_heads * qg * a.batch);
  const bool multi = a.q_per_wg > 1 && qt > 1;
  if (head_dim == 128) {
    if (multi) hipLaunchKernelGGL((attn_kernel<128, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((attn_kernel<128, false>), grid, dim3(256), 0, s, a);
  } else {
    if (multi) hipLaunchKernelGGL((attn_kernel<64, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((attn_kernel<64, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_attention_merge(int head_dim, const AttnArgs& a, hipStream_t s) {
  const int qn = a.n_heads / a.n_kv_heads * a.n_slots;
  const dim3 grid((qn * (head_dim / 4) + 255) / 256, a.n_kv_heads, a.batch);
  if (head_dim == 128) hipLaunchKernelGGL((attn_merge_kernel<128>), grid, dim3(256), 0, s, a);
  else if (head_dim == 64) hipLaunchKernelGGL((attn_merge_kernel<64>), grid, dim3(256), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace msd
