// Skinny weight-streaming GEMM for the verification pass: Y = norm(X) W^T with
// X = the block's rows (M = batch * n_slots <= 144) and W a bf16 weight
// matrix [N][K] read exactly once. This is where the verify step spends its
// bytes: every projection of every layer plus the two LM-head passes.
//
// Mapping (gfx950, wave64, MFMA 16x16x32 bf16 -> fp32):
//  * a workgroup of NW waves owns a 64-column output tile (128 columns for
//    the FFN up projection and the LM head, 32 for the QKV projection at
//    one row tile) and one of `splits` contiguous slices of K; its waves cut
//    the slice in NW k-ranges;
//  * weights are stored k-step-major (for each k-step, the 1 KB MFMA operands
//    of all 16-row groups one after the other), so the workgroups working at
//    the same k-step read one contiguous window of HBM; each wave keeps D
//    k-steps in flight with non-temporal loads, straight into the MFMA;
//  * the input is an activation image: X (times the pre-norm gain) already
//    split into bf16 hi + lo parts in MFMA operand order by the kernel that
//    produced it, so the loop is loads and MFMAs only (two MFMAs per weight
//    fragment, about 16-bit activations against the exact bf16 weights);
//  * operands are swapped (D = W X^T): each lane ends with 4 consecutive
//    output columns of one row, which makes the epilogues vector-friendly;
//  * the waves' tiles are summed in LDS in a fixed order; with split-K wave 0
//    publishes the tile with coherent stores and the last workgroup of the
//    tile to arrive sums all splits in split order. No floating-point
//    atomics: results are bit-reproducible;
//  * the row-wise pre-norm is applied after the product (its per-row scale
//    commutes with W), from (mean, M2) summaries the producer left behind;
//  * epilogues (residual + statistics, RoPE + KV append, SwiGLU / ReLU, LM
//    head statistics) write the next GEMM's activation image directly.
#include "kernels.h"

namespace msd {
namespace {

// Weights live in the k-step-major layout (see repack_kernel): fragment
// (G, ks) of a matrix with NG = rows / 16 groups is the 1 KB block at element
// (ks * NG + G) * 512, holding rows 16G..16G+15 x columns 32ks..32ks+31 in
// MFMA operand order (lane l: row 16G + l%16, columns 32ks + 8(l/16) .. +8).
// A tile is JT sub-tiles of 16 output columns (JT = 4: 64 columns; JT = 8:
// 128 columns). Returns the lane's pointer into fragment (group, 0) of the
// group feeding sub-tile j.
template <int JT>
__device__ __forceinline__ const uint16_t* weight_frag(const GemmArgs& a, int t, int j, int lane) {
  const uint16_t* base;
  int grp;
  if (a.map == MAP_QKV) {  // a tile is 8 JT rotary pairs of one head (JT = 4 or 2)
    constexpr int HJ = JT / 2;
    const int hd = a.head_dim, half = hd >> 1, tph = hd / (32 * HJ);
    const int hh = t / tph, gi = t - hh * tph;
    const int c0 = j < HJ ? gi * 16 * HJ + 16 * j : half + gi * 16 * HJ + 16 * (j - HJ);
    int hl = hh;
    base = a.w0;
    if (hh >= a.n_heads + a.n_kv_heads) {
      base = a.w2;
      hl = hh - a.n_heads - a.n_kv_heads;
    } else if (hh >= a.n_heads) {
      base = a.w1;
      hl = hh - a.n_heads;
    }
    grp = (hl * hd + c0) >> 4;
  } else if (a.map == MAP_GATEUP) {  // JT/2 gate groups, then the same JT/2 of up
    constexpr int HJ = JT / 2;
    base = j < HJ ? a.w0 : a.w1;
    grp = HJ * t + (j % HJ);
  } else {
    base = a.w0;
    grp = JT * t + j;
    const int last = (a.N >> 4) - 1;  // padding columns re-read a valid group; output masked
    if (grp > last) grp = last;
  }
  return base + (size_t)grp * 512 + lane * 8;
}

// Elements from one k-step of tile t's weights to the next: the group count
// of its matrix times 512 (the same for every sub-tile of a tile: one
// matrix, or the gate and up matrices of equal size).
template <int JT = 4>
__device__ __forceinline__ uint32_t weight_kstride(const GemmArgs& a, int t) {
  int rows;
  if (a.map == MAP_QKV) {
    const int hh = t / (a.head_dim / (16 * JT));
    rows = (hh < a.n_heads ? a.n_heads : a.n_kv_heads) * a.head_dim;
  } else if (a.map == MAP_GATEUP) {
    rows = a.N >> 1;
  } else {
    rows = a.N;
  }
  return (uint32_t)(rows >> 4) * 512u;
}

// Logical output column (index into biases and LayerNorm column sums) of
// value r of sub-tile j in lane group q of tile t.
template <int JT>
__device__ __forceinline__ int out_col(const GemmArgs& a, int t, int j, int q, int r) {
  if (a.map == MAP_QKV) {
    constexpr int HJ = JT / 2;
    const int hd = a.head_dim, half = hd >> 1, tph = hd / (32 * HJ);
    const int hh = t / tph, gi = t - hh * tph;
    const int dim = (j < HJ ? 0 : half) + gi * 16 * HJ + 16 * (j % HJ) + 4 * q + r;
    return hh * hd + dim;
  }
  if (a.map == MAP_GATEUP) {
    constexpr int HJ = JT / 2;
    const int f = 16 * HJ * t + 16 * (j % HJ) + 4 * q + r;
    return j < HJ ? f : (a.N >> 1) + f;
  }
  return 16 * JT * t + 16 * j + 4 * q + r;
}

// ---------------------------------------------------------------------------
// epilogue inputs that do not depend on the product
// ---------------------------------------------------------------------------
constexpr int kMaxPer = 40;  // pre-norm summaries per lane: K <= 40 * 4 * 64 = 10240
constexpr u32x4 kUnitGain = {0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};  // bf16 1.0 pairs

// Per lane (row 16 mt + l%16, lane group q = l/16) of one row tile. With one
// row tile the finishing wave loads them right after its k-loop, so that
// their round trip overlaps the wave reduction and the split-K hand-off;
// with more row tiles each row tile loads its own inside the epilogue.
struct EpiIn {
  float2 st[kMaxPer];  // pre-norm: the row's 64-column (mean, M2) summaries q, q+4, ...
  float4 x[4];         // EPI_RESID: residual x[m][64 t + 16 j + 4 q ..]
  u32x2 bias[4];       // EPI_RESID: its bias (bf16 pairs)
  u32x4 gain[2][2];    // EPI_RESID: gains of the two images, halves h = 0, 1
  int L;               // EPI_QKV: committed length of the row's sequence
  float2 cs[2][4];     // EPI_QKV: rotary (cos, sin) of the row's position
  u32x2 qb[2][2];      // EPI_QKV: bias (bf16 pairs), [j][lo / hi half]
};

template <int EPI>
__host__ __device__ constexpr bool has_norm() {
  return EPI != EPI_RESID;
}

// One row tile with a pre-norm (the QKV and FFN up projections): one more
// wave, beside the NW that stream the weights, loads the producer's row
// summaries at the start of the kernel and leaves each row's (mu, r) in
// LDS, so the epilogue after the k-loop has no summary loads or merge left.
// Only for 2- and 8-wave workgroups: a fifth wave would cost the 4-wave ones
// (the LM head, wide one-row-tile GEMMs) their second workgroup per compute
// unit, or registers.
template <int MT, int NW, int EPI>
__host__ __device__ constexpr bool norm_helper() {
  return MT == 1 && (NW == 2 || NW == 8) && has_norm<EPI>() && EPI != EPI_HEAD;
}
template <int MT, int NW, int EPI>
__host__ __device__ constexpr int block_waves() {
  return NW + (norm_helper<MT, NW, EPI>() ? 1 : 0);
}

// committed length of the sequence of row m (EPI_QKV)
__device__ __forceinline__ int row_len(const GemmArgs& a, int m) {
  return a.len[(m < a.M ? m : 0) / a.n_slots];
}

// the pre-norm summaries of the lane's row of row tile mt
__device__ __forceinline__ void stats_load(const GemmArgs& a, int mt, EpiIn& in) {
  const int lane = threadIdx.x & 63, q = lane >> 4, r16 = lane & 15;
  const int m = 16 * mt + r16;
  const int mm = m < a.M ? m : 0;
  if (a.norm.kind != 0) {
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
      const int tt = q + 4 * i;
      in.st[i] = a.norm.stats[(size_t)(tt < a.norm.tiles ? tt : 0) * a.M + mm];
    }
  }
}

template <int EPI, bool NORM = true, int JT = 4>
__device__ __forceinline__ void epi_load(const GemmArgs& a, int t, int mt, EpiIn& in) {
  const int lane = threadIdx.x & 63, q = lane >> 4, r16 = lane & 15;
  const int m = 16 * mt + r16;
  const int mm = m < a.M ? m : 0;
  if constexpr (has_norm<EPI>() && NORM) stats_load(a, mt, in);
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n0 = kTileN * t + 16 * j + 4 * q;
      in.x[j] = *reinterpret_cast<const float4*>(a.x + (size_t)mm * a.N + n0);
      in.bias[j] = a.b0 ? *reinterpret_cast<const u32x2*>(a.b0 + n0) : u32x2{0u, 0u};
    }
#pragma unroll
    for (int o = 0; o < 2; ++o)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        in.gain[o][h] = a.img_out[o].img && a.img_out[o].gain
                            ? *reinterpret_cast<const u32x4*>(a.img_out[o].gain + kTileN * t + 32 * h + 8 * q)
                            : kUnitGain;
  }
  if constexpr (EPI == EPI_QKV) {
    constexpr int HJ = JT / 2;  // rotary pairs of a tile: 16 HJ
    const int hd = a.head_dim, half = hd >> 1, tph = hd / (32 * HJ);
    const int H = a.n_heads, Hk = a.n_kv_heads;
    const int hh = t / tph, gi = t - hh * tph;
    const int which = hh < H ? 0 : (hh < H + Hk ? 1 : 2);
    const int hloc = hh - (which == 0 ? 0 : (which == 1 ? H : H + Hk));
    const uint16_t* bias = which == 0 ? a.b0 : (which == 1 ? a.b1 : a.b2);
    const int slot = mm - (mm / a.n_slots) * a.n_slots;
    int pos = in.L + a.depth[slot];
    pos = pos < 0 ? 0 : (pos < a.rope_rows ? pos : a.rope_rows - 1);  // out-of-range rows are flagged, not used
#pragma unroll
    for (int j = 0; j < HJ; ++j) {
      const int dlo = gi * 16 * HJ + 16 * j + 4 * q, dhi = half + dlo;
      if (which < 2 && a.rope) {
        const float2* cs = a.rope + (size_t)pos * half + dlo;
#pragma unroll
        for (int r = 0; r < 4; ++r) in.cs[j][r] = cs[r];
      }
      in.qb[j][0] = bias ? *reinterpret_cast<const u32x2*>(bias + hloc * hd + dlo) : u32x2{0u, 0u};
      in.qb[j][1] = bias ? *reinterpret_cast<const u32x2*>(bias + hloc * hd + dhi) : u32x2{0u, 0u};
    }
  }
}

// Per-row (mu, r) of the pre-norm from the producer's per-64-column
// (mean, M2) summaries. All summaries count 64 columns, so the row's mean is
// the mean of the summary means and
//   M2 = sum_i M2_i + 64 sum_i (mean_i - mean)^2
// (the exact merge of equal-count groups). The four lanes of a row each hold
// every fourth summary and their partial sums are combined by a butterfly,
// which gives all four lanes identical bits.
__device__ __forceinline__ void norm_finish(const GemmArgs& a, const EpiIn& in, float& mu,
                                            float& rs) {
  const int q = (threadIdx.x & 63) >> 4;
  const RowNorm& nm = a.norm;
  mu = 0.0f;
  rs = 1.0f;
  if (nm.kind == 0) return;
  float sm = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i)
    if (q + 4 * i < nm.tiles) sm += in.st[i].x;
  sm += __shfl_xor(sm, 16);
  sm += __shfl_xor(sm, 32);
  const float mean = sm / (float)nm.tiles;
  float m2 = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i)
    if (q + 4 * i < nm.tiles) {
      const float dv = in.st[i].x - mean;
      m2 += in.st[i].y + (float)kTileN * dv * dv;
    }
  m2 += __shfl_xor(m2, 16);
  m2 += __shfl_xor(m2, 32);
  const float var = m2 / (float)a.K;
  if (nm.kind == 1) {
    rs = 1.0f / sqrtf(var + mean * mean + nm.eps);
  } else {
    rs = 1.0f / sqrtf(var + nm.eps);
    mu = mean;
  }
}

// normalised value of an accumulator entry
__device__ __forceinline__ float normed(const GemmArgs& a, float acc, float mu, float rs, int col) {
  if (a.norm.kind == 2) return rs * acc - rs * mu * a.norm.col_g[col] + a.norm.col_b[col];
  return a.norm.kind == 1 ? rs * acc : acc;
}

constexpr int kScr = kTileN + 4;  // scratch row stride (floats)

// Image of 32 consecutive columns [c0, c0 + 32) of a 16-row tile held in
// scratch[16][kScr], times the lane's 8 gains (bf16 pairs), written as image
// k-step ks.
__device__ __forceinline__ void scratch_to_image(const float* scr, int c0, const u32x4& gw, int M,
                                                 int mt, int MT, int ks, uint16_t* img) {
  const int lane = threadIdx.x & 63, r16 = lane & 15, q = lane >> 4;
  const float* src = scr + r16 * kScr + c0 + 8 * q;
  const float4 v0 = *reinterpret_cast<const float4*>(src);
  const float4 v1 = *reinterpret_cast<const float4*>(src + 4);
  float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] *= bf_lo(gw[i]);
    v[2 * i + 1] *= bf_hi(gw[i]);
  }
  const bool valid = 16 * mt + r16 < M;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = valid ? v[e] : 0.0f;
  u32x4 h, l;
  split8_words(v, h, l);
  uint16_t* dst = img + img_offset(ks, mt, MT, lane);
  *reinterpret_cast<u32x4*>(dst) = h;
  *reinterpret_cast<u32x4*>(dst + 512) = l;
}

// ---------------------------------------------------------------------------
// epilogues (wave 0 of the finishing workgroup), one row tile mt at a time;
// lane l, value [j][r]: row 16 mt + l%16, column 64 t + 16 j + 4 (l/16) + r
// ---------------------------------------------------------------------------
__device__ void epi_resid(const GemmArgs& a, int t, int mt, const floatx4 (&acc)[4], float* scr,
                          const EpiIn& in) {
  const int lane = threadIdx.x & 63, r16 = lane & 15, q = lane >> 4;
  const int m = 16 * mt + r16;
  const bool valid = m < a.M;
  const int mm = valid ? m : 0;
  float v[4][4];
  float sum = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n0 = kTileN * t + 16 * j + 4 * q;
    const float bb[4] = {bf_lo(in.bias[j][0]), bf_hi(in.bias[j][0]), bf_lo(in.bias[j][1]),
                         bf_hi(in.bias[j][1])};
    const float xs[4] = {in.x[j].x, in.x[j].y, in.x[j].z, in.x[j].w};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      v[j][r] = valid ? xs[r] + (acc[j][r] + bb[r]) : 0.0f;
      sum += v[j][r];
    }
    if (valid)
      *reinterpret_cast<float4*>(a.x + (size_t)mm * a.N + n0) = make_float4(v[j][0], v[j][1], v[j][2], v[j][3]);
  }
  if (a.stats_out) {
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    const float mean = sum * (1.0f / kTileN);
    float m2 = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float dv = v[j][r] - mean;
        m2 += dv * dv;
      }
    m2 += __shfl_xor(m2, 16);
    m2 += __shfl_xor(m2, 32);
    if (q == 0 && valid) a.stats_out[(size_t)t * a.M + m] = make_float2(mean, m2);
  }
  if (a.img_out[0].img || a.img_out[1].img) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<float4*>(scr + r16 * kScr + 16 * j + 4 * q) =
          make_float4(v[j][0], v[j][1], v[j][2], v[j][3]);
    wave_lds_sync();
#pragma unroll
    for (int o = 0; o < 2; ++o) {
      if (!a.img_out[o].img) continue;
#pragma unroll
      for (int h = 0; h < 2; ++h)
        scratch_to_image(scr, 32 * h, in.gain[o][h], a.M, mt, a.MT, 2 * t + h, a.img_out[o].img);
    }
    wave_lds_sync();
  }
}

template <int JT>
__device__ void epi_swiglu(const GemmArgs& a, int t, int mt, const floatx4 (&acc)[JT], float* scr,
                           float mu, float rs) {
  constexpr int HJ = JT / 2;  // gate sub-tiles j < HJ pair with up sub-tiles j + HJ
  const int lane = threadIdx.x & 63, r16 = lane & 15, q = lane >> 4;
#pragma unroll
  for (int j = 0; j < HJ; ++j) {
    float act[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float g = normed(a, acc[j][r], mu, rs, out_col<JT>(a, t, j, q, r));
      const float u = normed(a, acc[j + HJ][r], mu, rs, out_col<JT>(a, t, j + HJ, q, r));
      act[r] = silu(g) * u;
    }
    *reinterpret_cast<float4*>(scr + r16 * kScr + 16 * j + 4 * q) =
        make_float4(act[0], act[1], act[2], act[3]);
  }
  wave_lds_sync();
#pragma unroll
  for (int h = 0; h < HJ / 2; ++h)  // 16 HJ activation columns = HJ / 2 image k-steps
    scratch_to_image(scr, 32 * h, kUnitGain, a.M, mt, a.MT, (HJ / 2) * t + h, a.act_img);
  wave_lds_sync();
}

__device__ void epi_relu(const GemmArgs& a, int t, int mt, const floatx4 (&acc)[4], float* scr,
                         float mu, float rs) {
  const int lane = threadIdx.x & 63, r16 = lane & 15, q = lane >> 4;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int col = out_col<4>(a, t, j, q, r);
      float y = normed(a, acc[j][r], mu, rs, col);
      if (a.b0) y += bf2f(a.b0[col]);
      v[r] = fmaxf(y, 0.0f);
    }
    *reinterpret_cast<float4*>(scr + r16 * kScr + 16 * j + 4 * q) = make_float4(v[0], v[1], v[2], v[3]);
  }
  wave_lds_sync();
#pragma unroll
  for (int h = 0; h < 2; ++h) scratch_to_image(scr, 32 * h, kUnitGain, a.M, mt, a.MT, 2 * t + h, a.act_img);
  wave_lds_sync();
}

template <int JT>
__device__ void epi_qkv(const GemmArgs& a, int t, int mt, const floatx4 (&acc)[JT], float mu,
                        float rs, const EpiIn& in) {
  constexpr int HJ = JT / 2;  // sub-tile j holds dims d of rotary pairs (d, d + half) with sub-tile j + HJ
  const int lane = threadIdx.x & 63, r16 = lane & 15, q = lane >> 4;
  const int hd = a.head_dim, half = hd >> 1, tph = hd / (32 * HJ);
  const int H = a.n_heads, Hk = a.n_kv_heads;
  const int hh = t / tph, gi = t - hh * tph;
  const int which = hh < H ? 0 : (hh < H + Hk ? 1 : 2);
  const int hloc = hh - (which == 0 ? 0 : (which == 1 ? H : H + Hk));
  const int m = 16 * mt + r16;
  if (m >= a.M) return;
  const int b = m / a.n_slots, slot = m - b * a.n_slots;
  const int L = in.L;
  if (L < 0 || L + a.n_slots > a.capacity) {
    if (q == 0 && slot == 0) atomicOr(a.status, 1u);
    return;
  }
#pragma unroll
  for (int j = 0; j < HJ; ++j) {
    const int dlo = gi * 16 * HJ + 16 * j + 4 * q, dhi = half + dlo;
    const float blo[4] = {bf_lo(in.qb[j][0][0]), bf_hi(in.qb[j][0][0]), bf_lo(in.qb[j][0][1]),
                          bf_hi(in.qb[j][0][1])};
    const float bhi[4] = {bf_lo(in.qb[j][1][0]), bf_hi(in.qb[j][1][0]), bf_lo(in.qb[j][1][1]),
                          bf_hi(in.qb[j][1][1])};
    float lo[4], hi[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      lo[r] = normed(a, acc[j][r], mu, rs, hh * hd + dlo + r) + blo[r];
      hi[r] = normed(a, acc[j + HJ][r], mu, rs, hh * hd + dhi + r) + bhi[r];
    }
    if (which < 2 && a.rope) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float2 c = in.cs[j][r];
        const float rl = lo[r] * c.x - hi[r] * c.y;
        const float rh = hi[r] * c.x + lo[r] * c.y;
        lo[r] = rl;
        hi[r] = rh;
      }
    }
    if (which == 0) {
      // the attention's operand image of this query row: head hloc is query
      // gq of kv head kvh; four consecutive dims sit in one lane's 8
      const int G = H / Hk, kvh = hloc / G, gq = hloc - kvh * G;
      const int qv = gq * a.n_slots + slot, qt = qv >> 4, ql = qv & 15;
      uint16_t* tile = a.q_img + (((size_t)b * Hk + kvh) * a.q_tiles + qt) * (size_t)(hd / 32) * 1024;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int d0 = h2 == 0 ? dlo : dhi;
        const float* v = h2 == 0 ? lo : hi;
        uint16_t* dst = tile + (size_t)(d0 >> 5) * 1024 + (ql + 16 * ((d0 & 31) >> 3)) * 8 + (d0 & 7);
        u32x2 hw, lw;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          hw[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
          lw[e] = pack_bf16x2(v[2 * e] - bf_lo(hw[e]), v[2 * e + 1] - bf_hi(hw[e]));
        }
        *reinterpret_cast<u32x2*>(dst) = hw;
        *reinterpret_cast<u32x2*>(dst + 512) = lw;
      }
    } else {
      uint16_t* cache = which == 1 ? a.k_cache : a.v_cache;
      uint16_t* row = cache + (((size_t)b * Hk + hloc) * a.capacity + L + slot) * hd;
      const u32x2 wl = {pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3])};
      const u32x2 wh = {pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3])};
      *reinterpret_cast<u32x2*>(row + dlo) = wl;
      *reinterpret_cast<u32x2*>(row + dhi) = wh;
    }
  }
}

// Per row of the tile: logits out, (max, sum exp), top-kappa rank keys.
template <int JT>
__device__ void epi_head(const GemmArgs& a, int t, int mt, const floatx4 (&acc)[JT], float mu,
                         float rs) {
  constexpr int TW = 16 * JT;  // tile width
  const int lane = threadIdx.x & 63, r16 = lane & 15, q = lane >> 4;
  const int m = 16 * mt + r16;
  const bool valid = m < a.M;
  float v[JT][4];
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < JT; ++j) {
    const int n0 = TW * t + 16 * j + 4 * q;
    const bool cv = TW * t + 16 * j < a.N;  // N % 16 == 0: whole groups
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      v[j][r] = cv ? normed(a, acc[j][r], mu, rs, cv ? n0 + r : 0) : -INFINITY;
      mx = fmaxf(mx, v[j][r]);
    }
    if (a.logits && valid && cv)
      *reinterpret_cast<float4*>(a.logits + (size_t)m * a.N + n0) =
          make_float4(v[j][0], v[j][1], v[j][2], v[j][3]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  float se = 0.0f;
#pragma unroll
  for (int j = 0; j < JT; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) se += v[j][r] == -INFINITY ? 0.0f : expf(v[j][r] - mx);
  se += __shfl_xor(se, 16);
  se += __shfl_xor(se, 32);
  if (q == 0 && valid) a.tile_ms[(size_t)t * a.M + m] = make_float2(mx, se);
  uint64_t key[JT][4];
#pragma unroll
  for (int j = 0; j < JT; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      key[j][r] = v[j][r] == -INFINITY ? 0ull : rank_key(v[j][r], TW * t + 16 * j + 4 * q + r);
  uint64_t* top = a.tile_top + ((size_t)t * a.M + (valid ? m : 0)) * a.kappa;
  for (int rr = 0; rr < a.kappa; ++rr) {
    uint64_t best = 0ull;
#pragma unroll
    for (int j = 0; j < JT; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) best = key[j][r] > best ? key[j][r] : best;
    uint64_t o = __shfl_xor(best, 16);
    best = o > best ? o : best;
    o = __shfl_xor(best, 32);
    best = o > best ? o : best;
#pragma unroll
    for (int j = 0; j < JT; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) key[j][r] = key[j][r] == best ? 0ull : key[j][r];
    if (q == 0 && valid) top[rr] = best;
  }
}

// The epilogue of row tile mt of a finished tile; `in` holds its inputs
// when they were loaded ahead (one row tile), otherwise they are loaded here.
// norm_sh: (mu, r) of the tile's 16 rows, already merged (then NLDS: the
// summaries are not loaded)
template <int EPI, int JT, bool AHEAD, bool NLDS = false>
__device__ __forceinline__ void epilogue_tile(const GemmArgs& a, int t, int mt, const floatx4 (&acc)[JT],
                                              float* scr, const EpiIn& in1, const float2* norm_sh = nullptr) {
  EpiIn inl;
  if constexpr (!AHEAD) {
    if constexpr (EPI == EPI_QKV) inl.L = row_len(a, 16 * mt + (threadIdx.x & 15));
    epi_load<EPI, !NLDS, JT>(a, t, mt, inl);
  }
  const EpiIn& in = AHEAD ? in1 : inl;
  float mu = 0.0f, rs = 1.0f;
  if constexpr (has_norm<EPI>()) {
    if (norm_sh) {  // the helper wave's (mu, r) of this lane's row
      const float2 v = norm_sh[threadIdx.x & 15];
      mu = v.x;
      rs = v.y;
    } else {
      norm_finish(a, in, mu, rs);
    }
  }
  if constexpr (EPI == EPI_SWIGLU) epi_swiglu<JT>(a, t, mt, acc, scr, mu, rs);
  else if constexpr (EPI == EPI_HEAD) epi_head<JT>(a, t, mt, acc, mu, rs);
  else if constexpr (EPI == EPI_QKV) epi_qkv<JT>(a, t, mt, acc, mu, rs, in);  // 64- or 32-column tiles
  else if constexpr (JT == 4) {  // the other epilogues run on 64-column tiles only
    if constexpr (EPI == EPI_RESID) epi_resid(a, t, mt, acc, scr, in);
    else epi_relu(a, t, mt, acc, scr, mu, rs);
  }
}

// The epilogues of the row tiles a wave owns (row tile mt belongs to wave
// mt % owners). At 9 row tiles one copy of the per-tile code runs in a loop
// (unrolled, the 9 copies made the kernel 3.8 times larger and slower by a
// little); each pass picks its row tile's accumulators by compile-time
// index, so acc is never indexed at run time (that would put it in scratch
// memory).
template <int MT, int EPI, int JT, bool NLDS = false>
__device__ __forceinline__ void epilogue_rows(const GemmArgs& a, int t, const floatx4 (&acc)[MT][JT],
                                              float* scr, int owner, int owners,
                                              const float2* norm_sh = nullptr) {
  if constexpr (MT <= 5) {
    // up to 5 row tiles: unrolled (the compact loop below costs these
    // variants their second wave per SIMD)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (mt % owners != owner) continue;
      EpiIn none;
      epilogue_tile<EPI, JT, false, NLDS>(a, t, mt, acc[mt], scr, none, NLDS ? norm_sh + 16 * mt : nullptr);
    }
    return;
  }
#pragma clang loop unroll(disable)
  for (int mt = owner; mt < MT; mt += owners) {
    floatx4 cur[JT];
#pragma unroll
    for (int mm = 0; mm < MT; ++mm)
      if (mm == mt)
#pragma unroll
        for (int j = 0; j < JT; ++j) cur[j] = acc[mm][j];
    EpiIn none;
    epilogue_tile<EPI, JT, false, NLDS>(a, t, mt, cur, scr, none, NLDS ? norm_sh + 16 * mt : nullptr);
  }
}

template <int MT, int JT>
struct KStep {
  bf16x8 w[JT];
  bf16x8 ah[MT], al[MT];
};

template <int MT, int NW, int EPI, int JT>
__global__ __launch_bounds__((64 * block_waves<MT, NW, EPI>())) void gemm_kernel(GemmArgs a) {
  // k-steps in flight per wave (measured per shape with the k-step-major
  // layout: the 2-wave 128-column FFN up tiles 5, 8-wave split-K tiles 6)
  constexpr int D = MT == 1 ? (JT == 8 ? (NW == 2 ? 5 : 4) : (JT == 2 ? 6 : (NW == 8 ? 4 : 8))) : (MT <= 3 ? 4 : 2);
  constexpr int RCH = MT < 3 ? MT : 3;  // row tiles per LDS reduction round
  constexpr int TF = MT * JT * 256;     // floats of one tile's partial
  __shared__ floatx4 red[NW][RCH * JT][kWave];
  // epilogue scratch: one region, or one a wave when the waves share the row
  // tiles' epilogues
  __shared__ __attribute__((aligned(16))) float scr_all[(MT == 1 ? 1 : NW) * 16 * kScr];
  __shared__ int last_sh;
  __shared__ float2 norm_sh[16];  // helper wave: (mu, r) per row of the tile

  const int lane = threadIdx.x & 63;
  // wave-uniform (scalar) so that the k-loop branches and waits are scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t = blockIdx.x / a.splits, s = blockIdx.x - t * a.splits;
  if constexpr (norm_helper<MT, NW, EPI>()) {
    if (wave == NW) {
      // the row norm, while the other waves stream; then the reduction's two
      // barriers, which order the LDS write before the epilogue reads it
      EpiIn hin;
      epi_load<EPI, true, JT>(a, t, 0, hin);
      float mu, rs;
      norm_finish(a, hin, mu, rs);
      if (lane < 16) norm_sh[lane] = make_float2(mu, rs);
      __syncthreads();
      __syncthreads();
      return;
    }
  }
  const int KS = a.K >> 5;
  const int kb0 = (int)((int64_t)KS * s / a.splits), ke0 = (int)((int64_t)KS * (s + 1) / a.splits);
  const int nk = ke0 - kb0;
  const int kb = kb0 + nk * wave / NW, ke = kb0 + nk * (wave + 1) / NW;
  const int n = ke - kb;

  const uint16_t* wp[JT];
#pragma unroll
  for (int j = 0; j < JT; ++j) wp[j] = weight_frag<JT>(a, t, j, lane);
  const size_t kstr = __builtin_amdgcn_readfirstlane(weight_kstride<JT>(a, t));
  const uint16_t* ap = a.a_img + lane * 8;

  // one row tile: the epilogue's inputs are loaded ahead (the sequence
  // length that addresses the rotary table before the k-loop)
  EpiIn in1;
  if constexpr (MT == 1 && EPI == EPI_QKV) in1.L = row_len(a, lane & 15);

  floatx4 acc[MT][JT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < JT; ++j) acc[mt][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Several row tiles: a wave takes its k-steps from a point rotated by the
  // tile index, so that workgroups running at the same time read different
  // k-steps of the activation image, which every workgroup shares (the same
  // k-step requested by every CU at once would queue on a few L2 channels).
  // The order is fixed per tile: sums stay bit-reproducible.
  const int rot = MT > 1 && n > 0 ? (int)((int64_t)n * (t & 15) / 16) : 0;
  auto kstep = [&](int i) {
    if constexpr (MT == 1) return kb + i;
    const int x = i + rot;
    return kb + (x >= n ? x - n : x);
  };
  KStep<MT, JT> st[D];
  auto issue = [&](KStep<MT, JT>& x, int k) {
#pragma unroll
    for (int j = 0; j < JT; ++j) x.w[j] = load_nt(wp[j] + (size_t)k * kstr);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const uint16_t* p = ap + (size_t)(k * MT + mt) * 1024;
      x.ah[mt] = load16(p);
      x.al[mt] = load16(p + 512);
    }
  };
  auto compute = [&](const KStep<MT, JT>& x) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int j = 0; j < JT; ++j) {
        acc[mt][j] = mfma16x16x32(x.w[j], x.ah[mt], acc[mt][j]);
        acc[mt][j] = mfma16x16x32(x.w[j], x.al[mt], acc[mt][j]);
      }
  };
  // D k-steps in flight per wave (n is wave-uniform). The steady-state loop
  // runs only over batches whose D refills are all real, so its body has no
  // branch and each wait leaves the D-1 younger k-steps in flight; the last
  // batch and a short run (n < D: every load issued up front) come after.
  if (n >= D) {
#pragma unroll
    for (int d = 0; d < D; ++d) issue(st[d], kstep(d));
    const int nfull = (n - D) / D;
    for (int b = 0; b < nfull; ++b) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        compute(st[d]);
        issue(st[d], kstep((b + 1) * D + d));
      }
    }
    const int done = (nfull + 1) * D, r = n - done;  // 0 <= r < D steps left after this batch
#pragma unroll
    for (int d = 0; d < D; ++d) {
      compute(st[d]);
      if (d < r) issue(st[d], kstep(done + d));
    }
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (d < r) compute(st[d]);
  } else {
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (d < n) issue(st[d], kstep(d));
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (d < n) compute(st[d]);
  }

  if constexpr (MT == 1) {
    if (wave == 0) epi_load<EPI, !norm_helper<MT, NW, EPI>(), JT>(a, t, 0, in1);
  }

  if constexpr (MT == 1) {
    // fixed-order sum of the waves' tiles
    if constexpr (NW > 1) {
      for (int m0 = 0; m0 < MT; m0 += RCH) {
  #pragma unroll
        for (int c = 0; c < RCH; ++c)
          if (m0 + c < MT)
  #pragma unroll
            for (int j = 0; j < JT; ++j) red[wave][c * JT + j][lane] = acc[m0 + c][j];
        __syncthreads();
        if (wave == 0) {
  #pragma unroll
          for (int c = 0; c < RCH; ++c)
            if (m0 + c < MT)
  #pragma unroll
              for (int j = 0; j < JT; ++j) {
                floatx4 v = red[0][c * JT + j][lane];
  #pragma unroll
                for (int w = 1; w < NW; ++w) v += red[w][c * JT + j][lane];
                acc[m0 + c][j] = v;
              }
        }
        __syncthreads();
      }
      if (wave != 0) return;
    }

    if (a.splits > 1) {
      // publish this split's tile; the last split to arrive sums all of them
      // (the tile's partials: [splits][TF] floats, lane l's 4 values at 4 l)
      const __amdgpu_buffer_rsrc_t part =
          coherent_region(a.partial + (size_t)t * a.splits * TF, (uint32_t)(a.splits * TF * 4));
  #pragma unroll
      for (int mt = 0; mt < MT; ++mt)
  #pragma unroll
        for (int j = 0; j < JT; ++j)
          store_coherent4(part, (uint32_t)((s * TF + (mt * JT + j) * 256 + lane * 4) * 4), acc[mt][j]);
      drain_stores();
      int old = 0;
      if (lane == 0) old = counter_add(&a.counters[t], 1);
      old = __shfl(old, 0);
      if (old != a.splits - 1) return;
  #pragma unroll
      for (int mt = 0; mt < MT; ++mt)
  #pragma unroll
        for (int j = 0; j < JT; ++j) acc[mt][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      for (int sp0 = 0; sp0 < a.splits; sp0 += 2) {
        // two splits' tiles in flight, summed in split order
        floatx4 pv[2][MT][JT];
  #pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int sp = sp0 + u < a.splits ? sp0 + u : sp0;
  #pragma unroll
          for (int mt = 0; mt < MT; ++mt)
  #pragma unroll
            for (int j = 0; j < JT; ++j)
              pv[u][mt][j] = load_coherent4(part, (uint32_t)((sp * TF + (mt * JT + j) * 256 + lane * 4) * 4));
        }
  #pragma unroll
        for (int u = 0; u < 2; ++u)
          if (sp0 + u < a.splits)
  #pragma unroll
            for (int mt = 0; mt < MT; ++mt)
  #pragma unroll
              for (int j = 0; j < JT; ++j) acc[mt][j] += pv[u][mt][j];
      }
      if (lane == 0) counter_reset(&a.counters[t]);
    }

    epilogue_tile<EPI, JT, true>(a, t, 0, acc[0], scr_all, in1,
                                 norm_helper<MT, NW, EPI>() ? norm_sh : nullptr);
  } else {
    // Several row tiles: row tile mt belongs to wave mt % NW, which sums it
    // over the waves (in wave order, as above) and finishes it, so that the
    // row tiles' hand-offs and epilogues run on all waves at once instead of
    // one after another on wave 0.
    auto mine = [&](int mt) { return mt % NW == wave; };
#pragma unroll
    for (int m0 = 0; m0 < MT; m0 += RCH) {
#pragma unroll
      for (int c = 0; c < RCH; ++c)
        if (m0 + c < MT)
#pragma unroll
          for (int j = 0; j < JT; ++j) red[wave][c * JT + j][lane] = acc[m0 + c][j];
      __syncthreads();
#pragma unroll
      for (int c = 0; c < RCH; ++c)
        if (m0 + c < MT && mine(m0 + c))
#pragma unroll
          for (int j = 0; j < JT; ++j) {
            floatx4 v = red[0][c * JT + j][lane];
#pragma unroll
            for (int w = 1; w < NW; ++w) v += red[w][c * JT + j][lane];
            acc[m0 + c][j] = v;
          }
      __syncthreads();
    }
    if (a.splits > 1) {
      // each wave publishes its row tiles of this split's tile; the
      // workgroup arrives once; the last split to arrive sums all of them
      // in split order, each wave its own row tiles
      const __amdgpu_buffer_rsrc_t part =
          coherent_region(a.partial + (size_t)t * a.splits * TF, (uint32_t)(a.splits * TF * 4));
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        if (mine(mt))
#pragma unroll
          for (int j = 0; j < JT; ++j)
            store_coherent4(part, (uint32_t)((s * TF + (mt * JT + j) * 256 + lane * 4) * 4), acc[mt][j]);
      drain_stores();
      __syncthreads();
      if (threadIdx.x == 0) last_sh = counter_add(&a.counters[t], 1) == a.splits - 1;
      __syncthreads();
      if (!last_sh) return;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        if (!mine(mt)) continue;
#pragma unroll
        for (int j = 0; j < JT; ++j) acc[mt][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        for (int sp0 = 0; sp0 < a.splits; sp0 += 2) {
          floatx4 pv[2][JT];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int sp = sp0 + u < a.splits ? sp0 + u : sp0;
#pragma unroll
            for (int j = 0; j < JT; ++j)
              pv[u][j] = load_coherent4(part, (uint32_t)((sp * TF + (mt * JT + j) * 256 + lane * 4) * 4));
          }
#pragma unroll
          for (int u = 0; u < 2; ++u)
            if (sp0 + u < a.splits)
#pragma unroll
              for (int j = 0; j < JT; ++j) acc[mt][j] += pv[u][j];
        }
      }
      if (threadIdx.x == 0) counter_reset(&a.counters[t]);
    }
    epilogue_rows<MT, EPI, JT>(a, t, acc, scr_all + wave * 16 * kScr, wave, NW);
  }
}

// ---------------------------------------------------------------------------
// Many row tiles: the activation shared through LDS
// ---------------------------------------------------------------------------
// With several row tiles a k-step of a 64-column tile is 2 MT JT MFMAs
// against JT weight fragments and 2 MT activation fragments: from 3 row
// tiles on the activation bytes outnumber the weight bytes, and a wave that
// kept both in flight for an HBM round trip would run out of registers. Here a workgroup owns NW
// adjacent 64-column tiles, one per compute wave, and one split of K. One
// more wave copies each k-step of the activation image (its 2 MT fragments
// are contiguous) into a ring of R LDS slots with direct global-to-LDS
// loads, P k-steps ahead of the compute waves, which read their operands
// from there: the image crosses L2 once per NW tiles instead of once per
// tile, and the compute waves keep only weights in flight (D k-steps). One
// barrier per k-step passes the slots between the loader and the compute
// waves. With splits of K each split writes its partial of the tile and
// gemm_epi_kernel sums them and runs the epilogues.
template <int MT>
__host__ __device__ constexpr int rows_depth() {  // weight k-steps in flight per compute wave
  return MT >= 9 ? 3 : (MT >= 5 ? 6 : 4);
}
// Up to 3 row tiles two workgroups share a compute unit (their LDS rings fit
// together): 10 waves, so up to 3 on a SIMD, 168 VGPRs each at most.
template <int MT>
__host__ __device__ constexpr int rows_waves_per_simd() {
  return MT <= 3 ? 3 : 1;
}
// Activation k-steps in flight: the loader waits on its own load counter
// (at most 63 loads outstanding) for the oldest, one 1 KB load per fragment.
template <int MT>
__host__ __device__ constexpr int rows_ahead() {
  return 63 / (2 * MT) + 1 < 8 ? 63 / (2 * MT) + 1 : 8;
}


template <int MT, int NW, int EPI>
__global__ __launch_bounds__(64 * (NW + 1), rows_waves_per_simd<MT>()) void gemm_rows_kernel(GemmArgs a) {
  constexpr int JT = 4;
  constexpr int D = rows_depth<MT>();
  constexpr int P = rows_ahead<MT>();
  constexpr int R = P + 1;    // LDS slots: a slot is refilled one barrier after its last read
  constexpr int AF = 2 * MT;  // activation fragments of a k-step: hi and lo of each row tile
  constexpr int TF = MT * JT * 256;
  __shared__ __attribute__((aligned(16))) u32x4 act_sh[R][AF][kWave];
  __shared__ __attribute__((aligned(16))) float scr_all[NW * 16 * kScr];
  __shared__ float2 norm_sh[MT * 16];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tw = blockIdx.x / a.splits, s = blockIdx.x - tw * a.splits;
  const int KS = a.K >> 5;
  const int kb = (int)((int64_t)KS * s / a.splits), ke = (int)((int64_t)KS * (s + 1) / a.splits);
  const int n = ke - kb;
  // k-steps from a point rotated by the workgroup's tiles (fixed per tile:
  // sums stay bit-reproducible), so that concurrent workgroups read different
  // k-steps of the shared image
  const int rot = n > 0 ? (int)((int64_t)n * (tw & 15) / 16) : 0;
  auto kstep = [&](int i) {
    const int x = i + rot;
    return kb + (x >= n ? x - n : x);
  };

  if (wave == NW) {
    // the loader: k-step i goes to slot i % R, issued after barrier i - P
    // (which the compute waves pass only once done with step i - P - 1, the
    // slot's previous content) and complete before barrier i
    const uint16_t* src = a.a_img + lane * 8;
    auto fetch = [&](int i, int slot) {
      const uint16_t* p = src + (size_t)kstep(i) * AF * 512;
#pragma unroll
      for (int f = 0; f < AF; ++f)
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(p + f * 512),
                                         (__attribute__((address_space(3))) void*)&act_sh[slot][f][0], 16, 0,
                                         0);
    };
#pragma unroll
    for (int p = 0; p < P; ++p)
      if (p < n) fetch(p, p);
    int slot_in = P % R;
    for (int i = 0; i < n; ++i) {
      // steps i + 1 .. i + P - 1 may stay in flight
      if (i + P <= n) wait_vmcnt<(P - 1) * AF>();
      else wait_vmcnt<0>();
      lds_barrier();
      if (i + P < n) {
        fetch(i + P, slot_in);
        slot_in = slot_in + 1 == R ? 0 : slot_in + 1;
      }
    }
    return;
  }

  // the pre-norm's (mu, r) of every row, merged once before the k-loop (the
  // summaries' registers are free then) and left in LDS for the epilogues;
  // barrier 0 below orders the writes before any read
  if constexpr (has_norm<EPI>()) {
    for (int mt = wave; mt < MT; mt += NW) {
      EpiIn nin;
      stats_load(a, mt, nin);
      float mu, rs;
      norm_finish(a, nin, mu, rs);
      if (lane < 16) norm_sh[16 * mt + lane] = make_float2(mu, rs);
    }
  }

  const int t = tw * NW + wave;
  const int tc = t < a.n_tiles ? t : a.n_tiles - 1;  // a wave past the last tile streams a valid one
  const uint16_t* wp[JT];
#pragma unroll
  for (int j = 0; j < JT; ++j) wp[j] = weight_frag<JT>(a, tc, j, lane);
  const size_t kstr = __builtin_amdgcn_readfirstlane(weight_kstride(a, tc));

  floatx4 acc[MT][JT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < JT; ++j) acc[mt][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  bf16x8 w[D][JT];
  auto issue = [&](bf16x8(&x)[JT], int i) {
    const int k = kstep(i);
#pragma unroll
    for (int j = 0; j < JT; ++j) x[j] = load_nt(wp[j] + (size_t)k * kstr);
  };
  // Row tile by row tile: the hi products of the JT sub-tiles, then their lo
  // products (4 MFMAs apart from the hi one they accumulate onto), while the
  // next row tile's two fragments are read from LDS. The order is pinned:
  // left to itself the scheduler ran every hi product first, which keeps
  // all MT lo fragments live, and with the 144 accumulator registers of 9
  // row tiles it then read each hi fragment into one register and waited
  // for it, an LDS round trip per row tile.
  auto compute = [&](const bf16x8(&x)[JT], int slot) {
    bf16x8 ah[2], al[2];
    ah[0] = __builtin_bit_cast(bf16x8, act_sh[slot][0][lane]);
    al[0] = __builtin_bit_cast(bf16x8, act_sh[slot][1][lane]);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (mt + 1 < MT) {
        ah[(mt + 1) & 1] = __builtin_bit_cast(bf16x8, act_sh[slot][2 * mt + 2][lane]);
        al[(mt + 1) & 1] = __builtin_bit_cast(bf16x8, act_sh[slot][2 * mt + 3][lane]);
      }
#pragma unroll
      for (int j = 0; j < JT; ++j) acc[mt][j] = mfma16x16x32(x[j], ah[mt & 1], acc[mt][j]);
#pragma unroll
      for (int j = 0; j < JT; ++j) acc[mt][j] = mfma16x16x32(x[j], al[mt & 1], acc[mt][j]);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // row tile 0's fragments
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (mt + 1 < MT) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // the next row tile's
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * JT, 0);              // this row tile's MFMAs
    }
  };
  // D k-steps of weights in flight; as in gemm_kernel the steady-state loop
  // runs only over batches whose D refills are all real (a branch in it
  // would make every batch wait for all its loads). Each k-step starts at a
  // barrier, after which its activation is in its slot.
  int slot = 0;
  auto step = [&](const bf16x8(&x)[JT]) {
    lds_barrier();
    compute(x, slot);
    slot = slot + 1 == R ? 0 : slot + 1;
  };
  if (n >= D) {
#pragma unroll
    for (int d = 0; d < D; ++d) issue(w[d], d);
    const int nfull = (n - D) / D;
    for (int b = 0; b < nfull; ++b) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        step(w[d]);
        issue(w[d], (b + 1) * D + d);
      }
    }
    const int done = (nfull + 1) * D, r = n - done;  // 0 <= r < D
#pragma unroll
    for (int d = 0; d < D; ++d) {
      step(w[d]);
      if (d < r) issue(w[d], done + d);
    }
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (d < r) step(w[d]);
  } else {
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (d < n) issue(w[d], d);
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (d < n) step(w[d]);
  }
  if (t >= a.n_tiles) return;

  if (a.splits > 1) {
    // this split's partial of the tile (all row tiles); gemm_epi_kernel sums
    // the splits in split order and runs the epilogue
    float* part = a.partial + ((size_t)t * a.splits + s) * TF + lane * 4;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int j = 0; j < JT; ++j) *reinterpret_cast<floatx4*>(part + (mt * JT + j) * 256) = acc[mt][j];
    return;
  }
  epilogue_rows<MT, EPI, JT, has_norm<EPI>()>(a, t, acc, scr_all + wave * 16 * kScr, 0, 1, norm_sh);
}

// The split sum and epilogue of gemm_rows_kernel with splits > 1, a kernel
// of their own: one wave per (64-column tile, row tile) sums that row
// tile's partials in split order and runs its epilogue, so that no wave sums
// and finishes all row tiles of its tile in series, and narrow GEMMs can
// take many splits of K (enough waves for the MFMA work of 144 rows).
template <int MT, int EPI>
__global__ __launch_bounds__(256) void gemm_epi_kernel(GemmArgs a) {
  constexpr int JT = 4;
  constexpr int TF = MT * JT * 256;
  __shared__ __attribute__((aligned(16))) float scr_all[4 * 16 * kScr];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int u = blockIdx.x * 4 + wave;
  const int t = u / MT, mt = u - t * MT;
  if (t >= a.n_tiles) return;
  const float* part = a.partial + (size_t)t * a.splits * TF + (mt * JT) * 256 + lane * 4;
  floatx4 acc[JT];
#pragma unroll
  for (int j = 0; j < JT; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
  constexpr int SB = 4;  // splits' partials in flight
  for (int sp0 = 0; sp0 < a.splits; sp0 += SB) {
    floatx4 pv[SB][JT];
#pragma unroll
    for (int q = 0; q < SB; ++q) {
      const int sp = sp0 + q < a.splits ? sp0 + q : sp0;
#pragma unroll
      for (int j = 0; j < JT; ++j)
        pv[q][j] = *reinterpret_cast<const floatx4*>(part + (size_t)sp * TF + j * 256);
    }
#pragma unroll
    for (int q = 0; q < SB; ++q)
      if (sp0 + q < a.splits)
#pragma unroll
        for (int j = 0; j < JT; ++j) acc[j] += pv[q][j];
  }
  EpiIn none;
  epilogue_tile<EPI, JT, false>(a, t, mt, acc, scr_all + wave * 16 * kScr, none);
}

template <int MT, int NW, int EPI>
hipError_t launch_rows(const GemmArgs& a, hipStream_t s, LaunchEvents ev) {
  const int wgs = (a.n_tiles + NW - 1) / NW;
  const bool two = a.splits > 1;
  hipExtLaunchKernelGGL((gemm_rows_kernel<MT, NW, EPI>), dim3(wgs * a.splits), dim3(64 * (NW + 1)), 0, s,
                        ev.start, two ? nullptr : ev.stop, 0, a);
  if (two) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipExtLaunchKernelGGL((gemm_epi_kernel<MT, EPI>), dim3((a.n_tiles * MT + 3) / 4), dim3(256), 0, s, nullptr,
                          ev.stop, 0, a);
  }
  return hipGetLastError();
}

template <int MT, int NW, int EPI, int JT>
hipError_t launch_cfg(const GemmArgs& a, hipStream_t s, LaunchEvents ev) {
  hipExtLaunchKernelGGL((gemm_kernel<MT, NW, EPI, JT>), dim3(a.n_tiles * a.splits),
                        dim3(64 * block_waves<MT, NW, EPI>()), 0, s, ev.start, ev.stop, 0, a);
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_epi(const GemmArgs& a, hipStream_t s, LaunchEvents ev) {
  if (a.jt == 8) {  // 128-column tiles: the SwiGLU FFN up projection (up to 3
                    // row tiles, 2 waves) and the LM head (one row tile, 4 waves)
    if constexpr (EPI == EPI_SWIGLU) {
      if (a.waves != 2) return hipErrorInvalidValue;
      switch (a.MT) {
        case 1: return launch_cfg<1, 2, EPI, 8>(a, s, ev);
        case 2: return launch_cfg<2, 2, EPI, 8>(a, s, ev);
        case 3: return launch_cfg<3, 2, EPI, 8>(a, s, ev);
        default: return hipErrorInvalidValue;
      }
    }
    if constexpr (EPI == EPI_HEAD) {
      if (a.waves != 4 || a.MT != 1) return hipErrorInvalidValue;
      return launch_cfg<1, 4, EPI, 8>(a, s, ev);
    }
    return hipErrorInvalidValue;
  }
  if constexpr (EPI == EPI_QKV) {
    // one row tile, 32-column tiles (16 rotary pairs of a head), 8 waves, whole K
    if (a.jt == 2) {
      if (a.MT != 1 || a.waves != 8 || a.wg_tiles != 1) return hipErrorInvalidValue;
      return launch_cfg<1, 8, EPI, 2>(a, s, ev);
    }
  }
  if (a.jt != 4) return hipErrorInvalidValue;
  if (a.wg_tiles > 1) {  // tiles per workgroup, the activation shared through LDS
    if (a.wg_tiles != 4) return hipErrorInvalidValue;
    switch (a.MT) {
      case 2: return launch_rows<2, 4, EPI>(a, s, ev);
      case 3: return launch_rows<3, 4, EPI>(a, s, ev);
      case 5: return launch_rows<5, 4, EPI>(a, s, ev);
      case 9: return launch_rows<9, 4, EPI>(a, s, ev);
      default: return hipErrorInvalidValue;
    }
  }
  switch (a.MT) {
    case 1: return a.waves == 8 ? launch_cfg<1, 8, EPI, 4>(a, s, ev) : launch_cfg<1, 4, EPI, 4>(a, s, ev);
    case 2: return launch_cfg<2, 4, EPI, 4>(a, s, ev);
    case 3: return launch_cfg<3, 4, EPI, 4>(a, s, ev);
    case 5: return launch_cfg<5, 4, EPI, 4>(a, s, ev);
    case 9: return launch_cfg<9, 4, EPI, 4>(a, s, ev);
    default: return hipErrorInvalidValue;
  }
}

// Row-major [rows][K] -> k-step-major fragments: fragment (G, ks), G < NG =
// rows / 16, at (ks * NG + G) * 512 elements holds rows 16G..16G+15, columns
// 32ks..32ks+31, lane l taking row 16G + l%16 and columns 32ks + 8(l/16) .. +8
// (16 bytes); dst is written sequentially.
__global__ __launch_bounds__(256) void repack_kernel(const uint16_t* __restrict__ src,
                                                     uint16_t* __restrict__ dst, int64_t rows,
                                                     int32_t K) {
  const int64_t NG = rows >> 4;
  const int64_t total = NG * (K >> 5) * 64;  // 16-byte lane chunks
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t lanes = i & 63, frag = i >> 6;
    const int64_t ks = frag / NG, G = frag - ks * NG;
    const int64_t row = 16 * G + (lanes & 15), col = 32 * ks + 8 * (lanes >> 4);
    *reinterpret_cast<u32x4*>(dst + i * 8) = *reinterpret_cast<const u32x4*>(src + row * K + col);
  }
}

// c[n] = sum_k W[n][k] g[k] and e[n] = sum_k W[n][k] b[k] of a row-major bf16
// matrix; one wave per row, fp64 accumulation.
__global__ __launch_bounds__(256) void colsum_kernel(const uint16_t* w, int64_t rows, int32_t K,
                                                     const uint16_t* g, const uint16_t* b, float* c,
                                                     float* e) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  double sg = 0.0, sb = 0.0;
  for (int k = lane; k < K; k += 64) {
    const double wv = bf2f(w[row * K + k]);
    sg += wv * bf2f(g[k]);
    if (b) sb += wv * bf2f(b[k]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    sg += __shfl_xor(sg, o);
    sb += __shfl_xor(sb, o);
  }
  if (lane == 0) {
    c[row] = (float)sg;
    if (e) e[row] = (float)sb;
  }
}

}  // namespace

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s, LaunchEvents ev) {
  if (a.n_tiles < 1 || a.splits < 1 || a.K % 32 || a.M < 1 || a.M > 16 * a.MT) return hipErrorInvalidValue;
  if (a.splits > 1 && (!a.partial || !a.counters)) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(a, s, ev);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, s, ev);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(a, s, ev);
    case EPI_RELU: return launch_epi<EPI_RELU>(a, s, ev);
    case EPI_HEAD: return launch_epi<EPI_HEAD>(a, s, ev);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_repack(const uint16_t* src, uint16_t* dst, int64_t rows, int32_t K, hipStream_t s) {
  if (rows % 16 || K % 32) return hipErrorInvalidValue;
  const int64_t total = (rows >> 4) * (K >> 5) * 64;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(repack_kernel, dim3((unsigned)blocks), dim3(256), 0, s, src, dst, rows, K);
  return hipGetLastError();
}

hipError_t launch_colsum(const uint16_t* w, int64_t rows, int32_t K, const uint16_t* g,
                         const uint16_t* b, float* c, float* e, hipStream_t s) {
  hipLaunchKernelGGL(colsum_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, w, rows, K,
                     g, b, c, e);
  return hipGetLastError();
}

}  // namespace msd
