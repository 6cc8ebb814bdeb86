// Skinny weight-streaming GEMM for the verification pass: Y = A W^T with
// A = the block's rows (M = batch * n_slots <= 144, fp32 activations) and W a
// bf16 weight matrix [N][K] read exactly once. This is where the verify step
// spends its bytes: every projection of every layer plus the two LM-head
// passes.
//
// Mapping (gfx950, wave64, MFMA 16x16x32 bf16 -> fp32):
//  * a workgroup (4 waves) owns a 64-column output tile and a contiguous
//    slice of K (split-K over `splits` workgroups per tile);
//  * inside the workgroup the slice is cut in 4 k-ranges, one per wave; each
//    wave holds the full 64 columns (4 MFMA column tiles) for MT row tiles;
//  * weights are stored fragment-major (one 1 KB MFMA B operand after the
//    other along K, per 16-row group) and streamed straight from HBM into
//    the MFMA with 16-byte loads, two batches of U k-steps in flight per
//    wave; the small A operand is L2-resident;
//  * the pre-norm of the block (RMSNorm or LayerNorm) is applied while A is
//    loaded, from per-row statistics the producing kernel left behind, and A
//    enters the MFMA as bf16 hi + lo parts (two MFMAs per weight tile, about
//    16-bit activations) while that costs nothing against the weight stream;
//  * the 4 waves' tiles are summed in LDS in a fixed order; with split-K each
//    workgroup publishes its tile with coherent stores and the last to arrive
//    sums all splits in split order and runs the epilogue. No floating-point
//    atomics: results are bit-reproducible.
#include "kernels.h"

namespace msd {
namespace {

constexpr int kRedStride = kTileN + 4;  // LDS row stride (floats), breaks bank aliasing

// Weights live in the fragment-major layout (see repack_kernel): the 16-row
// group G of a matrix is a contiguous run of K/32 fragments of 1 KB, fragment
// ks holding rows 16G..16G+15 x columns 32ks..32ks+31 in MFMA B-operand order
// (lane l: row 16G + l%16, columns 32ks + 8(l/16) .. +8). A wave's four
// column tiles are therefore four sequential HBM streams.
// Returns the lane's pointer into fragment 0 of the group feeding sub-tile j.
__device__ __forceinline__ const uint16_t* weight_frag(const GemmArgs& a, int t, int j, int lane) {
  const size_t run = (size_t)(a.K >> 5) * 512;  // elements per 16-row group
  const uint16_t* base;
  int grp;
  if (a.map == MAP_QKV) {
    const int hd = a.head_dim, half = hd >> 1, tph = hd >> 6;
    const int hh = t / tph, gi = t - hh * tph;
    const int c0 = j < 2 ? gi * 32 + 16 * j : half + gi * 32 + 16 * (j - 2);
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
  } else if (a.map == MAP_GATEUP) {
    base = j < 2 ? a.w0 : a.w1;
    grp = 2 * t + (j & 1);
  } else {
    base = a.w0;
    grp = 4 * t + j;
    const int last = (a.N >> 4) - 1;  // padding columns re-read a valid group; output masked
    if (grp > last) grp = last;
  }
  return base + (size_t)grp * run + lane * 8;
}

// ---------------------------------------------------------------------------
// epilogues: the reduced tile is red[m * kRedStride + c], m < M, c < 64
// ---------------------------------------------------------------------------

// x += y (+ bias); also the (mean, M2) of the 64 updated values of every row,
// from which the next pre-norm is built (Chan et al. pairwise combination).
__device__ void epi_resid(const GemmArgs& a, int t, const float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int n = t * kTileN + lane;
  const bool valid = n < a.N;
  for (int m = wave; m < a.M; m += nw) {
    float v = 0.0f;
    if (valid) {
      v = red[m * kRedStride + lane];
      if (a.b0) v += bf2f(a.b0[n]);
      float* xp = a.x + (size_t)m * a.N + n;
      v += *xp;
      *xp = v;
    }
    if (a.stats_out) {
      const float cnt = (float)min(kTileN, a.N - t * kTileN);
      const float mean = wave_sum(valid ? v : 0.0f) / cnt;
      const float dv = valid ? v - mean : 0.0f;
      const float m2 = wave_sum(dv * dv);
      if (lane == 0) a.stats_out[(size_t)t * a.M + m] = make_float2(mean, m2);
    }
  }
}

__device__ void epi_swiglu(const GemmArgs& a, int t, const float* red) {
  const int F = a.N >> 1;
  for (int i = threadIdx.x; i < a.M * 32; i += blockDim.x) {
    const int m = i >> 5, c = i & 31;
    const float g = red[m * kRedStride + c], u = red[m * kRedStride + 32 + c];
    a.out_f32[(size_t)m * F + t * 32 + c] = silu(g) * u;
  }
}

__device__ void epi_relu(const GemmArgs& a, int t, const float* red) {
  for (int i = threadIdx.x; i < a.M * kTileN; i += blockDim.x) {
    const int m = i / kTileN, c = i - m * kTileN, n = t * kTileN + c;
    if (n >= a.N) continue;
    float v = red[m * kRedStride + c];
    if (a.b0) v += bf2f(a.b0[n]);
    a.out_f32[(size_t)m * a.N + n] = fmaxf(v, 0.0f);
  }
}

__device__ void epi_qkv(const GemmArgs& a, int t, const float* red) {
  const int hd = a.head_dim, half = hd >> 1, tph = hd >> 6;
  const int H = a.n_heads, Hk = a.n_kv_heads;
  const int hh = t / tph, gi = t - hh * tph;
  const int which = hh < H ? 0 : (hh < H + Hk ? 1 : 2);
  const int hloc = hh - (which == 0 ? 0 : (which == 1 ? H : H + Hk));
  const uint16_t* bias = which == 0 ? a.b0 : (which == 1 ? a.b1 : a.b2);
  for (int i = threadIdx.x; i < a.M * 32; i += blockDim.x) {
    const int m = i >> 5, p = i & 31;
    const int col_lo = gi * 32 + p, col_hi = half + gi * 32 + p;
    float lo = red[m * kRedStride + p], hi = red[m * kRedStride + 32 + p];
    if (bias) {
      lo += bf2f(bias[hloc * hd + col_lo]);
      hi += bf2f(bias[hloc * hd + col_hi]);
    }
    const int b = m / a.n_slots, slot = m - b * a.n_slots;
    const int L = a.len[b];
    if (L + a.n_slots > a.capacity) {
      if (p == 0) atomicOr(a.status, 1u);
      continue;
    }
    const int pos = L + a.depth[slot];
    if (which < 2 && a.rope) {
      const float2 cs = a.rope[(size_t)pos * half + col_lo];
      const float rlo = lo * cs.x - hi * cs.y;
      const float rhi = hi * cs.x + lo * cs.y;
      lo = rlo;
      hi = rhi;
    }
    if (which == 0) {
      float* q = a.out_f32 + ((size_t)m * H + hloc) * hd;
      q[col_lo] = lo;
      q[col_hi] = hi;
    } else {
      uint16_t* cache = which == 1 ? a.k_cache : a.v_cache;
      uint16_t* row = cache + (((size_t)b * Hk + hloc) * a.capacity + L + slot) * hd;
      row[col_lo] = f2bf(lo);
      row[col_hi] = f2bf(hi);
    }
  }
}

// Per row of the tile: logits out, (max, sum exp), top-kappa rank keys.
__device__ void epi_head(const GemmArgs& a, int t, const float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int n = t * kTileN + lane;
  const bool valid = n < a.N;
  for (int m = wave; m < a.M; m += nw) {
    const float v = red[m * kRedStride + lane];
    if (a.logits && valid) a.logits[(size_t)m * a.N + n] = v;
    const float mx = wave_max(valid ? v : -INFINITY);
    const float se = wave_sum(valid ? expf(v - mx) : 0.0f);
    if (lane == 0) a.tile_ms[(size_t)t * a.M + m] = make_float2(mx, se);
    uint64_t key = valid ? rank_key(v, n) : 0ull;
    uint64_t* top = a.tile_top + ((size_t)t * a.M + m) * a.kappa;
    for (int r = 0; r < a.kappa; ++r) {
      const uint64_t best = wave_max_u64(key);
      if (key == best) key = 0ull;
      if (lane == 0) top[r] = best;
    }
  }
}

// Per-row (mu, scale) of the fused pre-norm from the producer's per-segment
// (mean, M2) pairs: mean = average of segment means; M2 = sum M2_t +
// cnt * sum (mean_t - mean)^2. RMSNorm uses E[x^2] = M2/K + mean^2.
__device__ void norm_rows(const GemmArgs& a, float2* rowstat) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int T = a.a_stats_tiles;
  const float cnt = (float)a.K / (float)T;
  for (int m = wave; m < a.M; m += nw) {
    // up to 4 segments per lane, loaded together (T <= 256)
    float2 st[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int t = lane + 64 * q;
      st[q] = a.a_stats[(size_t)(t < T ? t : 0) * a.M + m];
    }
    float sm = 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q) sm += lane + 64 * q < T ? st[q].x : 0.0f;
    const float mean = wave_sum(sm) / (float)T;
    float m2 = 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float d = st[q].x - mean;
      m2 += lane + 64 * q < T ? st[q].y + cnt * d * d : 0.0f;
    }
    m2 = wave_sum(m2);
    float mu, sc;
    if (a.a_norm == 2) {
      mu = mean;
      sc = 1.0f / sqrtf(m2 / (float)a.K + a.a_eps);
    } else {
      mu = 0.0f;
      sc = 1.0f / sqrtf(m2 / (float)a.K + mean * mean + a.a_eps);
    }
    if (lane == 0) rowstat[m] = make_float2(mu, sc);
  }
}

// Raw A-operand data of one MFMA k-step for one row tile: 8 fp32 values of
// the row, and for a fused pre-norm the 8 matching gains (and shifts).
struct ARaw {
  u32x4 x0, x1, g, b;
};

template <int MT, int U, int EPI, bool SPLIT, int NORM>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a) {
  __shared__ float red[MT * 16 * kRedStride];
  __shared__ float2 rowstat[MT * 16];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int t = blockIdx.x / a.splits, s = blockIdx.x - t * a.splits;
  const int KS = a.K >> 5;
  const int ks_b = (int)((int64_t)KS * s / a.splits);
  const int ks_e = (int)((int64_t)KS * (s + 1) / a.splits);
  const int nks = ks_e - ks_b;
  const int kb = ks_b + (nks * wave) / 4, ke = ks_b + (nks * (wave + 1)) / 4;

  const uint16_t* wp[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) wp[j] = weight_frag(a, t, j, lane);
  // rows past M read row 0 (always valid) and are zeroed after the load:
  // no divergent branch around loads, so the compiler keeps them in flight
  const float* ap[MT];
  float amask[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + r16;
    amask[mt] = m < a.M ? 1.0f : 0.0f;
    ap[mt] = a.A + (size_t)(m < a.M ? m : 0) * a.K + g * 8;
  }
  const uint16_t* gp = NORM ? a.a_g + g * 8 : nullptr;
  const uint16_t* bp = NORM == 2 ? a.a_b + g * 8 : nullptr;

  bf16x8 w0[U][4], w1[U][4];
  auto issue_w = [&](bf16x8 (&w)[U][4], int ks) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < 4; ++j) w[u][j] = load16(wp[j] + (size_t)(ks + u) * 512);
  };
  auto issue_a = [&](ARaw (&r)[U][MT], int ks) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const size_t ko = (size_t)(ks + u) * 32;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        r[u][mt].x0 = *reinterpret_cast<const u32x4*>(ap[mt] + ko);
        r[u][mt].x1 = *reinterpret_cast<const u32x4*>(ap[mt] + ko + 4);
      }
      if constexpr (NORM != 0) {
        const u32x4 gv = *reinterpret_cast<const u32x4*>(gp + ko);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) r[u][mt].g = gv;
      }
      if constexpr (NORM == 2) {
        const u32x4 bv = *reinterpret_cast<const u32x4*>(bp + ko);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) r[u][mt].b = bv;
      }
    }
  };

  // the weight stream of batch 0 goes out before the pre-norm statistics
  const int nb = (ke - kb) / U;
  if (nb > 0) issue_w(w0, kb);

  if constexpr (NORM != 0) {
    norm_rows(a, rowstat);
    lds_barrier();
  }
  float mu[MT], sc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    mu[mt] = 0.0f;
    sc[mt] = amask[mt];
    if constexpr (NORM != 0) {
      const float2 st = rowstat[(mt * 16 + r16) < a.M ? mt * 16 + r16 : 0];
      mu[mt] = st.x;
      sc[mt] = st.y * amask[mt];
    }
  }

  floatx4 acc[MT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[mt][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // A operand = (x - mu) * sc * g + b (pre-norm) or x * mask, then split into
  // bf16 hi + lo (two MFMAs per weight tile) or rounded once.
  auto compute = [&](const bf16x8 (&w)[U][4], const ARaw (&r)[U][MT]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        float v[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          v[i] = __uint_as_float(r[u][mt].x0[i]);
          v[4 + i] = __uint_as_float(r[u][mt].x1[i]);
        }
        if constexpr (NORM != 0) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t gw = r[u][mt].g[i];
            v[2 * i] = (v[2 * i] - mu[mt]) * sc[mt] * bf_lo(gw);
            v[2 * i + 1] = (v[2 * i + 1] - mu[mt]) * sc[mt] * bf_hi(gw);
            if constexpr (NORM == 2) {
              const uint32_t bw = r[u][mt].b[i];
              v[2 * i] += bf_lo(bw) * amask[mt];
              v[2 * i + 1] += bf_hi(bw) * amask[mt];
            }
          }
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) v[i] *= amask[mt];
        }
        bf16x8 hi, lo;
        if constexpr (SPLIT) split_vals(v, hi, lo);
        else hi = round_vals(v);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[mt][j] = mfma16x16x32(hi, w[u][j], acc[mt][j]);
          if constexpr (SPLIT) acc[mt][j] = mfma16x16x32(lo, w[u][j], acc[mt][j]);
        }
      }
  };

  // software pipeline: A of batch i, weights of batch i+1, then the MFMAs of
  // batch i; in-order completion lets the wait for A(i) leave W(i+1) in flight
  int i = 0;
  for (; i + 2 < nb; i += 2) {
    ARaw r[U][MT];
    issue_a(r, kb + i * U);
    issue_w(w1, kb + (i + 1) * U);
    compute(w0, r);
    issue_a(r, kb + (i + 1) * U);
    issue_w(w0, kb + (i + 2) * U);
    compute(w1, r);
  }
  if (nb - i == 2) {
    ARaw r[U][MT];
    issue_a(r, kb + i * U);
    issue_w(w1, kb + (i + 1) * U);
    compute(w0, r);
    issue_a(r, kb + (i + 1) * U);
    compute(w1, r);
  } else if (nb - i == 1) {
    ARaw r[U][MT];
    issue_a(r, kb + i * U);
    compute(w0, r);
  }
  // k-steps left over from whole batches, one batch-sized step at a time
  for (int ks = kb + nb * U; ks < ke; ++ks) {
    bf16x8 w[1][4];
#pragma unroll
    for (int j = 0; j < 4; ++j) w[0][j] = load16(wp[j] + (size_t)ks * 512);
    ARaw r[1][MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      r[0][mt].x0 = *reinterpret_cast<const u32x4*>(ap[mt] + (size_t)ks * 32);
      r[0][mt].x1 = *reinterpret_cast<const u32x4*>(ap[mt] + (size_t)ks * 32 + 4);
      if constexpr (NORM != 0) r[0][mt].g = *reinterpret_cast<const u32x4*>(gp + (size_t)ks * 32);
      if constexpr (NORM == 2) r[0][mt].b = *reinterpret_cast<const u32x4*>(bp + (size_t)ks * 32);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float v[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[q] = __uint_as_float(r[0][mt].x0[q]);
        v[4 + q] = __uint_as_float(r[0][mt].x1[q]);
      }
      if constexpr (NORM != 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[2 * q] = (v[2 * q] - mu[mt]) * sc[mt] * bf_lo(r[0][mt].g[q]);
          v[2 * q + 1] = (v[2 * q + 1] - mu[mt]) * sc[mt] * bf_hi(r[0][mt].g[q]);
          if constexpr (NORM == 2) {
            v[2 * q] += bf_lo(r[0][mt].b[q]) * amask[mt];
            v[2 * q + 1] += bf_hi(r[0][mt].b[q]) * amask[mt];
          }
        }
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] *= amask[mt];
      }
      bf16x8 hi, lo;
      if constexpr (SPLIT) split_vals(v, hi, lo);
      else hi = round_vals(v);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[mt][j] = mfma16x16x32(hi, w[0][j], acc[mt][j]);
        if constexpr (SPLIT) acc[mt][j] = mfma16x16x32(lo, w[0][j], acc[mt][j]);
      }
    }
  }

  // fixed-order sum of the 4 waves' tiles in LDS
  for (int w = 0; w < 4; ++w) {
    if (wave == w) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int idx = (mt * 16 + 4 * g + r) * kRedStride + 16 * j + r16;
            red[idx] = (w == 0 ? 0.0f : red[idx]) + acc[mt][j][r];
          }
    }
    __syncthreads();
  }

  if (a.splits > 1) {
    const size_t ld = (size_t)a.n_tiles * kTileN;
    float* dst = a.partial + (size_t)s * a.M * ld + (size_t)t * kTileN;
    for (int i = tid; i < a.M * kTileN; i += blockDim.x) {
      const int m = i / kTileN, c = i - m * kTileN;
      store_coherent(dst + (size_t)m * ld + c, red[m * kRedStride + c]);
    }
    drain_stores();
    __syncthreads();
    if (tid == 0) s_last = (counter_add(&a.counters[t], 1) == a.splits - 1);
    __syncthreads();
    if (!s_last) return;
    // splits summed in split order; 8 loads in flight per group (indices past
    // the last split read split 0 and are masked out)
    const float* src = a.partial + (size_t)t * kTileN;
    for (int i = tid; i < a.M * kTileN; i += blockDim.x) {
      const int m = i / kTileN, c = i - m * kTileN;
      const float* p = src + (size_t)m * ld + c;
      const size_t sstride = (size_t)a.M * ld;
      float v = 0.0f;
      for (int sp0 = 0; sp0 < a.splits; sp0 += 8) {
        float part[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int sp = sp0 + q < a.splits ? sp0 + q : 0;
          part[q] = load_coherent(p + sp * sstride);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) v += sp0 + q < a.splits ? part[q] : 0.0f;
      }
      red[m * kRedStride + c] = v;
    }
    if (tid == 0) counter_reset(&a.counters[t]);
    __syncthreads();
  }

  if constexpr (EPI == EPI_QKV) epi_qkv(a, t, red);
  else if constexpr (EPI == EPI_RESID) epi_resid(a, t, red);
  else if constexpr (EPI == EPI_SWIGLU) epi_swiglu(a, t, red);
  else if constexpr (EPI == EPI_RELU) epi_relu(a, t, red);
  else epi_head(a, t, red);
}

// Activations enter as bf16 hi + lo pairs (two MFMAs per weight tile) at
// every block size: a single bf16 rounding of the activations loses about
// three decimal digits per layer, which compounds over a deep target; at 144
// rows the doubled MFMA work still stays under the weight-stream time.
template <int MT, int EPI, int NORM>
hipError_t launch_mt(const GemmArgs& a, hipStream_t s) {
  constexpr int U = MT == 1 ? 4 : (MT <= 3 ? 2 : 1);
  constexpr bool SPLIT = true;
  hipLaunchKernelGGL((gemm_kernel<MT, U, EPI, SPLIT, NORM>), dim3(a.n_tiles * a.splits),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int EPI, int NORM>
hipError_t launch_epi(const GemmArgs& a, hipStream_t s) {
  const int mt = (a.M + 15) / 16;
  if (mt == 1) return launch_mt<1, EPI, NORM>(a, s);
  if (mt == 2) return launch_mt<2, EPI, NORM>(a, s);
  if (mt == 3) return launch_mt<3, EPI, NORM>(a, s);
  if (mt <= 9) return launch_mt<9, EPI, NORM>(a, s);
  return hipErrorInvalidValue;
}

template <int EPI>
hipError_t launch_norm_kind(const GemmArgs& a, hipStream_t s) {
  if (a.a_norm == 1) return launch_epi<EPI, 1>(a, s);
  if (a.a_norm == 2) return launch_epi<EPI, 2>(a, s);
  return launch_epi<EPI, 0>(a, s);
}

// Row-major [R][K] (src) -> fragment-major (dst), R % 16 == 0, K % 32 == 0:
// 16 bytes per thread, dst written sequentially.
__global__ void repack_kernel(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                              int64_t rows, int32_t K) {
  const int64_t ks_n = K >> 5;
  const int64_t n16 = rows * (int64_t)K / 8;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int lane = (int)(i & 63);
    const int64_t frag = i >> 6;
    const int64_t grp = frag / ks_n, ks = frag - grp * ks_n;
    const int64_t row = grp * 16 + (lane & 15);
    const int64_t col = ks * 32 + 8 * (lane >> 4);
    reinterpret_cast<u32x4*>(dst)[i] = *reinterpret_cast<const u32x4*>(src + row * K + col);
  }
}

}  // namespace

hipError_t launch_repack(const uint16_t* src, uint16_t* dst, int64_t rows, int32_t K,
                         hipStream_t s) {
  const int64_t n16 = rows * (int64_t)K / 8;
  int64_t grid = (n16 + 255) / 256;
  if (grid > 65536) grid = 65536;
  hipLaunchKernelGGL(repack_kernel, dim3((int)grid), dim3(256), 0, s, src, dst, rows, K);
  return hipGetLastError();
}

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_norm_kind<EPI_QKV>(a, s);
    case EPI_RESID: return launch_epi<EPI_RESID, 0>(a, s);
    case EPI_SWIGLU: return launch_norm_kind<EPI_SWIGLU>(a, s);
    case EPI_RELU: return launch_norm_kind<EPI_RELU>(a, s);
    case EPI_HEAD: return launch_norm_kind<EPI_HEAD>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace msd
