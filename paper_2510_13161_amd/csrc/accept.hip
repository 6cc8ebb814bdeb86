// Acceptance (the App. B operator: longest verified prefix of the draft
// block, then the next token) and the KV commit / rollback.
//
// One workgroup per sequence walks the block from the root. GREEDY reads the
// final head's argmax. The stochastic rules need the target law at the
// visited node, p = Softmax(z / T), over the whole vocabulary: its
// logsumexp and the inverse-CDF draw are workgroup reductions in fp64 over
// 1024 threads (contiguous id chunks per thread, chunk sums prefixed in id
// order). The
// sparse draft law q lives on <= 64 candidate ids, so the rejection residual
// r = normalise((r - q)^+) differs from a multiple f * p only on those ids:
// the kernel keeps f and the candidate values, never a dense vocab vector.
// With a workspace (AcceptArgs::stats) the vocabulary passes leave the walk:
// row_stats_kernel, a workgroup per (row, 1/kStatChunks of the vocabulary)
// over the whole device, stores each chunk's max of z / T and sum of
// exp(z / T - max) in fp64; the walk then takes the logsumexp from the
// chunk statistics, and an inverse-CDF draw picks its chunk from the chunk
// masses (corrected on the candidate ids) and scans that chunk only.
//
// Near-tie flags (optional): a decision that a logit error of tol_logit could
// flip marks the sequence. Bands: an argmax whose top-1 minus top-2 logit is
// below 2 tol; an accept test with |u - alpha| < 2 tol alpha / T (alpha moves
// by a factor exp(+-2 tol / T) when z_x and the normaliser each move by tol);
// an inverse-CDF draw with |u - c| < 4 tol min(c, 1 - c) at either edge c
// (cumulative fraction) of the chosen id's bin.
#include "kernels.h"

namespace msd {
namespace {

constexpr int kMaxCand = 64;
constexpr int kThreads = 1024;  // 16 waves: the fp64 vocabulary passes are latency-bound
constexpr int kStatChunks = kAcceptStatChunks;  // vocabulary chunks of the per-row statistics (one wave)

struct Shared {
  double red[kThreads];
  double red2[kThreads];
  double pre[kThreads + 1];
  double c_lo, c_hi;       // cumulative fractions at the edges of the drawn id's bin
  int cid[kMaxCand];       // candidate ids sorted ascending
  double rc[kMaxCand];     // residual mass at each sorted candidate
  double qc[kMaxCand];     // draft mass at each sorted candidate
  double pcand[kMaxCand];  // target probability p at each sorted candidate
  int tmp_id[kMaxCand];    // the node's candidate ids as given
  int tok[kMaxSlots];      // the sequence's block tokens
  float ua[kMaxSlots], us[kMaxSlots];  // its uniforms
  double wtot[kThreads / 64];  // per-wave totals of a block scan
  int n_c;
  int found;
  int result;
};

__device__ double block_reduce_max(double v, Shared& sh) {
  sh.red[threadIdx.x] = v;
  __syncthreads();
  for (int o = kThreads / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) sh.red[threadIdx.x] = fmax(sh.red[threadIdx.x], sh.red[threadIdx.x + o]);
    __syncthreads();
  }
  const double r = sh.red[0];
  __syncthreads();
  return r;
}

__device__ double block_reduce_sum(double v, Shared& sh) {
  sh.red[threadIdx.x] = v;
  __syncthreads();
  for (int o = kThreads / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) sh.red[threadIdx.x] += sh.red[threadIdx.x + o];
    __syncthreads();
  }
  const double r = sh.red[0];
  __syncthreads();
  return r;
}

// Top-1 minus top-2 value of a logit row (a repeated maximum gives 0).
__device__ double row_top2_gap(const float* z, int V, Shared& sh) {
  double t1 = -INFINITY, t2 = -INFINITY;
  for (int y = threadIdx.x; y < V; y += kThreads) {
    const double v = (double)z[y];
    if (v > t1) {
      t2 = t1;
      t1 = v;
    } else if (v > t2) {
      t2 = v;
    }
  }
  sh.red[threadIdx.x] = t1;
  sh.red2[threadIdx.x] = t2;
  __syncthreads();
  for (int o = kThreads / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      const double a1 = sh.red[threadIdx.x], a2 = sh.red2[threadIdx.x];
      const double b1 = sh.red[threadIdx.x + o], b2 = sh.red2[threadIdx.x + o];
      sh.red[threadIdx.x] = fmax(a1, b1);
      sh.red2[threadIdx.x] = fmax(fmin(a1, b1), fmax(a2, b2));
    }
    __syncthreads();
  }
  const double g = sh.red[0] - sh.red2[0];
  __syncthreads();
  return g;
}

__device__ bool icdf_near_tie(double u, double c_lo, double c_hi, double tol) {
  const double blo = 4.0 * tol * fmin(c_lo, 1.0 - c_lo);
  const double bhi = 4.0 * tol * fmin(c_hi, 1.0 - c_hi);
  return fabs(u - c_lo) < blo || fabs(u - c_hi) < bhi;
}

// log sum_y exp(z_y / T)
__device__ double row_lse(const float* z, int V, double invT, Shared& sh) {
  double mx = -INFINITY;
  for (int y = threadIdx.x; y < V; y += kThreads) mx = fmax(mx, (double)z[y] * invT);
  mx = block_reduce_max(mx, sh);
  double s = 0.0;
  for (int y = threadIdx.x; y < V; y += kThreads) s += exp((double)z[y] * invT - mx);
  s = block_reduce_sum(s, sh);
  return mx + log(s);
}

// Inverse-CDF draw from w(y) = f * exp(z_y/T - lse) off the candidates and
// sh.rc[j] on candidate sh.cid[j]: the smallest id whose cumulative mass
// exceeds u * total. Returns the id (all threads); sh.c_lo / sh.c_hi get the
// cumulative fractions at the edges of its bin.
__device__ int row_sample(const float* z, int V, double invT, double lse, double f, double u,
                          Shared& sh) {
  const int t = threadIdx.x;
  const int chunk = (V + kThreads - 1) / kThreads;
  const int y0 = min(V, t * chunk), y1 = min(V, y0 + chunk);
  int j = 0;
  while (j < sh.n_c && sh.cid[j] < y0) ++j;
  const int j0 = j;
  double s = 0.0;
  for (int y = y0; y < y1; ++y) {
    double w;
    if (j < sh.n_c && sh.cid[j] == y) w = sh.rc[j++];
    else w = f * exp((double)z[y] * invT - lse);
    s += w;
  }
  sh.red[t] = s;
  __syncthreads();
  if (t == 0) {
    double acc = 0.0;
    for (int i = 0; i < kThreads; ++i) {
      sh.pre[i] = acc;
      acc += sh.red[i];
    }
    sh.pre[kThreads] = acc;
    sh.result = -1;
    sh.found = 0;
  }
  __syncthreads();
  const double target = u * sh.pre[kThreads];
  if (sh.pre[t] <= target && target < sh.pre[t + 1]) {
    double cum = sh.pre[t];
    j = j0;
    int pick = -1;
    for (int y = y0; y < y1; ++y) {
      double w;
      if (j < sh.n_c && sh.cid[j] == y) w = sh.rc[j++];
      else w = f * exp((double)z[y] * invT - lse);
      if (w <= 0.0) continue;
      const double before = cum;
      cum += w;
      if (cum > target) {
        pick = y;
        sh.c_lo = before / sh.pre[kThreads];
        sh.c_hi = cum / sh.pre[kThreads];
        break;
      }
    }
    if (pick >= 0) {
      sh.result = pick;
      sh.found = 1;
    }
  }
  __syncthreads();
  if (!sh.found && t == 0) {
    // rounding left target at the total: the last id with mass
    for (int y = V - 1; y >= 0; --y) {
      double w = f * exp((double)z[y] * invT - lse);
      for (int i = 0; i < sh.n_c; ++i)
        if (sh.cid[i] == y) w = sh.rc[i];
      if (w > 0.0) {
        sh.result = y;
        break;
      }
    }
    sh.c_lo = sh.c_hi = u;  // drawn at the rounding edge: inside every band
  }
  __syncthreads();
  const int r = sh.result;
  __syncthreads();
  return r;
}

// Per row and vocabulary chunk c (ids [c ck, (c + 1) ck), ck = ceil(V /
// kStatChunks)): the chunk's max m of z / T and sum of exp(z / T - m), fp64,
// in a fixed order (thread-strided partials, then a tree over the threads).
// An empty chunk stores (-inf, 0).
__global__ __launch_bounds__(256) void row_stats_kernel(AcceptArgs a) {
  __shared__ double red[256];
  const int c = blockIdx.x, row = blockIdx.y, t = threadIdx.x;
  const int V = a.vocab, ck = (V + kStatChunks - 1) / kStatChunks;
  const int y0 = min(V, c * ck), y1 = min(V, y0 + ck);
  const float* z = a.logits + (size_t)row * V;
  const double invT = 1.0 / (double)a.temperature;
  double m = -INFINITY;
  for (int y = y0 + t; y < y1; y += 256) m = fmax(m, (double)z[y] * invT);
  red[t] = m;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] = fmax(red[t], red[t + o]);
    __syncthreads();
  }
  m = red[0];
  __syncthreads();
  double sum = 0.0;
  if (m != -INFINITY)
    for (int y = y0 + t; y < y1; y += 256) sum += exp((double)z[y] * invT - m);
  red[t] = sum;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] += red[t + o];
    __syncthreads();
  }
  if (t == 0) a.stats[(size_t)row * kStatChunks + c] = make_double2(m, red[0]);
}

// log sum_y exp(z_y / T) of a row from its chunk statistics (wave 0, lane c
// holding chunk c; every thread returns it).
__device__ double row_lse_stats(const double2* st, Shared& sh) {
  const int t = threadIdx.x;
  if (t < 64) {
    const double2 v = st[t];
    double M = v.x;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) M = fmax(M, __shfl_xor(M, o));
    double S = v.x == -INFINITY ? 0.0 : v.y * exp(v.x - M);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) S += __shfl_xor(S, o);
    if (t == 0) sh.red[0] = M + log(S);
  }
  __syncthreads();
  const double r = sh.red[0];
  __syncthreads();
  return r;
}

// Exclusive prefix of v over the workgroup in thread order (wave scans, then
// the wave totals); every thread also gets the total.
__device__ double block_scan(double v, double& total, Shared& sh) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  double x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh.wtot[wave] = x;
  __syncthreads();
  double before = 0.0, all = 0.0;
  for (int w = 0; w < kThreads / 64; ++w) {
    if (w < wave) before += sh.wtot[w];
    all += sh.wtot[w];
  }
  __syncthreads();
  total = all;
  return before + x - v;
}

// row_sample with the chunk statistics st of the row: the chunks' masses of
// w(y) = f p(y) off the candidates and sh.rc on them, the chunk holding the
// target u * total, then the smallest id of that chunk whose cumulative mass
// exceeds it (a thread per 1/kThreads of the chunk). sh.c_lo / sh.c_hi get
// the cumulative fractions at the edges of the drawn id's bin.
__device__ int row_sample_stats(const float* z, int V, double invT, double lse, double f, double u,
                                const double2* st, Shared& sh) {
  const int t = threadIdx.x;
  const int ck = (V + kStatChunks - 1) / kStatChunks;
  if (t < 64) {
    const double2 v = st[t];
    double off = v.x == -INFINITY ? 0.0 : v.y * exp(v.x - lse);  // sum of p over the chunk
    double cand = 0.0;
    const int c0 = t * ck, c1 = c0 + ck;
    for (int j = 0; j < sh.n_c; ++j)
      if (sh.cid[j] >= c0 && sh.cid[j] < c1) {
        off -= sh.pcand[j];
        cand += sh.rc[j];
      }
    double w = f * (off > 0.0 ? off : 0.0) + cand;
    double x = w;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const double y = __shfl_up(x, o);
      if (t >= o) x += y;
    }
    const double total = __shfl(x, 63);
    const double target = u * total;
    const double lo = x - w;
    // the first chunk whose span holds the target (the last chunk with mass
    // when rounding leaves the target at the total)
    const unsigned long long hit = __ballot(w > 0.0 && lo <= target && target < x);
    const unsigned long long any = __ballot(w > 0.0);
    const int pick = hit ? __ffsll((long long)hit) - 1 : (any ? 63 - __clzll((long long)any) : 0);
    const double lo_pick = __shfl(lo, pick);
    if (t == 0) {
      sh.result = pick;
      sh.pre[0] = lo_pick;
      sh.pre[1] = total;
      sh.c_lo = target;  // the target, for the scan below
    }
  }
  __syncthreads();
  const int c = sh.result;
  const double base = sh.pre[0], total = sh.pre[1], target = sh.c_lo;
  const int y0 = min(V, c * ck), y1 = min(V, y0 + ck);
  const int per = (y1 - y0 + kThreads - 1) / kThreads;
  const int a0 = min(y1, y0 + t * per), a1 = min(y1, a0 + per);
  auto weight = [&](int y) {
    for (int j = 0; j < sh.n_c; ++j)
      if (sh.cid[j] == y) return sh.rc[j];
    return f * exp((double)z[y] * invT - lse);
  };
  double s = 0.0;
  for (int y = a0; y < a1; ++y) s += weight(y);
  double tot_c;
  const double pre = base + block_scan(s, tot_c, sh);
  __syncthreads();
  if (t == 0) sh.found = 0;
  __syncthreads();
  if (pre <= target && target < pre + s) {
    double cum = pre;
    for (int y = a0; y < a1; ++y) {
      const double w = weight(y);
      if (w <= 0.0) continue;
      const double before = cum;
      cum += w;
      if (cum > target) {
        sh.result = y;
        sh.c_lo = before / total;
        sh.c_hi = cum / total;
        sh.found = 1;
        break;
      }
    }
  }
  __syncthreads();
  if (!sh.found && t == 0) {
    // rounding left the target past the chunk's recomputed mass: its last id
    // with mass, drawn at a rounding edge (inside every band)
    int r = -1;  // no mass anywhere: no token, as in row_sample
    for (int y = y1 - 1; y >= y0; --y)
      if (weight(y) > 0.0) {
        r = y;
        break;
      }
    sh.result = r;
    sh.c_lo = sh.c_hi = u;
  }
  __syncthreads();
  const int r = sh.result;
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kThreads) void accept_kernel(AcceptArgs a) {
  __shared__ Shared sh;
  const int b = blockIdx.x, t = threadIdx.x;
  const int ns = a.n_slots;
  int32_t* path = a.path + (size_t)b * ns;
  // the sequence's block tokens and uniforms, staged once (the walk reads
  // them one node at a time)
  for (int i = t; i < ns; i += kThreads) {
    path[i] = i == 0 ? 0 : -1;
    sh.tok[i] = a.tokens[(size_t)b * ns + i];
    sh.ua[i] = a.u_accept ? a.u_accept[(size_t)b * ns + i] : 0.0f;
    sh.us[i] = a.u_sample ? a.u_sample[(size_t)b * ns + i] : 0.0f;
  }
  const int32_t* tok = sh.tok;
  __syncthreads();

  const double tol = (double)a.tol_logit;
  const bool flags = a.near_tie != nullptr;
  if (a.mode == 0) {  // GREEDY
    if (!flags) {
      if (t == 0) {
        int cur = 0, depth = 0;
        for (;;) {
          const int want = a.argmax[(size_t)b * ns + cur];
          int nxt = -1;
          for (int ch = cur + 1; ch < ns; ++ch)
            if (a.topo.parent[ch] == cur && tok[ch] == want) {
              nxt = ch;
              break;
            }
          if (nxt < 0) {
            a.next_tok[b] = want;
            break;
          }
          cur = nxt;
          path[++depth] = cur;
        }
        a.acc_len[b] = depth;
      }
      return;
    }
    // with near-tie flags every thread walks (the top-2 gap of each visited
    // row is a workgroup reduction over the logits)
    int cur = 0, depth = 0;
    bool tie = false;
    for (;;) {
      const int want = a.argmax[(size_t)b * ns + cur];
      tie |= row_top2_gap(a.logits + ((size_t)b * ns + cur) * a.vocab, a.vocab, sh) < 2.0 * tol;
      int nxt = -1;
      for (int ch = cur + 1; ch < ns; ++ch)
        if (a.topo.parent[ch] == cur && tok[ch] == want) {
          nxt = ch;
          break;
        }
      if (nxt < 0) {
        if (t == 0) a.next_tok[b] = want;
        break;
      }
      cur = nxt;
      ++depth;
      if (t == 0) path[depth] = cur;
    }
    if (t == 0) {
      a.acc_len[b] = depth;
      a.near_tie[b] = tie ? 1 : 0;
    }
    return;
  }

  const double invT = 1.0 / (double)a.temperature;
  int cur = 0, depth = 0;
  bool tie = false;
  for (;;) {
    const float* z = a.logits + ((size_t)b * ns + cur) * a.vocab;
    const double2* st = a.stats ? a.stats + ((size_t)b * ns + cur) * kStatChunks : nullptr;
    const double lse = st ? row_lse_stats(st, sh) : row_lse(z, a.vocab, invT, sh);
    int next_child = -1, out_tok = -1;
    if (a.mode == 2) {  // MATCH: y ~ p, descend to the child carrying y
      if (t == 0) sh.n_c = 0;
      __syncthreads();
      const double u = (double)sh.us[cur];
      const int y = st ? row_sample_stats(z, a.vocab, invT, lse, 1.0, u, st, sh)
                       : row_sample(z, a.vocab, invT, lse, 1.0, u, sh);
      tie |= icdf_near_tie(u, sh.c_lo, sh.c_hi, tol);
      for (int ch = cur + 1; ch < ns; ++ch)
        if (a.topo.parent[ch] == cur && tok[ch] == y) {
          next_child = ch;
          break;
        }
      if (next_child < 0) out_tok = y;
    } else {  // REJECTION
      const int C = a.n_cand;
      const int* cid = a.cand_ids + ((size_t)b * ns + cur) * C;
      const float* cq = a.cand_q + ((size_t)b * ns + cur) * C;
      if (t < C) sh.tmp_id[t] = cid[t];
      __syncthreads();
      if (t < C) {  // rank-sort the (distinct) candidate ids
        const int my = sh.tmp_id[t];
        int rank = 0;
        for (int i = 0; i < C; ++i) rank += sh.tmp_id[i] < my;
        sh.cid[rank] = my;
        sh.qc[rank] = (double)cq[t];
        sh.rc[rank] = exp((double)z[my] * invT - lse);
        sh.pcand[rank] = sh.rc[rank];
      }
      if (t == 0) sh.n_c = C;
      __syncthreads();
      double f = 1.0;  // residual off the candidates = f * p
      for (int ch = cur + 1; ch < ns; ++ch) {
        if (a.topo.parent[ch] != cur) continue;
        const int x = tok[ch];
        int jx = -1;
        for (int i = 0; i < C; ++i)
          if (sh.cid[i] == x) jx = i;
        if (jx < 0 || !(sh.qc[jx] > 0.0)) {
          if (t == 0) atomicOr(a.status, 2u);
          out_tok = -1;
          next_child = -2;
          break;
        }
        const double ratio = sh.rc[jx] / sh.qc[jx];
        const double alpha = ratio < 1.0 ? ratio : 1.0;
        const double u = (double)sh.ua[ch];
        tie |= fabs(u - alpha) < 2.0 * tol * alpha * invT;
        if (u < alpha) {
          next_child = ch;
          break;
        }
        // rejected: r <- normalise((r - q)^+), q <- q without x, renormalised
        double pc = 0.0, rnew = 0.0;
        for (int i = 0; i < C; ++i) pc += sh.pcand[i];
        __syncthreads();
        if (t < C) {
          const double d = sh.rc[t] - sh.qc[t];
          sh.rc[t] = d > 0.0 ? d : 0.0;
        }
        __syncthreads();
        for (int i = 0; i < C; ++i) rnew += sh.rc[i];
        const double zr = rnew + f * (1.0 - pc);
        __syncthreads();
        if (zr > 0.0) {
          f /= zr;
          if (t < C) sh.rc[t] /= zr;
        }
        const double qx = sh.qc[jx];
        __syncthreads();
        if (t < C) {
          double qv = t == jx ? 0.0 : sh.qc[t];
          if (qx < 1.0) qv /= (1.0 - qx);
          sh.qc[t] = qv;
        }
        __syncthreads();
      }
      if (next_child == -2) {
        if (t == 0) {
          a.acc_len[b] = depth;
          a.next_tok[b] = -1;
          if (flags) a.near_tie[b] = 1;
        }
        return;
      }
      if (next_child < 0) {
        const double u = (double)sh.us[cur];
        out_tok = st ? row_sample_stats(z, a.vocab, invT, lse, f, u, st, sh)
                     : row_sample(z, a.vocab, invT, lse, f, u, sh);
        tie |= icdf_near_tie(u, sh.c_lo, sh.c_hi, tol);
      }
    }
    if (next_child < 0) {
      if (t == 0) a.next_tok[b] = out_tok;
      break;
    }
    cur = next_child;
    ++depth;
    if (t == 0) path[depth] = cur;
  }
  if (t == 0) {
    a.acc_len[b] = depth;
    if (flags) a.near_tie[b] = tie ? 1 : 0;
  }
}

// Move accepted rows len + path[r] -> len + r (r = 1..A) of every layer and
// kv head. Sources are staged in LDS first: a destination row may be the
// source of a later depth.
__global__ __launch_bounds__(256) void commit_copy_kernel(CommitArgs a) {
  extern __shared__ u32x4 stage[];  // [2][A][hd/8]
  const int h = blockIdx.x, b = blockIdx.y, l = blockIdx.z;
  const int A = a.acc_len[b];
  if (A <= 0 || A >= a.n_slots) return;
  const int L = a.len[b];
  if (L + a.n_slots > a.capacity) return;
  const int cpr = a.head_dim / 8;  // 16-byte chunks per row
  const size_t base = ((((size_t)l * a.batch_cap + b) * a.n_kv_heads + h) * a.capacity) * a.head_dim;
  const int32_t* path = a.path + (size_t)b * a.n_slots;
  const int n = A * cpr;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int r = i / cpr + 1, q = i - (r - 1) * cpr;
    const size_t src = base + (size_t)(L + path[r]) * a.head_dim + q * 8;
    stage[i] = *reinterpret_cast<const u32x4*>(a.k_cache + src);
    stage[n + i] = *reinterpret_cast<const u32x4*>(a.v_cache + src);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int r = i / cpr + 1, q = i - (r - 1) * cpr;
    const size_t dst = base + (size_t)(L + r) * a.head_dim + q * 8;
    *reinterpret_cast<u32x4*>(a.k_cache + dst) = stage[i];
    *reinterpret_cast<u32x4*>(a.v_cache + dst) = stage[n + i];
  }
}

__global__ void commit_len_kernel(CommitArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.batch) return;
  const int A = a.acc_len[b];
  if (A < 0 || A >= a.n_slots) return;
  if (a.len[b] + a.n_slots > a.capacity) return;
  a.len[b] += 1 + A;
}

}  // namespace

hipError_t launch_accept(const AcceptArgs& a, hipStream_t s) {
  if (a.stats) {
    hipLaunchKernelGGL(row_stats_kernel, dim3(kStatChunks, a.batch * a.n_slots), dim3(256), 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(accept_kernel, dim3(a.batch), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_commit(const CommitArgs& a, hipStream_t s) {
  if (a.copy_rows) {
    const size_t shmem = (size_t)2 * (a.n_slots - 1) * (a.head_dim / 8) * sizeof(u32x4);
    hipLaunchKernelGGL(commit_copy_kernel, dim3(a.n_kv_heads, a.batch, a.n_layers), dim3(256),
                       shmem, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(commit_len_kernel, dim3((a.batch + 63) / 64), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace msd
