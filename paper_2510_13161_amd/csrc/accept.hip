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

struct Shared {
  double red[kThreads];
  double red2[kThreads];
  double pre[kThreads + 1];
  double c_lo, c_hi;       // cumulative fractions at the edges of the drawn id's bin
  int cid[kMaxCand];       // candidate ids sorted ascending
  double rc[kMaxCand];     // residual mass at each sorted candidate
  double qc[kMaxCand];     // draft mass at each sorted candidate
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

__global__ __launch_bounds__(kThreads) void accept_kernel(AcceptArgs a) {
  __shared__ Shared sh;
  const int b = blockIdx.x, t = threadIdx.x;
  const int ns = a.n_slots;
  int32_t* path = a.path + (size_t)b * ns;
  const int32_t* tok = a.tokens + (size_t)b * ns;
  for (int i = t; i < ns; i += kThreads) path[i] = i == 0 ? 0 : -1;
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
    const double lse = row_lse(z, a.vocab, invT, sh);
    int next_child = -1, out_tok = -1;
    if (a.mode == 2) {  // MATCH: y ~ p, descend to the child carrying y
      if (t == 0) sh.n_c = 0;
      __syncthreads();
      const double u = (double)a.u_sample[(size_t)b * ns + cur];
      const int y = row_sample(z, a.vocab, invT, lse, 1.0, u, sh);
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
      if (t < C) {  // rank-sort the (distinct) candidate ids
        const int my = cid[t];
        int rank = 0;
        for (int i = 0; i < C; ++i) rank += cid[i] < my;
        sh.cid[rank] = my;
        sh.qc[rank] = (double)cq[t];
        sh.rc[rank] = exp((double)z[my] * invT - lse);
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
        const double u = (double)a.u_accept[(size_t)b * ns + ch];
        tie |= fabs(u - alpha) < 2.0 * tol * alpha * invT;
        if (u < alpha) {
          next_child = ch;
          break;
        }
        // rejected: r <- normalise((r - q)^+), q <- q without x, renormalised
        double pc = 0.0, rnew = 0.0;
        for (int i = 0; i < C; ++i) pc += exp((double)z[sh.cid[i]] * invT - lse);
        __syncthreads();
        if (t == 0) {
          for (int i = 0; i < C; ++i) {
            const double d = sh.rc[i] - sh.qc[i];
            sh.rc[i] = d > 0.0 ? d : 0.0;
          }
        }
        __syncthreads();
        for (int i = 0; i < C; ++i) rnew += sh.rc[i];
        const double zr = rnew + f * (1.0 - pc);
        __syncthreads();
        if (zr > 0.0) {
          f /= zr;
          if (t == 0)
            for (int i = 0; i < C; ++i) sh.rc[i] /= zr;
        }
        const double qx = sh.qc[jx];
        __syncthreads();
        if (t == 0) {
          sh.qc[jx] = 0.0;
          if (qx < 1.0)
            for (int i = 0; i < C; ++i) sh.qc[i] /= (1.0 - qx);
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
        const double u = (double)a.u_sample[(size_t)b * ns + cur];
        out_tok = row_sample(z, a.vocab, invT, lse, f, u, sh);
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
