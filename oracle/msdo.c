/*
 * msdo — fp64 CPU oracle of the Mirror-SD verification step.
 *
 * TEST INFRASTRUCTURE ONLY (see msdo.h): loaded by tests, the smoke check
 * and the benchmark's CPU-baseline leg, never by the product path.
 *
 * Plain loops, one output element per thread, fixed summation order (index
 * ascending), fp64 everywhere; inputs given as bf16 / fp32 are upcast
 * exactly. OpenMP only distributes independent output elements.
 *
 * Pins (what, other than itself, fixes each function; tests/test_oracle.py):
 *  msdo_embed/layer/head  block forward == token-by-token forward, bitwise
 *                         (Sec. 2: verification is a teacher-forced pass of
 *                         the same model); tree node == its root-to-node chain
 *                         (Sec. 3.1: a depth-r node holds the token at t + r);
 *                         one row over an empty cache returns v (softmax of a
 *                         single key); RoPE at position 0 is the identity;
 *                         an independent NumPy float64 forward of the same
 *                         architecture on the tiny model.
 *  msdo_topk              NumPy lexsort of the full row; lse against a
 *                         float128-free two-pass recompute.
 *  msdo_accept            GREEDY == autoregressive argmax decoding (Sec. 2,
 *                         App. B); planted mismatch at r* gives A = r*;
 *                         REJECTION output law by exact enumeration == p
 *                         (one child: Leviathan et al. 2023 Thm. 1; several
 *                         children drawn without replacement: recursive
 *                         rejection, Jeon et al. 2024); one-child acceptance
 *                         probability == sum_x min(p(x), q(x)).
 *  msdo_kv_commit         the committed rows equal a fresh forward of the
 *                         accepted sequence.
 */
#include "msdo.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static inline double bf(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

static void* xmalloc(size_t n) {
  void* p = calloc(n ? n : 1, 1);
  if (!p) abort();
  return p;
}

/* Pre-norm of one row. RMSNorm: x / sqrt(mean(x^2) + eps) * g.
 * LayerNorm: (x - mean) / sqrt(var + eps) * g + b (biased variance). */
static void norm_row(const msdo_cfg* c, const double* x, const uint16_t* g, const uint16_t* b,
                     double* y) {
  const int d = c->d_model;
  if (c->layer_norm) {
    double mu = 0.0;
    for (int k = 0; k < d; ++k) mu += x[k];
    mu /= d;
    double var = 0.0;
    for (int k = 0; k < d; ++k) var += (x[k] - mu) * (x[k] - mu);
    var /= d;
    double s = 1.0 / sqrt(var + c->norm_eps);
    for (int k = 0; k < d; ++k) y[k] = (x[k] - mu) * s * bf(g[k]) + (b ? bf(b[k]) : 0.0);
  } else {
    double ss = 0.0;
    for (int k = 0; k < d; ++k) ss += x[k] * x[k];
    double s = 1.0 / sqrt(ss / d + c->norm_eps);
    for (int k = 0; k < d; ++k) y[k] = x[k] * s * bf(g[k]);
  }
}

/* y[i][o] = sum_k W[o][k] x[i][k] (+ bias[o]); x [n][in], W [out][in], y [n][out]. */
static void linear(int n, int in, int out, const double* x, const uint16_t* W,
                   const uint16_t* bias, double* y) {
  double* xt = (double*)xmalloc((size_t)in * n * sizeof(double));
  for (int i = 0; i < n; ++i)
    for (int k = 0; k < in; ++k) xt[(size_t)k * n + i] = x[(size_t)i * in + k];
#pragma omp parallel
  {
    double* acc = (double*)xmalloc((size_t)n * sizeof(double));
#pragma omp for schedule(static)
    for (int o = 0; o < out; ++o) {
      for (int i = 0; i < n; ++i) acc[i] = 0.0;
      const uint16_t* wr = W + (size_t)o * in;
      for (int k = 0; k < in; ++k) {
        const double wv = bf(wr[k]);
        const double* xr = xt + (size_t)k * n;
        for (int i = 0; i < n; ++i) acc[i] += wv * xr[i];
      }
      const double b = bias ? bf(bias[o]) : 0.0;
      for (int i = 0; i < n; ++i) y[(size_t)i * out + o] = acc[i] + b;
    }
    free(acc);
  }
  free(xt);
}

/* Rotary position embedding, rotate-half form: for j < hd/2 and angle
 * a = pos * theta^(-2j/hd): (u_j, u_{j+hd/2}) <- (u_j cos a - u_{j+hd/2} sin a,
 * u_{j+hd/2} cos a + u_j sin a). */
static void rope(double* u, int hd, int pos, double theta) {
  const int half = hd / 2;
  for (int j = 0; j < half; ++j) {
    double a = (double)pos * pow(theta, -2.0 * (double)j / (double)hd);
    double cs = cos(a), sn = sin(a);
    double lo = u[j], hi = u[j + half];
    u[j] = lo * cs - hi * sn;
    u[j + half] = hi * cs + lo * sn;
  }
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

/* Nearest value with an 8-bit significand (the bf16 format), ties to even:
 * the representation of a K/V cache entry. (Range limits of bf16 are far
 * from the values seen here.) */
static double to_cache_format(double v) {
  if (v == 0.0 || !isfinite(v)) return v;
  int e;
  frexp(v, &e);                       /* v = f * 2^e, 0.5 <= |f| < 1 */
  const double scaled = ldexp(v, 8 - e);  /* 8 significant bits left of the point */
  return ldexp(nearbyint(scaled), e - 8);
}

void msdo_embed(const msdo_cfg* c, const msdo_global_w* g, int32_t n, const int32_t* tok,
                const int32_t* pos, double* x) {
  const int d = c->d_model;
  for (int i = 0; i < n; ++i) {
    const uint16_t* e = g->embed + (size_t)tok[i] * d;
    for (int k = 0; k < d; ++k) x[(size_t)i * d + k] = bf(e[k]);
    if (c->learned_pos) {
      const uint16_t* p = g->pos_embed + (size_t)pos[i] * d;
      for (int k = 0; k < d; ++k) x[(size_t)i * d + k] += bf(p[k]);
    }
  }
}

void msdo_layer(const msdo_cfg* c, const msdo_layer_w* w, int32_t n, double* x,
                const int32_t* pos, const int32_t* parent, int32_t n_ctx, int32_t ctx_stride,
                const uint16_t* ctx_k, const uint16_t* ctx_v, int32_t n_extra,
                const double* extra_k, const double* extra_v, double* blk_k, double* blk_v,
                int32_t kv_cache_bf16) {
  const int d = c->d_model, H = c->n_heads, Hk = c->n_kv_heads, hd = c->head_dim;
  const int qd = H * hd, kd = Hk * hd, F = c->d_ffn;
  const int group = H / Hk;
  const double scale = 1.0 / sqrt((double)hd);

  double* h = (double*)xmalloc((size_t)n * d * sizeof(double));
  double* q = (double*)xmalloc((size_t)n * qd * sizeof(double));
  double* o = (double*)xmalloc((size_t)n * qd * sizeof(double));
  double* y = (double*)xmalloc((size_t)n * d * sizeof(double));

  /* ancestors-or-self: anc[i*n + a] = 1 iff a lies on the root-to-i path */
  unsigned char* anc = (unsigned char*)xmalloc((size_t)n * n);
  memset(anc, 0, (size_t)n * n);
  for (int i = 0; i < n; ++i)
    for (int a = i; a >= 0; a = parent[a]) anc[(size_t)i * n + a] = 1;

  /* attention block: h = norm1(x); q, k, v = W h (+ b); rotary; attend */
  for (int i = 0; i < n; ++i) norm_row(c, x + (size_t)i * d, w->attn_g, w->attn_b, h + (size_t)i * d);
  linear(n, d, qd, h, w->wq, w->bq, q);
  linear(n, d, kd, h, w->wk, w->bk, blk_k);
  linear(n, d, kd, h, w->wv, w->bv, blk_v);
  if (!c->learned_pos) {
    for (int i = 0; i < n; ++i) {
      for (int hh = 0; hh < H; ++hh) rope(q + (size_t)i * qd + hh * hd, hd, pos[i], c->rope_theta);
      for (int hh = 0; hh < Hk; ++hh) rope(blk_k + (size_t)i * kd + hh * hd, hd, pos[i], c->rope_theta);
    }
  }
  /* the block's keys and values enter the KV cache, which stores the same
   * bf16 format as the given context, before any row attends to them */
  if (kv_cache_bf16) {
    for (size_t t = 0; t < (size_t)n * kd; ++t) {
      blk_k[t] = to_cache_format(blk_k[t]);
      blk_v[t] = to_cache_format(blk_v[t]);
    }
  }

  const int n_keys_max = n_ctx + n_extra + n;
#pragma omp parallel
  {
    double* s = (double*)xmalloc((size_t)n_keys_max * sizeof(double));
    const double** vrow = (const double**)xmalloc((size_t)n_keys_max * sizeof(double*));
#pragma omp for collapse(2) schedule(static)
    for (int i = 0; i < n; ++i)
      for (int hh = 0; hh < H; ++hh) {
        const int kh = hh / group;
        const double* qi = q + (size_t)i * qd + hh * hd;
        int nk = 0;
        /* scores, keys in position order */
        for (int j = 0; j < n_ctx; ++j) {
          const uint16_t* kr = ctx_k + ((size_t)kh * ctx_stride + j) * hd;
          double acc = 0.0;
          for (int t = 0; t < hd; ++t) acc += qi[t] * bf(kr[t]);
          s[nk] = acc * scale;
          vrow[nk] = NULL; /* context value row, read below by index */
          ++nk;
        }
        for (int e = 0; e < n_extra; ++e) {
          const double* kr = extra_k + ((size_t)e * Hk + kh) * hd;
          double acc = 0.0;
          for (int t = 0; t < hd; ++t) acc += qi[t] * kr[t];
          s[nk] = acc * scale;
          vrow[nk] = extra_v + ((size_t)e * Hk + kh) * hd;
          ++nk;
        }
        for (int a = 0; a < n; ++a) {
          if (!anc[(size_t)i * n + a]) continue;
          const double* kr = blk_k + ((size_t)a * Hk + kh) * hd;
          double acc = 0.0;
          for (int t = 0; t < hd; ++t) acc += qi[t] * kr[t];
          s[nk] = acc * scale;
          vrow[nk] = blk_v + ((size_t)a * Hk + kh) * hd;
          ++nk;
        }
        /* softmax over the keys, then the value average */
        double m = -INFINITY;
        for (int j = 0; j < nk; ++j) m = s[j] > m ? s[j] : m;
        double den = 0.0;
        for (int j = 0; j < nk; ++j) {
          s[j] = exp(s[j] - m);
          den += s[j];
        }
        double* oi = o + (size_t)i * qd + hh * hd;
        for (int t = 0; t < hd; ++t) oi[t] = 0.0;
        for (int j = 0; j < nk; ++j) {
          const double p = s[j] / den;
          if (j < n_ctx) {
            const uint16_t* vr = ctx_v + ((size_t)kh * ctx_stride + j) * hd;
            for (int t = 0; t < hd; ++t) oi[t] += p * bf(vr[t]);
          } else {
            const double* vr = vrow[j];
            for (int t = 0; t < hd; ++t) oi[t] += p * vr[t];
          }
        }
      }
    free(vrow);
    free(s);
  }

  /* x += W_o o (+ b_o) */
  linear(n, qd, d, o, w->wo, w->bo, y);
  for (size_t t = 0; t < (size_t)n * d; ++t) x[t] += y[t];

  /* feed-forward block: x += FFN(norm2(x)) */
  for (int i = 0; i < n; ++i) norm_row(c, x + (size_t)i * d, w->mlp_g, w->mlp_b, h + (size_t)i * d);
  double* a = (double*)xmalloc((size_t)n * F * sizeof(double));
  if (c->relu_ffn) {
    linear(n, d, F, h, w->w_up, w->b_up, a);
    for (size_t t = 0; t < (size_t)n * F; ++t) a[t] = a[t] > 0.0 ? a[t] : 0.0;
  } else {
    double* u = (double*)xmalloc((size_t)n * F * sizeof(double));
    linear(n, d, F, h, w->w_gate, NULL, a);
    linear(n, d, F, h, w->w_up, NULL, u);
    for (size_t t = 0; t < (size_t)n * F; ++t) a[t] = silu(a[t]) * u[t];
    free(u);
  }
  linear(n, F, d, a, w->w_down, w->b_down, y);
  for (size_t t = 0; t < (size_t)n * d; ++t) x[t] += y[t];

  free(a);
  free(anc);
  free(y);
  free(o);
  free(q);
  free(h);
}

void msdo_head(const msdo_cfg* c, const msdo_global_w* g, int32_t n, const double* x,
               double* logits) {
  const int d = c->d_model;
  double* h = (double*)xmalloc((size_t)n * d * sizeof(double));
  for (int i = 0; i < n; ++i) norm_row(c, x + (size_t)i * d, g->final_g, g->final_b, h + (size_t)i * d);
  linear(n, d, c->vocab, h, g->lm_head, NULL, logits);
  free(h);
}

/* log sum_y exp(z_y / T), max-subtracted, summed in ascending id order. */
static double logsumexp_t(int V, const double* z, double T) {
  double m = -INFINITY;
  for (int y = 0; y < V; ++y) m = z[y] / T > m ? z[y] / T : m;
  double s = 0.0;
  for (int y = 0; y < V; ++y) s += exp(z[y] / T - m);
  return m + log(s);
}

/* (a beats b) under the order: larger logit first, then smaller id. */
static int beats(double za, int ia, double zb, int ib) {
  return za > zb || (za == zb && ia < ib);
}

void msdo_topk(int32_t n, int32_t V, const double* logits, int32_t kappa, int32_t* ids,
               double* logp, double* lse) {
#pragma omp parallel for schedule(static)
  for (int i = 0; i < n; ++i) {
    const double* z = logits + (size_t)i * V;
    const double l = logsumexp_t(V, z, 1.0);
    if (lse) lse[i] = l;
    /* kappa rounds of selecting the best element not yet taken */
    for (int r = 0; r < kappa; ++r) {
      int best = -1;
      for (int y = 0; y < V; ++y) {
        int taken = 0;
        for (int t = 0; t < r; ++t) taken |= ids[(size_t)i * kappa + t] == y;
        if (taken) continue;
        if (best < 0 || beats(z[y], y, z[best], best)) best = y;
      }
      ids[(size_t)i * kappa + r] = best;
      logp[(size_t)i * kappa + r] = z[best] - l;
    }
  }
}

/* Inverse-CDF draw: the smallest id k with sum_{y<=k} r(y) > u * sum_y r(y),
 * sums in ascending id order. *c_lo / *c_hi receive the cumulative fractions
 * of the mass at the lower and upper edge of the chosen id's bin. */
static int sample_icdf(int V, const double* r, double u, double* c_lo, double* c_hi) {
  double total = 0.0;
  for (int y = 0; y < V; ++y) total += r[y];
  const double target = u * total;
  double cum = 0.0;
  int last = -1;
  for (int y = 0; y < V; ++y) {
    if (r[y] <= 0.0) continue;
    const double before = cum;
    cum += r[y];
    last = y;
    *c_lo = before / total;
    *c_hi = cum / total;
    if (cum > target) return y;
  }
  return last;
}

/* Near-tie bands (a decision a logit error of tol could flip):
 *  argmax        top-1 minus top-2 logit below 2 tol;
 *  accept test   |u - alpha| < 2 tol alpha / T (alpha moves by a factor
 *                exp(+-2 tol / T) when z_x and the normaliser each move by tol);
 *  inverse CDF   |u - c| < 4 tol min(c, 1 - c) at either edge c of the
 *                chosen bin (the cumulative mass below an edge moves by that
 *                relative amount).
 * Bands are open intervals, so tol = 0 flags nothing. */
static int argmax_near_tie(int V, const double* z, double tol) {
  double t1 = -INFINITY, t2 = -INFINITY;
  for (int y = 0; y < V; ++y) {
    if (z[y] > t1) {
      t2 = t1;
      t1 = z[y];
    } else if (z[y] > t2) {
      t2 = z[y];
    }
  }
  return t1 - t2 < 2.0 * tol;
}

static int icdf_near_tie(double u, double c_lo, double c_hi, double tol) {
  const double blo = 4.0 * tol * (c_lo < 1.0 - c_lo ? c_lo : 1.0 - c_lo);
  const double bhi = 4.0 * tol * (c_hi < 1.0 - c_hi ? c_hi : 1.0 - c_hi);
  return fabs(u - c_lo) < blo || fabs(u - c_hi) < bhi;
}

/* p_s = Softmax(z_s / T) as a dense vector. */
static void probs(int V, const double* z, double T, double* p) {
  const double l = logsumexp_t(V, z, T);
  for (int y = 0; y < V; ++y) p[y] = exp(z[y] / T - l);
}

static int argmax_row(int V, const double* z) {
  int best = 0;
  for (int y = 1; y < V; ++y)
    if (z[y] > z[best]) best = y;
  return best;
}

/*
 * Readings taken where the paper is silent (each listed in the design notes):
 *  - whole-tree verification; the accepted path is the longest root-to-node
 *    path whose tokens the target's rule accepts, children tried in slot order;
 *  - a next token is always returned: the correction after a mismatch, or
 *    the bonus drawn at the last accepted node when the path ends in a leaf;
 *  - REJECTION: at a node with children drawn from the sparse draft law q
 *    without replacement, child x is accepted iff u_accept[child] <
 *    min(1, r(x)/q(x)); after a rejection r <- normalise((r - q)^+) and
 *    q <- q without x, renormalised; if all are rejected the next token is
 *    drawn from r with u_sample[node]. r starts as p = Softmax(z/T).
 *  - MATCH: the paper's sample-and-compare: y ~ p at the node (u_sample);
 *    descend to the child carrying y, else y is the next token.
 */
int32_t msdo_accept(int32_t n, const int32_t* parent, const int32_t* tokens, int32_t V,
                    const double* logits, int32_t mode, double temperature, int32_t n_cand,
                    const int32_t* cand_ids, const float* cand_q, const float* u_accept,
                    const float* u_sample, double tol_logit, int32_t* acc_len, int32_t* next_tok,
                    int32_t* path, int32_t* tie_depth, int32_t* tie_next) {
  int cur = 0, depth = 0;
  path[0] = 0;
  *tie_depth = -1;
  *tie_next = 0;
  double* r = NULL;
  double* q = NULL;
  if (mode != MSDO_GREEDY) {
    r = (double*)xmalloc((size_t)V * sizeof(double));
    q = (double*)xmalloc((size_t)V * sizeof(double));
  }
  int status = 0;
  for (;;) {
    const double* z = logits + (size_t)cur * V;
    int next_child = -1;
    int out_tok = -1;
    int tie = 0;       /* a decision choosing the way down is in a band */
    int tie_draw = 0;  /* REJECTION: the final draw is in a band        */
    double c_lo = 0.0, c_hi = 1.0;
    if (mode == MSDO_GREEDY) {
      const int a = argmax_row(V, z);
      tie = argmax_near_tie(V, z, tol_logit);
      for (int ch = cur + 1; ch < n; ++ch)
        if (parent[ch] == cur && tokens[ch] == a) { next_child = ch; break; }
      if (next_child < 0) out_tok = a;
    } else if (mode == MSDO_MATCH) {
      probs(V, z, temperature, r);
      const double u = (double)u_sample[cur];
      const int y = sample_icdf(V, r, u, &c_lo, &c_hi);
      tie = icdf_near_tie(u, c_lo, c_hi, tol_logit);
      for (int ch = cur + 1; ch < n; ++ch)
        if (parent[ch] == cur && tokens[ch] == y) { next_child = ch; break; }
      if (next_child < 0) out_tok = y;
    } else {
      probs(V, z, temperature, r);
      for (int y = 0; y < V; ++y) q[y] = 0.0;
      for (int j = 0; j < n_cand; ++j)
        q[cand_ids[(size_t)cur * n_cand + j]] = (double)cand_q[(size_t)cur * n_cand + j];
      for (int ch = cur + 1; ch < n && next_child < 0; ++ch) {
        if (parent[ch] != cur) continue;
        const int x = tokens[ch];
        if (!(q[x] > 0.0)) { status = -1; break; }
        const double ratio = r[x] / q[x];
        const double alpha = ratio < 1.0 ? ratio : 1.0;
        const double u = (double)u_accept[ch];
        tie |= fabs(u - alpha) < 2.0 * tol_logit * alpha / temperature;
        if (u < alpha) { next_child = ch; break; }
        /* rejected: residual target and draft law without x */
        double zr = 0.0;
        for (int y = 0; y < V; ++y) {
          const double t = r[y] - q[y];
          r[y] = t > 0.0 ? t : 0.0;
          zr += r[y];
        }
        if (zr > 0.0)
          for (int y = 0; y < V; ++y) r[y] /= zr;
        const double qx = q[x];
        q[x] = 0.0;
        if (qx < 1.0)
          for (int y = 0; y < V; ++y) q[y] /= (1.0 - qx);
      }
      if (status) break;
      if (next_child < 0) {
        const double u = (double)u_sample[cur];
        out_tok = sample_icdf(V, r, u, &c_lo, &c_hi);
        tie_draw = icdf_near_tie(u, c_lo, c_hi, tol_logit);
      }
    }
    if (tie && *tie_depth < 0) *tie_depth = depth;
    if (next_child < 0) {
      *next_tok = out_tok;
      *tie_next = tie || tie_draw;
      break;
    }
    cur = next_child;
    path[++depth] = cur;
  }
  *acc_len = depth;
  free(r);
  free(q);
  return status;
}

int32_t msdo_kv_commit(int32_t n_layers, int32_t n_kv_heads, int32_t cap, int32_t head_dim,
                       uint16_t* k, uint16_t* v, int32_t len, int32_t acc_len,
                       const int32_t* path) {
  for (int l = 0; l < n_layers; ++l)
    for (int h = 0; h < n_kv_heads; ++h) {
      const size_t base = (((size_t)l * n_kv_heads + h) * cap) * head_dim;
      for (int r = 1; r <= acc_len; ++r) {
        const size_t dst = base + (size_t)(len + r) * head_dim;
        const size_t src = base + (size_t)(len + path[r]) * head_dim;
        memmove(k + dst, k + src, (size_t)head_dim * sizeof(uint16_t));
        memmove(v + dst, v + src, (size_t)head_dim * sizeof(uint16_t));
      }
    }
  return len + 1 + acc_len;
}
