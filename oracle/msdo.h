/*
 * msdo — the oracle of the Mirror-SD verification step.
 *
 * TEST INFRASTRUCTURE ONLY. This is a plain, slow, fp64 CPU statement of
 * what the verification step computes. Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the product path
 * (the HIP library) never links, calls or imports it, and the two share no
 * source.
 *
 * What it follows (Mirror Speculative Decoding, arXiv 2510.13161):
 *  - Sec. 2, autoregressive factorisation: next-token law = Softmax(W h_t);
 *    the target is a decoder-only transformer (pre-norm blocks).
 *  - Sec. 2, speculative verification: the target scores the whole draft
 *    window in one teacher-forced pass; A_t is the longest prefix on which
 *    draft and target tokens agree; a correction token follows.
 *  - Sec. 3.1, early-exit proxy p^(l) = Softmax(W_LM h^(l)) at l = l_e < N
 *    and the token channel M_t = Top-kappa(p^(l_e)) = {(v_i, log p_i)}.
 *  - Sec. 3.1, hypothesis tree T_t: a node at depth r holds the token at
 *    position t + r; the verifier scores the branch-complete rollout.
 *  - App. B, acceptance operator: A_t = max{ r : yhat_{t+j} = y^target_{t+j}
 *    for all j <= r }, identical for vanilla SD and Mirror-SD; the target's
 *    tokens come from p^(N) by greedy or stochastic sampling.
 *
 * Every floating-point quantity is fp64. Weights, cached K/V and the
 * draft probabilities are inputs given as bf16 / fp32 and are upcast
 * exactly. Each output element is produced by one thread with a fixed
 * summation order, so results do not depend on the thread count.
 *
 * Parity pins are listed per function in oracle/msdo.c.
 */
#ifndef MSDO_H
#define MSDO_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
  int32_t layer_norm;   /* 0: RMSNorm, 1: LayerNorm                     */
  int32_t relu_ffn;     /* 0: SwiGLU FFN, 1: ReLU FFN                   */
  int32_t learned_pos;  /* 0: rotary positions, 1: learned position table */
  int32_t has_bias;     /* linear layers carry biases                   */
  double rope_theta, norm_eps;
} msdo_cfg;

/* Per-layer weights, bf16 bits, row-major [out][in]; unused entries NULL. */
typedef struct {
  const uint16_t *attn_g, *attn_b;
  const uint16_t *wq, *wk, *wv, *bq, *bk, *bv;
  const uint16_t *wo, *bo;
  const uint16_t *mlp_g, *mlp_b;
  const uint16_t *w_gate, *w_up, *b_up, *w_down, *b_down;
} msdo_layer_w;

typedef struct {
  const uint16_t *embed;      /* [V][d]                            */
  const uint16_t *pos_embed;  /* [P][d] or NULL                    */
  const uint16_t *final_g, *final_b;
  const uint16_t *lm_head;    /* [V][d]; the embedding when tied   */
} msdo_global_w;

/* x[i] = E[tok[i]] (+ P[pos[i]]). x is [n][d]. */
void msdo_embed(const msdo_cfg* c, const msdo_global_w* g, int32_t n, const int32_t* tok,
                const int32_t* pos, double* x);

/*
 * One decoder layer over a block of n rows of ONE sequence, in place on x.
 *  pos[i]        absolute position of row i.
 *  parent[i]     block topology (parent[0] = -1, parent[i] < i); row i
 *                attends to every key before the block and to the block rows
 *                that are its ancestors or itself.
 *  ctx_k/ctx_v   cached keys/values before the block, bf16 bits
 *                [n_kv_heads][ctx_stride][head_dim], rows [0, n_ctx).
 *  extra_k/v     further cached rows after the context, fp64
 *                [n_extra][n_kv_heads][head_dim] (rows an earlier call of
 *                this oracle produced and committed), may be NULL if 0.
 *  blk_k/blk_v   out: the block's own rotated keys / values, fp64
 *                [n][n_kv_heads][head_dim].
 *  kv_cache_bf16 1: the block's keys / values are stored in the cache's bf16
 *                format (nearest 8-bit significand, ties to even) before
 *                any row attends to them; 0: kept at fp64.
 * Key order for row i: context rows, extra rows, then block rows in slot
 * order (positions ascending).
 */
void msdo_layer(const msdo_cfg* c, const msdo_layer_w* w, int32_t n, double* x,
                const int32_t* pos, const int32_t* parent, int32_t n_ctx, int32_t ctx_stride,
                const uint16_t* ctx_k, const uint16_t* ctx_v, int32_t n_extra,
                const double* extra_k, const double* extra_v, double* blk_k, double* blk_v,
                int32_t kv_cache_bf16);

/* logits[i][v] = (W_LM norm_f(x_i))_v, [n][V]. */
void msdo_head(const msdo_cfg* c, const msdo_global_w* g, int32_t n, const double* x,
               double* logits);

/* Per row: the kappa largest logits (ties: smaller id first) and
 * log-softmax values logp = z - logsumexp(z); lse[i] is also returned. */
void msdo_topk(int32_t n, int32_t V, const double* logits, int32_t kappa, int32_t* ids,
               double* logp, double* lse);

enum { MSDO_GREEDY = 0, MSDO_REJECTION = 1, MSDO_MATCH = 2 };

/*
 * Acceptance for ONE sequence (App. B acceptance operator; Sec. 2 greedy
 * rule; stochastic rule per the readings listed in msdo.c).
 *  logits      [n][V] final-layer logits of the block rows.
 *  cand_ids/q  [n][n_cand] sparse draft law at each node (REJECTION only).
 *  u_accept    [n] uniform used when child c is tested (REJECTION).
 *  u_sample    [n] uniform used when sampling at node s (REJECTION/MATCH).
 *  tol_logit   logit tolerance of the near-tie bands (0: none flagged).
 * Out: *acc_len = A, *next_tok, path[0..A] (slot of the accepted node at each
 * depth; path[0] = 0). Near-tie bands (see msdo.c): *tie_depth = depth of
 * the first node where a decision choosing the way down (an argmax, a MATCH
 * draw, a REJECTION accept test) falls in a band, -1 if none; *tie_next = 1
 * if the decision that produced the next token falls in one. Returns 0, or
 * -1 if a child token has no draft mass at its parent (REJECTION).
 */
int32_t msdo_accept(int32_t n, const int32_t* parent, const int32_t* tokens, int32_t V,
                    const double* logits, int32_t mode, double temperature, int32_t n_cand,
                    const int32_t* cand_ids, const float* cand_q, const float* u_accept,
                    const float* u_sample, double tol_logit, int32_t* acc_len, int32_t* next_tok,
                    int32_t* path, int32_t* tie_depth, int32_t* tie_next);

/*
 * Commit for ONE sequence on bf16 caches [n_layers][n_kv_heads][cap][head_dim]:
 * rows len+path[r] move to len+r for r = 1..A (the root row stays at len);
 * returns the new committed length len + 1 + A.
 */
int32_t msdo_kv_commit(int32_t n_layers, int32_t n_kv_heads, int32_t cap, int32_t head_dim,
                       uint16_t* k, uint16_t* v, int32_t len, int32_t acc_len,
                       const int32_t* path);

#ifdef __cplusplus
}
#endif
#endif
