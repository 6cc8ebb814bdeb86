/*
 * msd.h — C ABI of the Mirror-SD verification step on MI355X (gfx950).
 *
 * Mirror Speculative Decoding (arXiv 2510.13161) overlaps a draft model with
 * the target's verification pass. This library is the target side of one
 * decoding step, on one GPU:
 *
 *   msd_verify_block     Sec. 2 (speculative verification: one teacher-forced
 *                        pass of the target over the draft window) and
 *                        Sec. 3.1 (the window may be the branch-complete
 *                        hypothesis tree; a depth-r node holds the token at
 *                        position t + r). Emits the early-exit message on the
 *                        way (Sec. 3.1: p^(l_e) = Softmax(W_LM h^(l_e)),
 *                        M_t = Top-kappa(p^(l_e)) = {(v_i, log p_i)}).
 *   msd_early_exit_topk  the Sec. 3.1 token channel on its own, from a residual.
 *   msd_accept           App. B acceptance operator: the longest verified
 *                        prefix A_t, the accepted path and the next token
 *                        (Sec. 2 greedy rule; stochastic rules, see below).
 *   msd_kv_commit        Sec. 2: commit the accepted tokens (and the root) to
 *                        the KV cache; everything else rolls back.
 *   msd_reuse_select     Sec. 3.1 reuse criterion and next-window selection,
 *                        App. E fallback statistics.
 *
 * Conventions
 *  - Every pointer marked "device" is HIP device memory owned by the caller;
 *    "host" pointers are read during the call only. The library never takes
 *    ownership of caller memory; it allocates device memory only in
 *    msd_model_create (the rotary table; for LayerNorm models the column
 *    sums of the matrices that consume a LayerNorm output; a staging buffer
 *    for the weight rearrangement, freed before it returns) and never per
 *    call.
 *  - All work is enqueued asynchronously on the caller's `stream`; nothing
 *    blocks, nothing throws across the ABI. The per-step calls (everything
 *    but msd_model_create / msd_model_destroy) allocate nothing, issue no
 *    memset and never wait on the host, so they can be captured in a HIP
 *    graph; msd_model_create synchronises the device and cannot.
 *  - Host-checkable errors (NULL pointers, sizes out of range, topology that
 *    is not a forest in slot order, workspace too small) return a negative
 *    msd_status and enqueue nothing; msd_last_error() then describes it.
 *  - Device-detected errors (a committed length plus the block exceeding the
 *    cache capacity; a draft token outside its parent's candidate set) set a
 *    non-zero code in the caller's device status word and the affected
 *    sequence's outputs are left unspecified.
 *  - Row-major everywhere. bf16 = IEEE binary16-brain, stored as 16 bits.
 */
#ifndef MSD_H
#define MSD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MSD_OK = 0,
  MSD_ERR_INVALID_ARG = -1, /* NULL pointer or out-of-range scalar             */
  MSD_ERR_SHAPE = -2,       /* shapes the kernels do not support               */
  MSD_ERR_CAPACITY = -3,    /* block does not fit the cache (host-detectable)  */
  MSD_ERR_UNSUPPORTED = -4, /* mode / option not available                     */
  MSD_ERR_WORKSPACE = -5,   /* workspace NULL or smaller than required         */
  MSD_ERR_HIP = -6          /* a HIP runtime call failed                       */
} msd_status;

/* Device status word codes (OR-ed in by kernels). */
#define MSD_DEV_CAPACITY 1u  /* len[b] + n_slots > capacity                    */
#define MSD_DEV_CANDIDATE 2u /* REJECTION: child token without draft mass      */
#define MSD_DEV_TOKEN 4u     /* a block token outside [0, vocab)               */

/* Thread-local text of the last non-OK status returned on this thread. */
const char* msd_last_error(void);

enum { MSD_NORM_RMS = 0, MSD_NORM_LAYER = 1 };
enum { MSD_ACT_SWIGLU = 0, MSD_ACT_RELU = 1 };
enum { MSD_POS_ROPE = 0, MSD_POS_LEARNED = 1 };

/*
 * Decoder-only target (Sec. 2: p(y_t | .) = Softmax(W h_t)): n_layers pre-norm
 * blocks (attention, then FFN), a final norm and the LM head.
 *  norm          RMSNorm (x / sqrt(mean x^2 + eps) * g) or LayerNorm.
 *  act           SwiGLU (down(silu(gate h) * up h)) or ReLU (down(relu(up h + b)) + b).
 *  pos           rotary (rotate-half pairs (j, j + head_dim/2), angle
 *                pos * rope_theta^(-2j/head_dim)) or a learned table added to
 *                the embedding.
 *  max_positions largest position + 1 the model will see (rotary table size /
 *                learned table rows).
 * Limits: head_dim in {64, 128}; n_heads % n_kv_heads == 0; d_model,
 * n_heads*head_dim and d_ffn multiples of 64; vocab >= 64 and a multiple of 16.
 */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
  int32_t norm, act, pos, has_bias, tied_head;
  int32_t max_positions;
  float rope_theta, norm_eps;
} msd_model_config;

/* Tensor slots. All tensors are device bf16, row-major [out][in] for
 * matrices. Absent tensors (biases without has_bias, LayerNorm shifts with
 * RMSNorm, the learned table with rotary positions, the gate with ReLU, the
 * separate head when tied) are NULL. */
enum {
  MSD_T_EMBED = 0,     /* [vocab][d_model]                              */
  MSD_T_POS_EMBED,     /* [max_positions][d_model]   (learned only)     */
  MSD_T_FINAL_G,       /* [d_model]                                     */
  MSD_T_FINAL_B,       /* [d_model]                  (LayerNorm only)   */
  MSD_T_LM_HEAD,       /* [vocab][d_model]           (NULL when tied)   */
  MSD_T_GLOBAL_COUNT
};
enum {
  MSD_L_ATTN_G = 0, MSD_L_ATTN_B,
  MSD_L_WQ,          /* [n_heads*head_dim][d_model]     */
  MSD_L_WK,          /* [n_kv_heads*head_dim][d_model]  */
  MSD_L_WV,          /* [n_kv_heads*head_dim][d_model]  */
  MSD_L_BQ, MSD_L_BK, MSD_L_BV,
  MSD_L_WO,          /* [d_model][n_heads*head_dim]     */
  MSD_L_BO,
  MSD_L_MLP_G, MSD_L_MLP_B,
  MSD_L_W_GATE,      /* [d_ffn][d_model]  (SwiGLU)      */
  MSD_L_W_UP,        /* [d_ffn][d_model]                */
  MSD_L_B_UP,        /* [d_ffn]           (ReLU)        */
  MSD_L_W_DOWN,      /* [d_model][d_ffn]                */
  MSD_L_B_DOWN,      /* [d_model]         (ReLU)        */
  MSD_L_COUNT
};
#define MSD_TENSOR_INDEX(layer, slot) (MSD_T_GLOBAL_COUNT + (layer) * MSD_L_COUNT + (slot))
#define MSD_N_TENSORS(n_layers) (MSD_T_GLOBAL_COUNT + (n_layers) * MSD_L_COUNT)

typedef struct msd_model msd_model;

/* Validates the configuration and tensor table (n_tensors must equal
 * MSD_N_TENSORS(n_layers)) and builds the model on the current HIP device.
 * The tensors stay caller-owned and must outlive the model.
 * Weight layout: the call rearranges every projection matrix (q, k, v, o,
 * gate, up, down and the LM head; the embedding too when tied) IN PLACE into
 * the library's k-step-major layout (for each 32-column k-step, the 1 KB
 * MFMA operands of all 16-row groups one after the other), so the
 * workgroups of a projection, which advance through K together, read one
 * contiguous window of HBM.
 * After the call those tensors are opaque to the caller, and one set of
 * tensors can back only one model. The call synchronises the device and
 * briefly allocates a temporary buffer the size of the largest matrix.
 * Launch-shape overrides, read from the environment here (tuning and tests;
 * results differ only by floating-point summation order): MSD_GEMM_TARGET_WGS
 * (split-K sized for about this many workgroups per GEMM; unset, for the
 * best balance over the device's compute units), MSD_GEMM_WAVES (4 or 8),
 * MSD_QKV_JT (the QKV projection's tile width at one row tile in 16-column
 * sub-tiles: 2 unset, whole K; 4: 64-column tiles with splits of K) and
 * MSD_ATTN_SPANS (256-key spans per attention workgroup: 1 forces the
 * one-span kernel, 2 or more the ring-fed one at head dim 128, else the
 * streaming one; unset, chosen per call), MSD_ATTN_RING (0: the streaming
 * kernel also at head dim 128; 1 unset),
 * MSD_ATTN_DEFER (the attention's chunk merge in a kernel of its own: 1
 * always, 0 never; unset, from 6 chunks on),
 * MSD_ROWS_MIN_MT (row tiles from which GEMMs with 256 or more 64-column
 * tiles may run the kernel that shares the activation through LDS: 3 unset;
 * it runs where its workgroups balance the compute units),
 * MSD_ROWS_MIN_TILES (forces that kernel on GEMMs with at least this many
 * tiles), MSD_ROWS_MAX_SPLITS (its splits of K at most, 4 unset) and
 * MSD_ROWS_NARROW (narrower GEMMs of 3 or more row tiles in that kernel
 * with many splits and their split sum and epilogue in a second kernel: 0
 * never, 2 at any size; unset, for matrices of 32M weights or more) and
 * MSD_ROWS_NARROW_MT (the row tiles from which that applies: 3 unset). */
msd_status msd_model_create(const msd_model_config* cfg, const void* const* tensors,
                            int32_t n_tensors, msd_model** out);
void msd_model_destroy(msd_model* model);

/* KV cache, device bf16 [n_layers][batch_cap][n_kv_heads][capacity][head_dim]
 * for k and v; len[b] (device int32) = committed positions of sequence b.
 * The block's rows go to positions len[b] + slot. */
typedef struct {
  void* k;
  void* v;
  int32_t* len;       /* device [batch_cap]                                  */
  uint32_t* status;   /* device word; kernels OR MSD_DEV_* codes into it     */
  int32_t batch_cap, capacity;
} msd_kv_cache;

/* Draft block shared by every sequence of the batch.
 * Slot 0 is the root: the last committed token, not yet in the cache, at
 * position len[b]; slot i sits at position len[b] + depth(i).
 * parent == NULL means a chain (parent[i] = i - 1); otherwise parent[0] = -1
 * and 0 <= parent[i] < i. */
typedef struct {
  int32_t batch, n_slots;   /* 1 <= n_slots <= 64, batch <= batch_cap;
                               batch * n_slots <= 144 for msd_verify_block */
  const int32_t* tokens;    /* device [batch][n_slots]                     */
  const int32_t* parent;    /* host [n_slots] or NULL                      */
} msd_block;

/* Early-exit request: after layer `layer` (1-indexed, 1 <= layer <= n_layers-1)
 * write, for every block row, the kappa (1..32) most likely tokens under the
 * final-normed LM head (ties: smaller id first) and their log-probabilities
 * (log-softmax over the full vocabulary). If `ready` is non-NULL it is
 * recorded on the stream once ids/logp are complete. */
typedef struct {
  int32_t layer;
  int32_t kappa;
  int32_t* ids;       /* device [batch*n_slots][kappa] */
  float* logp;        /* device [batch*n_slots][kappa] */
  hipEvent_t ready;
} msd_ee_request;

/* Workspace needed by msd_verify_block / msd_early_exit_topk / msd_accept
 * for this batch, block size, kappa and cache capacity. */
size_t msd_workspace_bytes(const msd_model* model, int32_t batch, int32_t n_slots,
                           int32_t kappa, int32_t capacity);

/*
 * Verification pass of the target over the block (Sec. 2; Sec. 3.1 tree).
 * Writes the block's K/V into the cache after len[b] (len is not changed:
 * only msd_kv_commit advances it). Outputs, rows m = b*n_slots + slot:
 *  logits  device fp32 [M][vocab] final-layer logits, or NULL
 *  argmax  device int32 [M] (ties: smaller id), required
 *  lse     device fp32 [M] logsumexp of the logits, or NULL
 *  ee      early-exit request, or NULL
 * ws must hold msd_workspace_bytes(model, batch, n_slots, kappa, capacity).
 */
msd_status msd_verify_block(const msd_model* model, msd_kv_cache* kv, const msd_block* block,
                            const msd_ee_request* ee, float* logits, int32_t* argmax,
                            float* lse, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * msd_verify_block without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same kernels and outputs, with the scratch in a
 * static device array of the library, MSD_STATIC_SCRATCH_BYTES (64 MiB) per
 * GPU, held from the first msd_model_create on that GPU until the process
 * ends. The call allocates nothing. A block whose workspace
 * (msd_workspace_bytes) exceeds that size returns MSD_ERR_WORKSPACE and
 * enqueues nothing: the 14B-shaped chain and tree blocks and the 66B-shaped
 * tree fit, long-context batches (batch 16 at 8K contexts) do not. Every call
 * on one GPU shares its scratch, which keeps the last call's contents (the
 * kernels clear what must start at zero): calls that overlap on one GPU,
 * from different streams or threads, race and must be ordered by the caller.
 */
#define MSD_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
msd_status msd_verify_block_static(const msd_model* model, msd_kv_cache* kv, const msd_block* block,
                                   const msd_ee_request* ee, float* logits, int32_t* argmax,
                                   float* lse, hipStream_t stream);

/*
 * Token channel of Sec. 3.1 from a residual: hidden is device fp32 [M][d_model]
 * (the residual stream after some layer); applies the final norm and the LM
 * head and writes the kappa best ids and log-probabilities per row.
 */
msd_status msd_early_exit_topk(const msd_model* model, const float* hidden, int32_t M,
                               int32_t kappa, int32_t* ids, float* logp, void* ws,
                               size_t ws_bytes, hipStream_t stream);

enum { MSD_GREEDY = 0, MSD_REJECTION = 1, MSD_MATCH = 2 };

/*
 * Sampling inputs of the stochastic rules (unused by MSD_GREEDY).
 * REJECTION: at a node whose children were drawn from the sparse draft law
 * q (cand_ids/cand_q at that node) without replacement, child x is accepted
 * iff u_accept[child] < min(1, r(x)/q(x)); after a rejection
 * r <- normalise((r - q)^+) and x leaves q; if every child is rejected the
 * next token is drawn from r with u_sample[node] (inverse CDF over ids
 * ascending); r starts as p = Softmax(logits / temperature). With a single
 * child this is Leviathan et al. 2023; it leaves the target law intact.
 * MATCH: the paper's sample-and-compare (Sec. 3.1, App. B): y is drawn from p
 * with u_sample[node]; descend to the child carrying y, else y is next.
 * tol_logit: logit tolerance of the near-tie flags (any mode; >= 0).
 */
typedef struct {
  int32_t mode;
  float temperature;
  int32_t n_cand;           /* <= 64                                       */
  const int32_t* cand_ids;  /* device [batch][n_slots][n_cand]             */
  const float* cand_q;      /* device [batch][n_slots][n_cand], rows sum 1 */
  const float* u_accept;    /* device [batch][n_slots] in [0, 1)           */
  const float* u_sample;    /* device [batch][n_slots] in [0, 1)           */
  float tol_logit;
} msd_sampling;

/*
 * App. B acceptance operator over the verified block, per sequence:
 *  acc_len  device int32 [batch]  A_b = accepted draft tokens (depth reached)
 *  next_tok device int32 [batch]  correction (mismatch) or bonus token
 *  path     device int32 [batch][n_slots]; path[b][r] = slot accepted at depth r,
 *           path[b][0] = 0; entries after A_b are -1
 *  near_tie device uint8 [batch] or NULL: 1 when some decision of the walk
 *           lies where a logit error of tol_logit could flip it, else 0.
 *           Bands: GREEDY, a visited row whose top-1 minus top-2 logit is
 *           below 2 tol; REJECTION, an accept test with |u - alpha| <
 *           2 tol alpha / T; an inverse-CDF draw (REJECTION, MATCH) with
 *           |u - c| < 4 tol min(c, 1 - c) at either edge c (cumulative
 *           fraction) of the drawn id's bin. tol is sampling->tol_logit (0
 *           when sampling is NULL: nothing is flagged); GREEDY flags read
 *           logits.
 * GREEDY reads argmax only (children tried in slot order); the stochastic
 * modes read logits (fp32 [M][vocab]). sampling may be NULL for GREEDY.
 * status: device word for MSD_DEV_CANDIDATE, may be NULL for GREEDY and MATCH.
 * ws / ws_bytes: optional device scratch, 16-byte aligned. For REJECTION and
 * MATCH with ws_bytes >= batch * n_slots * MSD_ACCEPT_WS_PER_ROW, per-row
 * vocabulary statistics (64 chunks of fp64 max and sum) are computed there by
 * a kernel spread over the device, and the walk reads the logsumexp and the
 * inverse-CDF chunk masses from them (scanning only the drawn chunk);
 * otherwise (NULL, or smaller) one workgroup per sequence makes the
 * vocabulary passes itself. The decisions are the same either way up to
 * fp64 summation order (inside the near-tie bands). GREEDY ignores ws.
 */
#define MSD_ACCEPT_WS_PER_ROW 1024
msd_status msd_accept(const msd_model* model, const msd_block* block, const float* logits,
                      const int32_t* argmax, const msd_sampling* sampling, int32_t* acc_len,
                      int32_t* next_tok, int32_t* path, uint8_t* near_tie, uint32_t* status,
                      void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Commit / rollback (Sec. 2): for every layer, row len[b] + path[b][r] of
 * the cache moves to len[b] + r for r = 1..A_b, then len[b] += 1 + A_b (the
 * root and the accepted tokens). Rows past the new length are stale.
 */
msd_status msd_kv_commit(const msd_model* model, msd_kv_cache* kv, const msd_block* block,
                         const int32_t* acc_len, const int32_t* path, hipStream_t stream);

/*
 * Reuse criterion and next-window selection (Sec. 3.1, "Verification vs.
 * reuse criterion" and "Operational selection of the next window") with the
 * fallback statistics of App. E.
 *
 * The hypothesis tree T_t is what the draft built from the early-exit top-k
 * roots: node i at depth d_i (roots d = 1) holds the token for position
 * t + d_i, where position t + 1 is the one the current block's root row
 * predicts. Topology is shared by the batch, tokens are per sequence.
 */
#define MSD_MAX_TREE_NODES 256
typedef struct {
  int32_t n_nodes;          /* 1 <= n_nodes <= MSD_MAX_TREE_NODES            */
  const int32_t* parent;    /* host [n_nodes]; -1 = root, else 0 <= p < i   */
  const int32_t* tokens;    /* device [batch][n_nodes]                       */
} msd_hyp_tree;

enum { MSD_NEXT_BRANCH = 0, MSD_NEXT_CONTINUE = 1, MSD_NEXT_FRESH = 2 };

/* Running fallback statistics (device memory, zeroed once by the caller and
 * accumulated by every call; calls sharing one must be stream-ordered).
 * One trial = one sequence of one step. FF = fallbacks / trials; the mean
 * overlap mass is omega_sum / omega_trials (App. E: FF <= 1 - Omega). */
typedef struct {
  uint64_t trials;
  uint64_t fallbacks;        /* F_t = 1: fresh rollout                        */
  uint64_t fallbacks_tau1;   /* of which A_t = 0                              */
  uint64_t omega_trials;     /* trials with Omega computed                    */
  double omega_sum;
} msd_reuse_stats;

/*
 * Per sequence b, with A = acc_len[b], tau = A + 1 and the corrected prefix
 * Pi+ = (tokens of the accepted slots path[b][1..A], next_tok[b]):
 * reuse iff Pi+ is the token sequence of a root-to-node path of T_t ending at
 * depth tau. Writes
 *  next_case device int32 [batch]: MSD_NEXT_BRANCH (A = 0 and a root carries
 *            the correction: the branch under that root is the next window),
 *            MSD_NEXT_CONTINUE (A >= 1 and Pi+ is a path: the continuation
 *            below its node), MSD_NEXT_FRESH (fallback: a fresh rollout)
 *  next_node device int32 [batch]: the matched node (smallest index when
 *            several match), -1 on fallback.
 * Omega (optional, all of logits, lse, ee_ids non-NULL): the overlap mass at
 * the root row, Omega_k = sum over the early-exit top-k ids of
 * softmax(logits)[id] (Sec. 3.1, sampling width at early exit; App. E),
 * fp64 accumulation, written to omega[b] if
 * omega is non-NULL; logits/lse/ee_ids are the verify call's outputs
 * ([M][vocab], [M], [M][kappa]). stats may be NULL.
 */
msd_status msd_reuse_select(const msd_model* model, const msd_block* block, const int32_t* acc_len,
                            const int32_t* next_tok, const int32_t* path, const msd_hyp_tree* tree,
                            const float* logits, const float* lse, const int32_t* ee_ids,
                            int32_t kappa, int32_t* next_case, int32_t* next_node, float* omega,
                            msd_reuse_stats* stats, hipStream_t stream);

/*
 * Instrumentation (benchmarking only): when set, msd_verify_block times the
 * launch of kernel class `kclass` in layer i (i < n; classes: 0 QKV
 * projection, 1 attention, 2 output projection, 3 FFN up projection, 4 FFN
 * down projection) with begin[i] / end[i]: for the projections the events
 * are attached to the kernel dispatch itself (begin stamped when its first
 * kernel starts, end when its last one ends: the kernels' own duration);
 * for attention they are recorded on the stream around its launches. The events are
 * caller-owned HIP events; a NULL pair skips that layer (sampling a few
 * layers keeps the events' own cost low); pass n = 0 to switch it off. Not
 * thread-safe with concurrent verify calls on the same model.
 */
enum { MSD_K_QKV = 0, MSD_K_ATTN = 1, MSD_K_OPROJ = 2, MSD_K_FFN_UP = 3, MSD_K_FFN_DOWN = 4 };
msd_status msd_set_profile(msd_model* model, int32_t kclass, hipEvent_t* begin, hipEvent_t* end,
                           int32_t n);

#ifdef __cplusplus
}
#endif
#endif /* MSD_H */
