// Launch interfaces of the verification kernels (host side).
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

#include "common.h"

namespace msd {

// ---------------------------------------------------------------------------
// skinny weight-streaming GEMM: Y[M][N] = norm(X)[M][K] W^T, W [N][K] bf16
// ---------------------------------------------------------------------------
enum GemmMap : int32_t {
  MAP_PLAIN = 0,   // output column n <- row n of w0 (rows >= N are padding)
  MAP_QKV = 1,     // 64-wide tiles hold 32 rotary pairs of one q/k/v head
  MAP_GATEUP = 2,  // a tile: 8 jt rows of w0 (gate), then the same 8 jt rows of w1 (up)
};

enum GemmEpi : int32_t {
  EPI_QKV = 0,     // (+bias) rotary, q -> q buffer, k/v -> cache slots
  EPI_RESID = 1,   // x[m][n] += y (+bias), row statistics, images of x
  EPI_SWIGLU = 2,  // act = silu(gate) * up -> activation image
  EPI_RELU = 3,    // act = relu(y + bias) -> activation image
  EPI_HEAD = 4,    // logits (+ per-tile max / sum-exp / top-kappa)
};

constexpr int kTileN = 64;   // output columns per tile
constexpr int kMaxMT = 9;    // up to 144 rows (9 MFMA row tiles)

// Pre-norm of the GEMM input, applied after the product: the input image
// holds x * g (the norm gain folded in by its producer), so
//   RMSNorm:   y = r * (W (x g))                    r = 1 / sqrt(mean x^2 + eps)
//   LayerNorm: y = r * (W (x g)) - r mu c + e       r = 1 / sqrt(var x + eps)
// with c = W g and e = W b per output column, and (mu, var) rebuilt from the
// producer's per-64-column (mean, M2) summaries.
struct RowNorm {
  int32_t kind;            // 0 none, 1 RMSNorm, 2 LayerNorm
  const float2* stats;     // [tiles][M] (mean, M2) over 64-column tiles
  int32_t tiles;           // = K / 64
  float eps;
  const float* col_g;      // LayerNorm: c [N]
  const float* col_b;      // LayerNorm: e [N]
};

// An activation image an epilogue writes, with an optional per-column gain.
struct ImageOut {
  uint16_t* img;
  const uint16_t* gain;
};

struct GemmArgs {
  const uint16_t* a_img;   // input image [K/32][MT][2][64][8]
  int32_t M, MT, K, N;     // N = logical output columns (padding masked)
  int32_t n_tiles, splits, waves;
  int32_t jt;              // 16-column sub-tiles per tile: 4 (64 columns), 8 (128
                           // columns: EPI_SWIGLU with up to 3 row tiles and 2 waves,
                           // EPI_HEAD with one row tile and 4 waves) or 2 (32 columns:
                           // EPI_QKV with one row tile and 8 waves)
  int32_t wg_tiles;        // 64-column tiles per workgroup: 1, or 4 (2 to 9 row tiles:
                           // one compute wave a tile and a wave that stages the
                           // activation through LDS; then waves = 4, and with
                           // splits > 1 a second kernel sums the splits and runs
                           // the epilogue)
  int32_t map;
  const uint16_t* w0;
  const uint16_t* w1;
  const uint16_t* w2;
  int32_t n_heads, n_kv_heads, head_dim;  // MAP_QKV
  float* partial;          // [n_tiles][splits][MT * jt * 256] (splits > 1)
  int32_t* counters;       // [n_tiles], zero on entry, left zero on exit
  RowNorm norm;
  const uint16_t* b0;      // bias of w0 (q / plain / up)
  const uint16_t* b1;      // bias of w1 (k)
  const uint16_t* b2;      // bias of w2 (v)
  // EPI_RESID
  float* x;                // residual [M][N]
  float2* stats_out;       // [n_tiles][M] (mean, M2) of the updated rows
  ImageOut img_out[2];     // images of the updated x (K = N)
  // EPI_QKV
  uint16_t* q_img;         // q as the attention's split-bf16 operand image:
                           // [batch][Hkv][q_tiles][hd/32][hi|lo][64 lanes][8]; lane l
                           // of tile qt: query qt*16 + l%16 (= gq*n_slots + slot of
                           // head kvh*G + gq), dims 32 kk + 8 (l/16) .. +8
  int32_t q_tiles;         // 16-query tiles per kv head: ceil(G * n_slots / 16)
  uint16_t* k_cache;       // this layer's [batch_cap][Hkv][cap][hd]
  uint16_t* v_cache;
  const int32_t* len;      // committed lengths [batch]
  uint32_t* status;
  int32_t capacity, n_slots;
  const float2* rope;      // [max_positions][hd/2] (cos, sin), or null
  int32_t rope_rows;
  int32_t depth[kMaxSlots];
  // EPI_SWIGLU / EPI_RELU
  uint16_t* act_img;       // image of the activation (K = d_ffn)
  // EPI_HEAD
  float* logits;           // [M][N] or null
  float2* tile_ms;         // [n_tiles][M] (max, sum exp)
  uint64_t* tile_top;      // [n_tiles][M][kappa] rank keys
  int32_t kappa;
};

// HIP events attached to a launch (hipExtLaunchKernel): start is stamped when
// the first kernel of the launch begins, stop when its last one ends, so they
// time the kernels themselves, not the queue around them. Null: none.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s, LaunchEvents ev = {});
// row-major [rows][K] -> k-step-major weight fragments (src and dst distinct)
hipError_t launch_repack(const uint16_t* src, uint16_t* dst, int64_t rows, int32_t K,
                         hipStream_t s);
// c[n] = sum_k W[n][k] g[k] (and e with b) for a row-major bf16 matrix, fp64
// accumulation, fp32 out; b may be null.
hipError_t launch_colsum(const uint16_t* w, int64_t rows, int32_t K, const uint16_t* g,
                         const uint16_t* b, float* c, float* e, hipStream_t s);

// ---------------------------------------------------------------------------
// block rows -> residual, statistics and image
// ---------------------------------------------------------------------------
struct RowsArgs {
  // source of row m: hidden[m] (fp32, if non-null) or E[tokens[m]] (+ P[pos])
  const float* hidden;
  const int32_t* tokens;   // [M]
  const uint16_t* embed;   // [V][d]
  const uint16_t* pos_embed;
  int32_t embed_frag;      // the table is stored as k-step-major fragments (tied LM head)
  const int32_t* len;
  int32_t M, MT, d, n_slots, max_positions, vocab;
  uint32_t* status;        // MSD_DEV_TOKEN on an id outside [0, vocab)
  float* x;                // [M][d] (may be null with hidden)
  float2* stats;           // [d/64][M] (mean, M2)
  ImageOut img;            // image of the rows (K = d)
  uint16_t* zero_img;      // another image whose padding rows are cleared
  int32_t zero_img_k;
  int32_t* zero_i32;       // counters to clear
  int64_t n_zero;
  int32_t depth[kMaxSlots];
};
hipError_t launch_rows(const RowsArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// verify attention
// ---------------------------------------------------------------------------
constexpr int kMaxAttnChunks = 128;   // key chunks per (sequence, kv head)
constexpr int kMaxCapacity = 32768;   // cache positions
constexpr int kAttnChunk = 256;       // keys per workgroup (4 waves x 64)

struct AttnArgs {
  const uint16_t* q_img;    // rotated q as operand image (GemmArgs::q_img), padding rows unset
  const uint16_t* k_cache;  // this layer [batch_cap][Hkv][cap][hd]
  const uint16_t* v_cache;
  const int32_t* len;
  uint32_t* status;
  uint16_t* out_img;        // image of the output (K = H * hd)
  int32_t MT;
  int32_t* counters;        // [batch][Hkv][query-tile groups]: zero on entry, left zero
  float* part_o;            // [batch][Hkv][chunks][Qn][hd]
  float* part_ml;           // [batch][Hkv][chunks][Qn][2] (max of score * log2 e, sum exp2)
  int32_t batch, n_heads, n_kv_heads, capacity, n_slots;
  int32_t max_chunks;       // 256-key chunks of the longest sequence
  int32_t q_per_wg;         // query tiles a workgroup takes in turn (its K and V
                            // operands loaded once for all of them)
  int32_t nb;               // 256-key spans per workgroup chunk: 1, or more for the
                            // streaming kernel (then q_per_wg <= 3)
  float scale;
  int32_t defer;            // 1: chunks only publish their partials; a second
                            // kernel merges them (no in-kernel hand-off)
  int32_t ring;             // 1: attn_ring_kernel (head dim 128, chunks of nb spans,
                            // q_per_wg <= 4 tiles a workgroup)
  Topo topo;
};
hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t s);
// the deferred chunk merge (after launch_attention with a.defer = 1, same args)
hipError_t launch_attention_merge(int head_dim, const AttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// head merge (per row): top-kappa, argmax, logsumexp
// ---------------------------------------------------------------------------
struct HeadMergeArgs {
  const float2* tile_ms;
  const uint64_t* tile_top;
  int32_t n_tiles, M, kappa;
  float2* part_ms;     // [M][parts] (parts = head_parts(n_tiles))
  uint64_t* part_top;  // [M][parts][kappa]
  int32_t* ids;    // [M][kappa] or null
  float* logp;     // [M][kappa] or null
  int32_t* argmax; // [M] or null
  float* lse;      // [M] or null
};
int head_parts(int n_tiles);  // 256 tiles per part, at most 64 parts
hipError_t launch_head_merge(const HeadMergeArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// acceptance and commit
// ---------------------------------------------------------------------------
struct AcceptArgs {
  int32_t mode;
  float temperature;
  int32_t batch, n_slots, vocab, n_cand;
  const int32_t* tokens;     // [batch][n_slots]
  const float* logits;       // [M][V]
  const int32_t* argmax;     // [M]
  const int32_t* cand_ids;   // [batch][n_slots][n_cand]
  const float* cand_q;
  const float* u_accept;     // [batch][n_slots]
  const float* u_sample;
  int32_t* acc_len;
  int32_t* next_tok;
  int32_t* path;             // [batch][n_slots]
  uint8_t* near_tie;         // [batch] or null
  float tol_logit;           // half-width scale of the near-tie bands
  uint32_t* status;
  double2* stats;            // [M][kAcceptStatChunks] (max of z / T, sum exp(z / T - max))
                             // per vocabulary chunk, or null (the walk's own passes)
  Topo topo;
};
constexpr int kAcceptStatChunks = 64;
hipError_t launch_accept(const AcceptArgs& a, hipStream_t s);

struct CommitArgs {
  uint16_t* k_cache;         // [L][batch_cap][Hkv][cap][hd]
  uint16_t* v_cache;
  int32_t* len;
  const int32_t* acc_len;
  const int32_t* path;
  int32_t n_layers, batch, batch_cap, n_kv_heads, capacity, head_dim, n_slots;
  int32_t copy_rows;         // 0 for a chain (rows already in place)
};
hipError_t launch_commit(const CommitArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// reuse criterion, next-window selection, fallback statistics
// ---------------------------------------------------------------------------
constexpr int kMaxTreeNodes = 256;

struct TreeTopo {
  int16_t parent[kMaxTreeNodes];  // -1 = root
  uint8_t depth[kMaxTreeNodes];   // roots 1
  int32_t n_nodes;
};

struct ReuseStats {  // layout of msd_reuse_stats
  uint64_t trials, fallbacks, fallbacks_tau1, omega_trials;
  double omega_sum;
};

struct ReuseArgs {
  int32_t batch, n_slots;
  const int32_t* tokens;       // the verified block [batch][n_slots]
  const int32_t* acc_len;      // [batch]
  const int32_t* next_tok;     // [batch]
  const int32_t* path;         // [batch][n_slots]
  const int32_t* tree_tokens;  // [batch][n_nodes]
  const float* logits;         // [M][vocab] or null (no Omega)
  const float* lse;            // [M]
  const int32_t* ee_ids;       // [M][kappa]
  int32_t kappa, vocab;
  int32_t* next_case;          // [batch]
  int32_t* next_node;          // [batch]
  float* omega;                // [batch] or null
  ReuseStats* stats;           // or null
  TreeTopo tree;
};
hipError_t launch_reuse(const ReuseArgs& a, hipStream_t s);

}  // namespace msd
