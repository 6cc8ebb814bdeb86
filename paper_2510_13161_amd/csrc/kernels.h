// Launch interfaces of the verification kernels (host side).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace msd {

// ---------------------------------------------------------------------------
// skinny weight-streaming GEMM: Y[M][N] = X[M][K] W^T, W [N][K] bf16
// ---------------------------------------------------------------------------
enum GemmMap : int32_t {
  MAP_PLAIN = 0,   // output column n <- row n of w0 (rows >= n0 are padding)
  MAP_QKV = 1,     // 64-wide tiles hold 32 rotary pairs of one q/k/v head
  MAP_GATEUP = 2,  // 64-wide tiles: 32 rows of w0 (gate) then the same 32 of w1 (up)
};

enum GemmEpi : int32_t {
  EPI_QKV = 0,     // (+bias) rotary, q -> q buffer, k/v -> cache slots
  EPI_RESID = 1,   // x[m][n] += y (+bias)
  EPI_SWIGLU = 2,  // act[m][f] = silu(gate) * up
  EPI_RELU = 3,    // act[m][n] = relu(y + bias)
  EPI_HEAD = 4,    // logits (+ per-tile max / sum-exp / top-kappa)
};

constexpr int kTileN = 64;   // output columns per workgroup tile
constexpr int kMaxMT = 9;    // up to 144 rows (9 MFMA row tiles)

struct GemmArgs {
  const float* A;      // fp32 activations [M][K]
  int32_t M, K, N;     // N = logical output columns (padding masked)
  int32_t n_tiles, splits;
  int32_t map;
  const uint16_t* w0;
  const uint16_t* w1;
  const uint16_t* w2;
  int32_t n_heads, n_kv_heads, head_dim;  // MAP_QKV
  float* partial;      // [splits][M][n_tiles*64] fp32 (splits > 1)
  int32_t* counters;   // [n_tiles], zero on entry, left zero on exit
  // epilogues
  const uint16_t* b0;  // bias of w0 (q / plain / up)
  const uint16_t* b1;  // bias of w1 (k)
  const uint16_t* b2;  // bias of w2 (v)
  float* x;            // EPI_RESID residual [M][N]
  float* out_f32;      // EPI_QKV q [M][H*hd]; EPI_SWIGLU / EPI_RELU act [M][F]
  uint16_t* k_cache;   // EPI_QKV this layer's [batch_cap][Hkv][cap][hd]
  uint16_t* v_cache;
  const int32_t* len;  // committed lengths [batch]
  uint32_t* status;
  int32_t capacity, n_slots;
  const float2* rope;  // [max_positions][hd/2] (cos, sin), or null
  int32_t rope_rows;
  // pre-norm fused into the A load: 0 none, 1 RMSNorm, 2 LayerNorm, from the
  // producer's per-segment (mean, M2) of each row: a_stats [a_stats_tiles][M]
  int32_t a_norm, a_stats_tiles;
  const float2* a_stats;
  const uint16_t* a_g;
  const uint16_t* a_b;
  float a_eps;
  float2* stats_out;   // EPI_RESID: [n_tiles][M] (mean, M2) of the updated rows
  int32_t weights_nt;  // stream weights with non-temporal loads
  float* logits;       // EPI_HEAD [M][N] or null
  float2* tile_ms;     // EPI_HEAD [n_tiles][M] (max, sum exp)
  uint64_t* tile_top;  // EPI_HEAD [n_tiles][M][kappa] rank keys
  int32_t kappa;
  int32_t depth[kMaxSlots];
};

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s);
// row-major [rows][K] -> fragment-major weight layout (src and dst distinct)
hipError_t launch_repack(const uint16_t* src, uint16_t* dst, int64_t rows, int32_t K,
                         hipStream_t s);

// ---------------------------------------------------------------------------
// embedding / norms
// ---------------------------------------------------------------------------
struct EmbedArgs {
  const int32_t* tokens;   // [M]
  const uint16_t* embed;   // [V][d]
  const uint16_t* pos_embed;
  int32_t embed_frag;      // the table is stored fragment-major (tied LM head)
  const int32_t* len;
  int32_t M, d, n_slots, max_positions, vocab;
  uint32_t* status;        // MSD_DEV_TOKEN on an id outside [0, vocab)
  float* x;                // [M][d]
  float2* stats;           // [M] (mean, M2) of each embedded row
  int32_t* zero_i32;       // counters to clear
  int64_t n_zero;
  int32_t depth[kMaxSlots];
};
hipError_t launch_embed(const EmbedArgs& a, hipStream_t s);

// (mean, M2) of each row of x [M][d] (one segment per row)
hipError_t launch_row_stats(const float* x, int M, int d, float2* stats, hipStream_t s);
hipError_t launch_zero_i32(int32_t* p, int64_t n, hipStream_t s);

// ---------------------------------------------------------------------------
// verify attention
// ---------------------------------------------------------------------------
constexpr int kMaxAttnSpans = 512;    // key spans per (sequence, kv head)
constexpr int kMaxCapacity = 32768;   // cache positions

struct AttnArgs {
  const float* q;           // fp32 [M][H][hd] (rotated)
  const uint16_t* k_cache;  // this layer [batch_cap][Hkv][cap][hd]
  const uint16_t* v_cache;
  const int32_t* len;
  uint32_t* status;
  float* out;               // fp32 [M][H*hd]
  float* part_o;            // [batch][Hkv][max_spans][Qn][hd]
  float* part_ml;           // [batch][Hkv][max_spans][Qn][2] (max, sum exp)
  int32_t batch, n_heads, n_kv_heads, capacity, n_slots;
  int32_t span, max_spans;  // keys per wave (multiple of 64), spans per sequence
  float scale;
  Topo topo;
};
hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// head merge (per row): top-kappa, argmax, logsumexp
// ---------------------------------------------------------------------------
struct HeadMergeArgs {
  const float2* tile_ms;
  const uint64_t* tile_top;
  int32_t n_tiles, M, kappa;
  int32_t* ids;    // [M][kappa] or null
  float* logp;     // [M][kappa] or null
  int32_t* argmax; // [M] or null
  float* lse;      // [M] or null
};
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
  uint32_t* status;
  Topo topo;
};
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

}  // namespace msd
