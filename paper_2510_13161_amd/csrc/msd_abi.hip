// C ABI of the verification step (include/msd.h): argument checks, block
// topology preparation, workspace layout and the launch sequence. Every call
// is asynchronous on the caller's stream and allocates nothing.
#include <stdlib.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "msd.h"

using namespace msd;

static_assert(sizeof(msd_reuse_stats) == sizeof(ReuseStats), "reuse statistics layout");
static_assert(MSD_MAX_TREE_NODES == kMaxTreeNodes, "hypothesis tree bound");

// Scratch of msd_verify_block_static, for callers that cannot allocate: one
// copy per GPU, held by the loaded code object until the process ends. Host
// code never uses this name as an address (on the host it is a stand-in);
// the device address comes from hipGetSymbolAddress, per device.
constexpr size_t kStaticScratchBytes = MSD_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

struct msd_model {
  msd_model_config cfg;
  void* scratch = nullptr;         // this device's copy of `scratch` (msd_verify_block_static)
  std::vector<const uint16_t*> t;  // MSD_N_TENSORS(n_layers) entries
  float2* rope = nullptr;          // [max_positions][head_dim/2] (cos, sin)
  float* colsums = nullptr;        // LayerNorm column sums c = W g, e = W b (model create)
  std::vector<const float*> qkv_c, qkv_e, up_c, up_e;
  const float* head_c = nullptr;
  const float* head_e = nullptr;
  int32_t n_cus = 256;             // compute units of the model's device
  int32_t target_wgs = 0;          // > 0: split-K sized for about this many workgroups
  int32_t waves = 8;               // waves of a split-K workgroup for one row tile
  int32_t qkv_jt = 2;              // 16-column sub-tiles of the QKV projection's tiles at one row tile (2 or 4)
  int32_t rows_max_splits = 4;     // its splits of K at most
  int32_t rows_min_tiles = 256;    // 64-column tiles of a GEMM that takes the LDS-shared kernel
  int32_t rows_min_mt = 3;         // row tiles from which it does
  bool rows_forced = false;        // MSD_ROWS_MIN_TILES set: no balance check
  int32_t rows_narrow = 1;         // narrow GEMMs from 5 row tiles on: many splits, deferred epilogue
                                   // (0 off, 1 large matrices, 2 any)
  int32_t rows_narrow_mt = 3;      // row tiles from which it does
  int32_t attn_spans = 0;          // attention spans per chunk (0: chosen per call; 1: one-span kernel)
  int32_t attn_defer = -1;         // chunk merge in its own kernel: -1 by chunk count, 0 never, 1 always
  int32_t attn_ring = 1;           // chunks of several spans at head dim 128: the ring-fed kernel (0: streaming)
  int32_t prof_class = -1;         // instrumentation (msd_set_profile)
  std::vector<hipEvent_t> prof_begin, prof_end;
};

namespace {

thread_local std::string g_err;

msd_status fail(msd_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define MSD_HIP(call)                                                                    \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess) return fail(MSD_ERR_HIP, std::string(#call) + ": " + hipGetErrorString(e_)); \
  } while (0)

inline const uint16_t* T(const msd_model* m, int idx) { return m->t[idx]; }
inline const uint16_t* LT(const msd_model* m, int l, int slot) {
  return m->t[MSD_TENSOR_INDEX(l, slot)];
}
inline const uint16_t* head_w(const msd_model* m) {
  return m->cfg.tied_head ? T(m, MSD_T_EMBED) : T(m, MSD_T_LM_HEAD);
}

inline size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

// Row tiles of the kernels for M rows: 1, 2 or 3, else 5 (up to 80 rows),
// else the 9-tile variant.
inline int row_tiles(int M) {
  const int mt = (M + 15) / 16;
  return mt <= 3 ? mt : (mt <= 5 ? 5 : kMaxMT);
}

// Split-K factor. A workgroup streams its 1/s of a tile at about one
// compute unit's rate, so a GEMM lasts as long as its busiest unit: W =
// n_tiles * s workgroups over C units put ceil(W / C) of them on one unit.
// s maximises the balance W / (C ceil(W / C)) (the smallest s on a tie),
// with W <= per_cu * C (more would wait for a second dispatch round; per_cu
// is how many of these workgroups a unit holds) unless s = 1, and at least
// 2 k-steps per wave. Measured: 66B tree, O and down projections (144
// tiles, 4-wave workgroups, two a unit) 2 -> 3 splits: 59.4 -> 46.4 us and
// 207.6 -> 154.2 us. m->target_wgs > 0 instead asks for about that many
// workgroups (tuning).
int splits_for(const msd_model* m, int n_tiles, int K, int waves, int per_cu) {
  const int ks = K / 32;
  int max_s = ks / (2 * waves);
  if (max_s < 1) max_s = 1;
  if (m->target_wgs > 0) {
    const int want = std::max(1, (m->target_wgs + n_tiles / 2) / n_tiles);
    return want < max_s ? want : max_s;
  }
  const int64_t C = m->n_cus;
  int best = 1;
  double best_bal = 0.0;
  for (int s = 1; s <= max_s; ++s) {
    const int64_t W = (int64_t)n_tiles * s;
    if (s > 1 && W > (int64_t)per_cu * C) break;
    const double bal = (double)W / (double)(C * ((W + C - 1) / C));
    if (bal > best_bal + 1e-9) {
      best = s;
      best_bal = bal;
    }
  }
  return best;
}

// Several row tiles, wide GEMMs (256 or more 64-column tiles): 4 tiles a
// workgroup sharing the activation through LDS (one workgroup per compute
// unit from 5 row tiles on, by its LDS ring and registers; two up to 3).
// Splits of K as for split-K above, for the best balance of
// ceil(n_tiles / 4) * s workgroups over the units within one dispatch
// round, at most m->rows_max_splits (each split adds an fp32 partial of the
// whole [M][64] tile to write and read back) and at least 8 k-steps a
// split. Returns 0 where no split count balances at least 3/4 of the units
// (then the split-K kernel runs), unless the kernel is forced. Measured:
// 14B batch 16, FFN up (108 workgroup tiles, 2 splits) and LM head (594,
// whole K): 136.8 -> 97.0 us and 740 -> 522 us; 66B tree (3 row tiles, one
// workgroup a unit then): QKV (108, 2 splits) 118.3 -> 97.2 us, LM head
// (197) 224.8 -> 166.5 us, its FFN up (144 workgroup tiles: 0.56 at best)
// 168.8 -> 177.7 us.
int rows_splits(const msd_model* m, int n_tiles, int K, int per_cu) {
  const int64_t C = m->n_cus;
  const int64_t wg = (n_tiles + 3) / 4;
  const int max_s = std::max(1, std::min(m->rows_max_splits, (K / 32) / 8));
  int best = 1;
  double best_bal = 0.0;
  for (int s = 1; s <= max_s; ++s) {
    const int64_t W = wg * s;
    if (s > 1 && W > per_cu * C) break;
    const double bal = (double)W / (double)(C * ((W + C - 1) / C));
    if (bal > best_bal + 1e-9) {
      best = s;
      best_bal = bal;
    }
  }
  if (m->rows_forced) return best;
  return best_bal >= 0.75 ? best : 0;
}

// Narrow GEMMs (fewer tiles than m->rows_min_tiles) from 3 row tiles on:
// the same kernel with many splits of K, so that the 144-row MFMA work
// spreads over the chip, and the split sum plus epilogue in a kernel of its
// own (one wave per row tile) instead of in the last split to arrive; the
// split count as above, at most kRowsNarrowSplits, for matrices of at least
// kRowsNarrowMinWeights weights (each split writes and the epilogue kernel
// reads an fp32 partial of all M rows: 35 MB at 12 splits of a 5120-column
// output). m->rows_narrow: 0 off, 1 that rule, 2 any size (tests). Measured at 14B batch 16 (µs, GEMM +
// epilogue kernel against the split-K kernel): QKV 32.6 + 13.6 against
// 51.7, FFN down 43.8 + 10.2 against 66.4, but the O projection (26M
// weights, 13 k-steps a split) 34.0 + 10.5 against 36.3; 66B tree (3 row
// tiles, two workgroups a unit, 7 splits, 12 MB of partials): O 46.4 ->
// 31.5 + 7.3, down 154.2 -> 116.9 + 7.3, 30.0 -> 28.1 ms per step; at 2
// row tiles (14B tree) slower, 8.41 -> 8.78 ms.
constexpr int kRowsNarrowSplits = 16;
constexpr int64_t kRowsNarrowMinWeights = 32ll << 20;
int rows_narrow_splits(const msd_model* m, int n_tiles, int K, int per_cu) {
  const int64_t C = m->n_cus;
  const int64_t wg = (n_tiles + 3) / 4;
  const int max_s = std::max(1, std::min(kRowsNarrowSplits, (K / 32) / 8));
  int best = 1;
  double best_bal = 0.0;
  for (int s = 1; s <= max_s; ++s) {
    const int64_t W = wg * s;
    if (s > 1 && W > per_cu * C) break;
    const double bal = (double)W / (double)(C * ((W + C - 1) / C));
    if (bal > best_bal + 1e-9) {
      best = s;
      best_bal = bal;
    }
  }
  return best;
}

struct GemmShape {
  int n_tiles, K, splits, waves, jt;
  int wg_tiles = 1;
};

struct Shapes {
  GemmShape qkv, o, up, down, head;
};

// Tiles and waves per workgroup. With one row tile, a GEMM with fewer
// 64-column tiles than the workgroup target runs split-K workgroups of
// m->waves (8) waves, one with more (the LM head) whole-K workgroups of 4
// waves. Several row tiles: 64-column tiles, 4 waves. The SwiGLU FFN up
// projection with up to 3 row tiles: whole-K 128-column tiles of 2 waves
// (216 workgroups at the 14B shape, one dispatch round: at most one per CU).
Shapes shapes(const msd_model* m, int M) {
  const msd_model_config& c = m->cfg;
  const bool one = row_tiles(M) == 1;
  Shapes s;
  s.qkv.n_tiles = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim / kTileN;
  s.qkv.K = c.d_model;
  s.o.n_tiles = c.d_model / kTileN;
  s.o.K = c.n_heads * c.head_dim;
  s.up.n_tiles = c.act == MSD_ACT_SWIGLU ? c.d_ffn / 32 : c.d_ffn / kTileN;
  s.up.K = c.d_model;
  s.down.n_tiles = c.d_model / kTileN;
  s.down.K = c.d_ffn;
  s.head.n_tiles = (c.vocab + kTileN - 1) / kTileN;
  s.head.K = c.d_model;
  for (GemmShape* g : {&s.qkv, &s.o, &s.up, &s.down, &s.head}) {
    g->jt = 4;
    g->waves = one && g->n_tiles < m->n_cus ? m->waves : 4;
  }
  if (row_tiles(M) <= 3 && c.act == MSD_ACT_SWIGLU && c.d_ffn % 64 == 0) {
    s.up.jt = 8;
    s.up.n_tiles = c.d_ffn / 64;
    s.up.waves = 2;
  }
  // The QKV projection at one row tile, where twice its 64-column tile count
  // still fits the compute units: 32-column tiles (16 rotary pairs of a head)
  // of 8 waves, whole K (no split hand-off), 224 workgroups at the 14B
  // shape. Measured at the 14B chain: 18.82 -> 18.06 us per launch against
  // 64-column tiles with 2 splits of K.
  if (one && m->qkv_jt == 2 && 2 * s.qkv.n_tiles <= m->n_cus) {
    s.qkv.jt = 2;
    s.qkv.n_tiles = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim / 32;
    s.qkv.waves = 8;
  }
  if (one) {  // the LM head at one row tile: 128-column tiles of 4 waves
    s.head.jt = 8;
    s.head.n_tiles = (c.vocab + 2 * kTileN - 1) / (2 * kTileN);
    s.head.waves = 4;
  }
  for (GemmShape* g : {&s.qkv, &s.o, &s.up, &s.down, &s.head}) {
    const int rs = row_tiles(M) >= m->rows_min_mt && g->n_tiles >= m->rows_min_tiles && g->jt == 4
                       ? rows_splits(m, g->n_tiles, g->K, row_tiles(M) <= 3 ? 2 : 1)
                       : 0;
    if (rs > 0) {  // 4 tiles a workgroup, the activation shared in LDS
      g->wg_tiles = 4;
      g->waves = 4;
      g->splits = rs;
    } else if (m->rows_narrow && row_tiles(M) >= m->rows_narrow_mt && g->jt == 4 && g->n_tiles < m->rows_min_tiles &&
               (m->rows_narrow == 2 || (int64_t)g->n_tiles * kTileN * g->K >= kRowsNarrowMinWeights)) {
      g->wg_tiles = 4;
      g->waves = 4;
      g->splits = rows_narrow_splits(m, g->n_tiles, g->K, row_tiles(M) <= 3 ? 2 : 1);
    } else {
      g->splits = splits_for(m, g->n_tiles, g->K, g->waves, g->waves >= 8 ? 1 : 2);
    }
  }
  return s;
}

struct Layout {
  size_t x, stats, q, img_x, img_h, img_f, img_attn, img_act, partial, counters, part_o, part_ml,
      tile_ms, tile_top, head_ms, head_top, total;
  int64_t n_counters, n_gemm_counters;
  int32_t MT, max_chunks;
};

// image bytes of an [M][K] activation
inline size_t img_bytes(int K, int MT) { return (size_t)(K / 32) * MT * 1024 * sizeof(uint16_t); }

Layout layout(const msd_model* m, int batch, int n_slots, int kappa, int capacity) {
  const msd_model_config& c = m->cfg;
  const int M = batch * n_slots;
  const Shapes s = shapes(m, M);
  const int kmax = kappa > 1 ? kappa : 1;
  const int qd = c.n_heads * c.head_dim;
  Layout L{};
  L.MT = row_tiles(M);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  L.x = take((size_t)M * c.d_model * sizeof(float));
  L.stats = take((size_t)(c.d_model / kTileN) * M * sizeof(float2));
  // q as the attention's operand image: per sequence and kv head, the GQA
  // group's queries in 16-row tiles, hi + lo bf16 parts
  const int q_tiles = ((c.n_heads / c.n_kv_heads) * n_slots + 15) / 16;
  L.q = take((size_t)batch * c.n_kv_heads * q_tiles * (c.head_dim / 32) * 1024 * sizeof(uint16_t));
  L.img_x = take(img_bytes(c.d_model, L.MT));
  L.img_h = take(img_bytes(c.d_model, L.MT));
  L.img_f = take(img_bytes(c.d_model, L.MT));
  L.img_attn = take(img_bytes(qd, L.MT));
  L.img_act = take(img_bytes(c.d_ffn, L.MT));
  size_t part = 0;
  int max_tiles = 0;
  for (const GemmShape* g : {&s.qkv, &s.o, &s.up, &s.down, &s.head}) {
    if (g->splits > 1) {
      const size_t p = (size_t)g->n_tiles * g->splits * L.MT * g->jt * 256 * sizeof(float);
      part = p > part ? p : part;
      max_tiles = g->n_tiles > max_tiles ? g->n_tiles : max_tiles;
    }
  }
  L.partial = take(part);
  // the GEMMs' split-K counters, then the attention's chunk counters (one per
  // sequence, kv head and query tile); all cleared by the rows kernel
  const int attn_qt = ((c.n_heads / c.n_kv_heads) * n_slots + 15) / 16;
  L.n_gemm_counters = max_tiles;
  L.n_counters = max_tiles + (int64_t)batch * c.n_kv_heads * attn_qt;
  L.counters = take((size_t)L.n_counters * sizeof(int32_t));
  L.max_chunks = (capacity + kAttnChunk - 1) / kAttnChunk;
  const size_t qn = (size_t)(c.n_heads / c.n_kv_heads) * n_slots;
  const size_t nparts = (size_t)batch * c.n_kv_heads * L.max_chunks * qn;
  L.part_o = take(nparts * c.head_dim * sizeof(float));
  L.part_ml = take(nparts * sizeof(float2));
  L.tile_ms = take((size_t)s.head.n_tiles * M * sizeof(float2));
  L.tile_top = take((size_t)s.head.n_tiles * M * kmax * sizeof(uint64_t));
  const int parts = head_parts(s.head.n_tiles);
  L.head_ms = take((size_t)parts * M * sizeof(float2));
  L.head_top = take((size_t)parts * M * kmax * sizeof(uint64_t));
  L.total = off;
  return L;
}

msd_status make_topo(const msd_block* blk, Topo* topo) {
  const int n = blk->n_slots;
  topo->n_slots = n;
  topo->max_depth = 0;
  for (int i = 0; i < kMaxSlots; ++i) {
    topo->anc[i] = 0;
    topo->depth[i] = 0;
    topo->parent[i] = -1;
  }
  for (int i = 0; i < n; ++i) {
    const int p = blk->parent ? blk->parent[i] : i - 1;
    if (i == 0 && p != -1) return fail(MSD_ERR_SHAPE, "parent[0] must be -1");
    if (i > 0 && (p < 0 || p >= i)) return fail(MSD_ERR_SHAPE, "parent[i] must lie in [0, i)");
    topo->parent[i] = p;
    topo->depth[i] = i == 0 ? 0 : topo->depth[p] + 1;
    topo->anc[i] = (i == 0 ? 0ull : topo->anc[p]) | (1ull << i);
    if (topo->depth[i] > topo->max_depth) topo->max_depth = topo->depth[i];
  }
  return MSD_OK;
}

// row_limit: the block's rows go through the GEMMs (at most kMaxMT row
// tiles); acceptance and commit work per sequence and take any batch.
msd_status check_block(const msd_model* m, const msd_block* blk, bool row_limit = true) {
  if (!m || !blk) return fail(MSD_ERR_INVALID_ARG, "null model or block");
  if (blk->n_slots < 1 || blk->n_slots > kMaxSlots)
    return fail(MSD_ERR_SHAPE, "n_slots must lie in [1, 64]");
  if (blk->batch < 1) return fail(MSD_ERR_SHAPE, "batch must be >= 1");
  if (row_limit && (size_t)blk->batch * blk->n_slots > (size_t)kMaxMT * 16)
    return fail(MSD_ERR_SHAPE, "batch * n_slots must be <= 144");
  if (!blk->tokens) return fail(MSD_ERR_INVALID_ARG, "null tokens");
  return MSD_OK;
}

// Query tiles per attention workgroup: one each while (chunks x kv heads x
// sequences x query tiles) stays within kAttnTargetWgs workgroups (8 per CU:
// the chain and the trees, where the most parallelism wins for a
// latency-bound step; measured: grouping the 14B tree's 8 tiles by 3 took
// 57 us against 51 us); beyond that (batches of long contexts), groups of
// tiles share one load of their chunk's K and V instead of each re-reading it
// (14B batch 16: 414 us against 508 us).
constexpr int64_t kAttnTargetWgs = 2048;
int attn_q_per_wg(int max_chunks, int n_kv_heads, int batch, int q_tiles) {
  const int64_t base = (int64_t)max_chunks * n_kv_heads * batch;
  int64_t groups = kAttnTargetWgs / (base > 0 ? base : 1);
  if (groups < 1) groups = 1;
  if (groups > q_tiles) groups = q_tiles;
  return (int)((q_tiles + groups - 1) / groups);
}

// Attention launch shape: query tiles per workgroup and 256-key spans per
// chunk. Where the grid of one-span chunks (the group's query tiles 3 at a
// time, fewest re-reads of K and V) exceeds what the chip holds at once, a
// workgroup takes nb spans in turn (the streaming kernel) with nb chosen for
// about one workgroup per compute unit: its loads stream while it computes
// and the chunk hand-off and final merge shrink nb-fold (14B batch 16:
// 207 us against 105 us; 14B tree 43 against 34; 66B tree 59 against 35).
// Short contexts keep one-span chunks, their tiles grouped as above.
constexpr int64_t kAttnStreamWgs = 256;
struct AttnShape {
  int q_per_wg, nb;
  bool ring;
};
// Chunks of several spans take attn_ring_kernel at head dim 128 (up to 4
// query tiles a workgroup, K and V fed through an LDS ring; m->attn_ring 0
// keeps attn_stream_kernel, up to 3 tiles).
AttnShape attn_shape(const msd_model* m, int max_chunks, int n_kv_heads, int batch, int q_tiles,
                     int head_dim) {
  const bool ring = m->attn_ring != 0 && head_dim == 128;
  const int qs = std::min(ring ? 4 : 3, q_tiles);
  const int64_t grid1 = (int64_t)max_chunks * n_kv_heads * batch * ((q_tiles + qs - 1) / qs);
  int64_t nb = m->attn_spans > 0 ? m->attn_spans : (grid1 + kAttnStreamWgs - 1) / kAttnStreamWgs;
  nb = std::min<int64_t>(nb, max_chunks);
  if (nb >= 2) return {qs, (int)nb, ring};
  return {attn_q_per_wg(max_chunks, n_kv_heads, batch, q_tiles), 1, false};
}

// Chunk merge in a kernel of its own (instead of the last chunk to arrive)
// from kAttnDeferChunks chunks of the cache's capacity on (m->attn_defer: -1
// that rule, 0 never, 1 always). Measured: the 14B tree (9 chunks of 2
// spans) 8.62 -> 8.30 ms per step; where the last-arrival merge is short
// (the chain's 5 one-span chunks, 2 or 3 chunks at batch 16 and the 66B
// tree) the extra launch does not pay.
constexpr int kAttnDeferChunks = 6;
bool attn_defer(const msd_model* m, int max_chunks, int nb) {
  const int chunks = (max_chunks + nb - 1) / nb;
  if (chunks <= 1 || m->attn_defer == 0) return false;
  return m->attn_defer == 1 || chunks >= kAttnDeferChunks;
}

GemmArgs gemm_base(const msd_model* m, const Layout& L, char* ws, int M, const GemmShape& sh, int N) {
  GemmArgs g{};
  g.M = M;
  g.MT = L.MT;
  g.K = sh.K;
  g.N = N;
  g.n_tiles = sh.n_tiles;
  g.splits = sh.splits;
  g.waves = sh.waves;
  g.jt = sh.jt;
  g.wg_tiles = sh.wg_tiles;
  g.partial = reinterpret_cast<float*>(ws + L.partial);
  g.counters = reinterpret_cast<int32_t*>(ws + L.counters);
  g.n_heads = m->cfg.n_heads;
  g.n_kv_heads = m->cfg.n_kv_heads;
  g.head_dim = m->cfg.head_dim;
  return g;
}

// the pre-norm of a GEMM's input, applied in its epilogue
RowNorm prenorm(const msd_model* m, const float2* stats, const float* col_g, const float* col_b) {
  RowNorm n{};
  n.kind = m->cfg.norm == MSD_NORM_LAYER ? 2 : 1;
  n.stats = stats;
  n.tiles = m->cfg.d_model / kTileN;
  n.eps = m->cfg.norm_eps;
  n.col_g = col_g;
  n.col_b = col_b;
  return n;
}

// final norm + LM head + per-row merge (used at the early exit and at the end)
msd_status run_head(const msd_model* m, const Shapes& s, const Layout& L, char* ws, int M,
                    const float2* stats, int kappa, float* logits, int32_t* ids, float* logp,
                    int32_t* argmax, float* lse, hipStream_t stream) {
  const msd_model_config& c = m->cfg;
  GemmArgs g = gemm_base(m, L, ws, M, s.head, c.vocab);
  g.a_img = reinterpret_cast<const uint16_t*>(ws + L.img_f);
  g.norm = prenorm(m, stats, m->head_c, m->head_e);
  g.map = MAP_PLAIN;
  g.w0 = head_w(m);
  g.logits = logits;
  g.tile_ms = reinterpret_cast<float2*>(ws + L.tile_ms);
  g.tile_top = reinterpret_cast<uint64_t*>(ws + L.tile_top);
  g.kappa = kappa;
  MSD_HIP(launch_gemm(EPI_HEAD, g, stream));
  HeadMergeArgs hm{g.tile_ms,
                   g.tile_top,
                   s.head.n_tiles,
                   M,
                   kappa,
                   reinterpret_cast<float2*>(ws + L.head_ms),
                   reinterpret_cast<uint64_t*>(ws + L.head_top),
                   ids,
                   logp,
                   argmax,
                   lse};
  MSD_HIP(launch_head_merge(hm, stream));
  return MSD_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// The profiled class's events of a layer, to attach to a GEMM launch.
LaunchEvents prof_events(const msd_model* m, int kclass, int layer) {
  LaunchEvents ev;
  if (m->prof_class == kclass && layer < (int)m->prof_begin.size()) {
    ev.start = m->prof_begin[layer];
    ev.stop = m->prof_end[layer];
  }
  return ev;
}

hipError_t prof_mark(const msd_model* m, int kclass, int layer, bool begin, hipStream_t s) {
  if (m->prof_class != kclass || layer >= (int)m->prof_begin.size()) return hipSuccess;
  hipEvent_t ev = begin ? m->prof_begin[layer] : m->prof_end[layer];
  return ev ? hipEventRecord(ev, s) : hipSuccess;
}

// Device address of the current device's `scratch`, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

msd_status static_scratch_address(void** out) {
  int dev = -1;
  MSD_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(MSD_ERR_UNSUPPORTED, "device index above 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    MSD_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(MSD_ERR_HIP, "hipGetSymbolAddress returned a null scratch address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MSD_OK;
}

msd_status verify_prepare(const msd_model* m, msd_kv_cache* kv, const msd_block* blk,
                          const msd_ee_request* ee, const int32_t* argmax, Topo* topo, Layout* Lout);
msd_status verify_launch(const msd_model* m, msd_kv_cache* kv, const msd_block* blk,
                         const msd_ee_request* ee, float* logits, int32_t* argmax, float* lse,
                         char* w, const Topo& topo, const Layout& L, hipStream_t stream);

}  // namespace

extern "C" {

const char* msd_last_error(void) { return g_err.c_str(); }

msd_status msd_model_create(const msd_model_config* cfg, const void* const* tensors,
                            int32_t n_tensors, msd_model** out) {
  if (!cfg || !tensors || !out) return fail(MSD_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  const msd_model_config& c = *cfg;
  if (c.n_layers < 1 || c.d_model < 64 || c.n_heads < 1 || c.n_kv_heads < 1 || c.vocab < 64 ||
      c.d_ffn < 64)
    return fail(MSD_ERR_SHAPE, "model sizes out of range");
  if (c.head_dim != 64 && c.head_dim != 128) return fail(MSD_ERR_SHAPE, "head_dim must be 64 or 128");
  if (c.n_heads % c.n_kv_heads) return fail(MSD_ERR_SHAPE, "n_heads must be a multiple of n_kv_heads");
  if (c.d_model % 64 || c.d_ffn % 64) return fail(MSD_ERR_SHAPE, "d_model and d_ffn must be multiples of 64");
  if (c.vocab % 16) return fail(MSD_ERR_SHAPE, "vocab must be a multiple of 16");
  if (head_parts((c.vocab + kTileN - 1) / kTileN) > 64) return fail(MSD_ERR_SHAPE, "vocab must be <= 1048576");
  if (c.norm != MSD_NORM_RMS && c.norm != MSD_NORM_LAYER) return fail(MSD_ERR_INVALID_ARG, "norm kind");
  if (c.act != MSD_ACT_SWIGLU && c.act != MSD_ACT_RELU) return fail(MSD_ERR_INVALID_ARG, "act kind");
  if (c.pos != MSD_POS_ROPE && c.pos != MSD_POS_LEARNED) return fail(MSD_ERR_INVALID_ARG, "pos kind");
  if (c.max_positions < 1) return fail(MSD_ERR_SHAPE, "max_positions must be >= 1");
  if (!(c.norm_eps > 0.0f)) return fail(MSD_ERR_INVALID_ARG, "norm_eps must be > 0");
  if (c.pos == MSD_POS_ROPE && !(c.rope_theta > 0.0f)) return fail(MSD_ERR_INVALID_ARG, "rope_theta must be > 0");
  if (n_tensors != MSD_N_TENSORS(c.n_layers)) return fail(MSD_ERR_SHAPE, "n_tensors != MSD_N_TENSORS(n_layers)");

  auto need = [&](int idx, const char* what) -> bool {
    if (!tensors[idx]) {
      g_err = std::string("missing tensor: ") + what;
      return false;
    }
    if (!aligned16(tensors[idx])) {
      g_err = std::string("tensor not 16-byte aligned: ") + what;
      return false;
    }
    return true;
  };
  const bool ln = c.norm == MSD_NORM_LAYER, bias = c.has_bias != 0;
  if (!need(MSD_T_EMBED, "embed") || !need(MSD_T_FINAL_G, "final_g")) return MSD_ERR_INVALID_ARG;
  if (!c.tied_head && !need(MSD_T_LM_HEAD, "lm_head")) return MSD_ERR_INVALID_ARG;
  if (ln && !need(MSD_T_FINAL_B, "final_b")) return MSD_ERR_INVALID_ARG;
  if (c.pos == MSD_POS_LEARNED && !need(MSD_T_POS_EMBED, "pos_embed")) return MSD_ERR_INVALID_ARG;
  for (int l = 0; l < c.n_layers; ++l) {
    const int b = MSD_TENSOR_INDEX(l, 0);
    for (int s : {MSD_L_ATTN_G, MSD_L_WQ, MSD_L_WK, MSD_L_WV, MSD_L_WO, MSD_L_MLP_G, MSD_L_W_UP,
                  MSD_L_W_DOWN})
      if (!need(b + s, "layer weight")) return MSD_ERR_INVALID_ARG;
    if (c.act == MSD_ACT_SWIGLU && !need(b + MSD_L_W_GATE, "w_gate")) return MSD_ERR_INVALID_ARG;
    if (ln && (!need(b + MSD_L_ATTN_B, "attn_b") || !need(b + MSD_L_MLP_B, "mlp_b")))
      return MSD_ERR_INVALID_ARG;
    if (bias) {
      for (int s : {MSD_L_BQ, MSD_L_BK, MSD_L_BV, MSD_L_BO})
        if (!need(b + s, "attention bias")) return MSD_ERR_INVALID_ARG;
      if (c.act == MSD_ACT_RELU && (!need(b + MSD_L_B_UP, "b_up") || !need(b + MSD_L_B_DOWN, "b_down")))
        return MSD_ERR_INVALID_ARG;
    }
  }

  msd_model* m = new msd_model();
  m->cfg = c;
  m->t.resize(n_tensors);
  for (int i = 0; i < n_tensors; ++i) m->t[i] = static_cast<const uint16_t*>(tensors[i]);
  // tensors the model does not use are ignored
  if (!ln) {
    m->t[MSD_T_FINAL_B] = nullptr;
    for (int l = 0; l < c.n_layers; ++l) {
      m->t[MSD_TENSOR_INDEX(l, MSD_L_ATTN_B)] = nullptr;
      m->t[MSD_TENSOR_INDEX(l, MSD_L_MLP_B)] = nullptr;
    }
  }
  if (!bias)
    for (int l = 0; l < c.n_layers; ++l)
      for (int s : {MSD_L_BQ, MSD_L_BK, MSD_L_BV, MSD_L_BO, MSD_L_B_UP, MSD_L_B_DOWN})
        m->t[MSD_TENSOR_INDEX(l, s)] = nullptr;
  if (c.pos != MSD_POS_LEARNED) m->t[MSD_T_POS_EMBED] = nullptr;
  {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
      m->n_cus = cus;
  }
  if (const char* e = getenv("MSD_GEMM_TARGET_WGS")) {
    const int v = atoi(e);
    if (v > 0) m->target_wgs = v;
  }
  if (const char* e = getenv("MSD_GEMM_WAVES")) {
    const int v = atoi(e);
    if (v == 4 || v == 8) m->waves = v;
  }
  if (const char* e = getenv("MSD_QKV_JT")) {
    const int v = atoi(e);
    if (v == 2 || v == 4) m->qkv_jt = v;
  }
  if (const char* e = getenv("MSD_ROWS_NARROW")) {
    const int v = atoi(e);
    if (v >= 0 && v <= 2) m->rows_narrow = v;
  }
  if (const char* e = getenv("MSD_ROWS_NARROW_MT")) {
    const int v = atoi(e);
    if (v >= 2 && v <= kMaxMT) m->rows_narrow_mt = v;
  }
  if (const char* e = getenv("MSD_ROWS_MIN_MT")) {
    const int v = atoi(e);
    if (v >= 2 && v <= kMaxMT) m->rows_min_mt = v;
  }
  if (const char* e = getenv("MSD_ROWS_MIN_TILES")) {
    const int v = atoi(e);
    if (v >= 1) {
      m->rows_min_tiles = v;
      m->rows_forced = true;
    }
  }
  if (const char* e = getenv("MSD_ROWS_MAX_SPLITS")) {
    const int v = atoi(e);
    if (v >= 1 && v <= 64) m->rows_max_splits = v;
  }
  if (const char* e = getenv("MSD_ATTN_DEFER")) {
    const int v = atoi(e);
    if (v >= -1 && v <= 1) m->attn_defer = v;
  }
  if (const char* e = getenv("MSD_ATTN_RING")) {
    const int v = atoi(e);
    if (v == 0 || v == 1) m->attn_ring = v;
  }
  if (const char* e = getenv("MSD_ATTN_SPANS")) {
    const int v = atoi(e);
    if (v >= 1 && v <= kMaxAttnChunks) m->attn_spans = v;
  }

  // LayerNorm models: column sums c = W g and e = W b of every matrix that
  // consumes a LayerNorm output (q/k/v, the FFN up projections, the LM head),
  // from the row-major weights before they are rearranged
  if (ln) {
    const int qd = c.n_heads * c.head_dim, kd = c.n_kv_heads * c.head_dim;
    const size_t n_qkv = (size_t)qd + 2 * kd;
    const size_t n_up = (size_t)(c.act == MSD_ACT_SWIGLU ? 2 : 1) * c.d_ffn;
    const size_t per_layer = 2 * (n_qkv + n_up);
    const size_t total = per_layer * c.n_layers + 2 * (size_t)c.vocab;
    hipError_t e = hipMalloc(&m->colsums, total * sizeof(float));
    float* p = m->colsums;
    for (int l = 0; e == hipSuccess && l < c.n_layers; ++l) {
      float* qc = p;
      float* qe = p + n_qkv;
      float* uc = p + 2 * n_qkv;
      float* ue = uc + n_up;
      p += per_layer;
      m->qkv_c.push_back(qc);
      m->qkv_e.push_back(qe);
      m->up_c.push_back(uc);
      m->up_e.push_back(ue);
      const uint16_t* ag = LT(m, l, MSD_L_ATTN_G);
      const uint16_t* ab = LT(m, l, MSD_L_ATTN_B);
      const uint16_t* mg = LT(m, l, MSD_L_MLP_G);
      const uint16_t* mb = LT(m, l, MSD_L_MLP_B);
      e = launch_colsum(LT(m, l, MSD_L_WQ), qd, c.d_model, ag, ab, qc, qe, 0);
      if (e == hipSuccess) e = launch_colsum(LT(m, l, MSD_L_WK), kd, c.d_model, ag, ab, qc + qd, qe + qd, 0);
      if (e == hipSuccess)
        e = launch_colsum(LT(m, l, MSD_L_WV), kd, c.d_model, ag, ab, qc + qd + kd, qe + qd + kd, 0);
      if (c.act == MSD_ACT_SWIGLU) {
        if (e == hipSuccess) e = launch_colsum(LT(m, l, MSD_L_W_GATE), c.d_ffn, c.d_model, mg, mb, uc, ue, 0);
        if (e == hipSuccess)
          e = launch_colsum(LT(m, l, MSD_L_W_UP), c.d_ffn, c.d_model, mg, mb, uc + c.d_ffn, ue + c.d_ffn, 0);
      } else if (e == hipSuccess) {
        e = launch_colsum(LT(m, l, MSD_L_W_UP), c.d_ffn, c.d_model, mg, mb, uc, ue, 0);
      }
    }
    if (e == hipSuccess) {
      m->head_c = p;
      m->head_e = p + c.vocab;
      e = launch_colsum(head_w(m), c.vocab, c.d_model, T(m, MSD_T_FINAL_G), T(m, MSD_T_FINAL_B), p,
                        p + c.vocab, 0);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(0);
    if (e != hipSuccess) {
      if (m->colsums) (void)hipFree(m->colsums);
      delete m;
      return fail(MSD_ERR_HIP, std::string("layer-norm column sums: ") + hipGetErrorString(e));
    }
  } else {
    m->qkv_c.assign(c.n_layers, nullptr);
    m->qkv_e.assign(c.n_layers, nullptr);
    m->up_c.assign(c.n_layers, nullptr);
    m->up_e.assign(c.n_layers, nullptr);
  }

  // every projection matrix goes k-step-major, in place, through one
  // temporary buffer as large as the largest matrix
  {
    struct Mat {
      uint16_t* p;
      int64_t rows;
      int32_t K;
    };
    std::vector<Mat> mats;
    auto add = [&](const uint16_t* p, int64_t rows, int32_t K) {
      mats.push_back(Mat{const_cast<uint16_t*>(p), rows, K});
    };
    const int qd = c.n_heads * c.head_dim, kd = c.n_kv_heads * c.head_dim;
    for (int l = 0; l < c.n_layers; ++l) {
      add(m->t[MSD_TENSOR_INDEX(l, MSD_L_WQ)], qd, c.d_model);
      add(m->t[MSD_TENSOR_INDEX(l, MSD_L_WK)], kd, c.d_model);
      add(m->t[MSD_TENSOR_INDEX(l, MSD_L_WV)], kd, c.d_model);
      add(m->t[MSD_TENSOR_INDEX(l, MSD_L_WO)], c.d_model, qd);
      if (c.act == MSD_ACT_SWIGLU) add(m->t[MSD_TENSOR_INDEX(l, MSD_L_W_GATE)], c.d_ffn, c.d_model);
      add(m->t[MSD_TENSOR_INDEX(l, MSD_L_W_UP)], c.d_ffn, c.d_model);
      add(m->t[MSD_TENSOR_INDEX(l, MSD_L_W_DOWN)], c.d_model, c.d_ffn);
    }
    add(c.tied_head ? m->t[MSD_T_EMBED] : m->t[MSD_T_LM_HEAD], c.vocab, c.d_model);
    size_t biggest = 0;
    for (const Mat& x : mats) biggest = std::max(biggest, (size_t)x.rows * x.K * 2);
    void* tmp = nullptr;
    hipError_t e = hipMalloc(&tmp, biggest);
    for (size_t i = 0; e == hipSuccess && i < mats.size(); ++i) {
      const size_t bytes = (size_t)mats[i].rows * mats[i].K * 2;
      e = hipMemcpyAsync(tmp, mats[i].p, bytes, hipMemcpyDeviceToDevice, 0);
      if (e == hipSuccess) e = launch_repack(static_cast<uint16_t*>(tmp), mats[i].p, mats[i].rows, mats[i].K, 0);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(0);
    if (tmp) (void)hipFree(tmp);
    if (e != hipSuccess) {
      if (m->colsums) (void)hipFree(m->colsums);
      delete m;
      return fail(MSD_ERR_HIP, std::string("weight repack: ") + hipGetErrorString(e));
    }
  }

  if (c.pos == MSD_POS_ROPE) {
    const int half = c.head_dim / 2;
    std::vector<float2> tab((size_t)c.max_positions * half);
    for (int p = 0; p < c.max_positions; ++p)
      for (int j = 0; j < half; ++j) {
        const double a = (double)p * std::pow((double)c.rope_theta, -2.0 * j / c.head_dim);
        tab[(size_t)p * half + j] = make_float2((float)std::cos(a), (float)std::sin(a));
      }
    hipError_t e = hipMalloc(&m->rope, tab.size() * sizeof(float2));
    if (e == hipSuccess) e = hipMemcpy(m->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      if (m->rope) (void)hipFree(m->rope);
      if (m->colsums) (void)hipFree(m->colsums);
      delete m;
      return fail(MSD_ERR_HIP, std::string("rotary table: ") + hipGetErrorString(e));
    }
  }
  // the static scratch of this device (msd_verify_block_static)
  const msd_status sst = static_scratch_address(&m->scratch);
  if (sst != MSD_OK) {
    const std::string msg = g_err;
    if (m->rope) (void)hipFree(m->rope);
    if (m->colsums) (void)hipFree(m->colsums);
    delete m;
    return fail(sst, "static scratch: " + msg);
  }
  *out = m;
  return MSD_OK;
}

void msd_model_destroy(msd_model* m) {
  if (!m) return;
  if (m->rope) (void)hipFree(m->rope);
  if (m->colsums) (void)hipFree(m->colsums);
  delete m;
}

size_t msd_workspace_bytes(const msd_model* m, int32_t batch, int32_t n_slots, int32_t kappa,
                           int32_t capacity) {
  if (!m || batch < 1 || n_slots < 1 || capacity < 1) return 0;
  return layout(m, batch, n_slots, kappa, capacity).total;
}

msd_status msd_verify_block(const msd_model* m, msd_kv_cache* kv, const msd_block* blk,
                            const msd_ee_request* ee, float* logits, int32_t* argmax, float* lse,
                            void* ws, size_t ws_bytes, hipStream_t stream) {
  Topo topo;
  Layout L;
  msd_status st = verify_prepare(m, kv, blk, ee, argmax, &topo, &L);
  if (st != MSD_OK) return st;
  if (!ws || ws_bytes < L.total) return fail(MSD_ERR_WORKSPACE, "workspace too small");
  return verify_launch(m, kv, blk, ee, logits, argmax, lse, static_cast<char*>(ws), topo, L, stream);
}

msd_status msd_verify_block_static(const msd_model* m, msd_kv_cache* kv, const msd_block* blk,
                                   const msd_ee_request* ee, float* logits, int32_t* argmax,
                                   float* lse, hipStream_t stream) {
  Topo topo;
  Layout L;
  msd_status st = verify_prepare(m, kv, blk, ee, argmax, &topo, &L);
  if (st != MSD_OK) return st;
  if (L.total > kStaticScratchBytes)
    return fail(MSD_ERR_WORKSPACE, "this block needs " + std::to_string(L.total) +
                                       " bytes of scratch; the static scratch holds " +
                                       std::to_string(kStaticScratchBytes) +
                                       " (use msd_verify_block with a workspace)");
  if (!m->scratch) return fail(MSD_ERR_HIP, "static scratch address unavailable");
  return verify_launch(m, kv, blk, ee, logits, argmax, lse, static_cast<char*>(m->scratch), topo, L,
                       stream);
}

}  // extern "C"

namespace {

// Host checks of a verify call; fills the block topology and the workspace
// layout. Enqueues nothing.
msd_status verify_prepare(const msd_model* m, msd_kv_cache* kv, const msd_block* blk,
                          const msd_ee_request* ee, const int32_t* argmax, Topo* topo, Layout* Lout) {
  msd_status st = check_block(m, blk);
  if (st != MSD_OK) return st;
  if (!kv || !kv->k || !kv->v || !kv->len || !kv->status) return fail(MSD_ERR_INVALID_ARG, "null kv cache field");
  if (!argmax) return fail(MSD_ERR_INVALID_ARG, "null argmax");
  if (blk->batch > kv->batch_cap) return fail(MSD_ERR_SHAPE, "batch exceeds the cache's batch_cap");
  if (kv->capacity < blk->n_slots) return fail(MSD_ERR_CAPACITY, "cache capacity below n_slots");
  const msd_model_config& c = m->cfg;
  if (kv->capacity > c.max_positions) return fail(MSD_ERR_CAPACITY, "cache capacity exceeds max_positions");
  if (kv->capacity > kMaxCapacity) return fail(MSD_ERR_CAPACITY, "cache capacity above 32768");
  int kappa = 1;
  if (ee) {
    if (ee->layer < 1 || ee->layer > c.n_layers - 1) return fail(MSD_ERR_INVALID_ARG, "early-exit layer out of [1, n_layers-1]");
    if (ee->kappa < 1 || ee->kappa > kMaxKappa) return fail(MSD_ERR_INVALID_ARG, "kappa out of [1, 32]");
    if (!ee->ids || !ee->logp) return fail(MSD_ERR_INVALID_ARG, "null early-exit outputs");
    kappa = ee->kappa;
  }
  st = make_topo(blk, topo);
  if (st != MSD_OK) return st;
  *Lout = layout(m, blk->batch, blk->n_slots, kappa, kv->capacity);
  return MSD_OK;
}

// The verify pass proper: rows, N layers (early exit after layer l_e), final
// head, all on `stream`, using the workspace at w laid out as L.
msd_status verify_launch(const msd_model* m, msd_kv_cache* kv, const msd_block* blk,
                         const msd_ee_request* ee, float* logits, int32_t* argmax, float* lse,
                         char* w, const Topo& topo, const Layout& L, hipStream_t stream) {
  msd_status st = MSD_OK;
  const msd_model_config& c = m->cfg;
  const int M = blk->batch * blk->n_slots;
  const Shapes s = shapes(m, M);
  const int d = c.d_model, qd = c.n_heads * c.head_dim;
  float* x = reinterpret_cast<float*>(w + L.x);
  float2* stats = reinterpret_cast<float2*>(w + L.stats);
  uint16_t* q_img = reinterpret_cast<uint16_t*>(w + L.q);
  const int q_tiles = ((c.n_heads / c.n_kv_heads) * blk->n_slots + 15) / 16;
  uint16_t* img_x = reinterpret_cast<uint16_t*>(w + L.img_x);
  uint16_t* img_h = reinterpret_cast<uint16_t*>(w + L.img_h);
  uint16_t* img_f = reinterpret_cast<uint16_t*>(w + L.img_f);
  uint16_t* img_attn = reinterpret_cast<uint16_t*>(w + L.img_attn);
  uint16_t* img_act = reinterpret_cast<uint16_t*>(w + L.img_act);
  int32_t* counters = reinterpret_cast<int32_t*>(w + L.counters);
  const size_t layer_elems = (size_t)kv->batch_cap * c.n_kv_heads * kv->capacity * c.head_dim;

  // block rows: residual, statistics and the first attention input image;
  // also clears the counters and the padding rows of the attention image
  RowsArgs ra{};
  ra.tokens = blk->tokens;
  ra.embed = T(m, MSD_T_EMBED);
  ra.pos_embed = T(m, MSD_T_POS_EMBED);
  ra.embed_frag = c.tied_head;
  ra.len = kv->len;
  ra.M = M;
  ra.MT = L.MT;
  ra.d = d;
  ra.n_slots = blk->n_slots;
  ra.max_positions = c.max_positions;
  ra.vocab = c.vocab;
  ra.status = kv->status;
  ra.x = x;
  ra.stats = stats;
  ra.img = ImageOut{img_x, LT(m, 0, MSD_L_ATTN_G)};
  ra.zero_img = img_attn;
  ra.zero_img_k = qd;
  ra.zero_i32 = counters;
  ra.n_zero = L.n_counters;
  for (int i = 0; i < kMaxSlots; ++i) ra.depth[i] = topo.depth[i];
  MSD_HIP(launch_rows(ra, stream));

  for (int l = 0; l < c.n_layers; ++l) {
    uint16_t* kc = static_cast<uint16_t*>(kv->k) + (size_t)l * layer_elems;
    uint16_t* vc = static_cast<uint16_t*>(kv->v) + (size_t)l * layer_elems;

    GemmArgs g = gemm_base(m, L, w, M, s.qkv, qd + 2 * c.n_kv_heads * c.head_dim);
    g.a_img = img_x;
    g.norm = prenorm(m, stats, m->qkv_c[l], m->qkv_e[l]);
    g.map = MAP_QKV;
    g.w0 = LT(m, l, MSD_L_WQ);
    g.w1 = LT(m, l, MSD_L_WK);
    g.w2 = LT(m, l, MSD_L_WV);
    g.b0 = LT(m, l, MSD_L_BQ);
    g.b1 = LT(m, l, MSD_L_BK);
    g.b2 = LT(m, l, MSD_L_BV);
    g.q_img = q_img;
    g.q_tiles = q_tiles;
    g.k_cache = kc;
    g.v_cache = vc;
    g.len = kv->len;
    g.status = kv->status;
    g.capacity = kv->capacity;
    g.n_slots = blk->n_slots;
    g.rope = m->rope;
    g.rope_rows = c.max_positions;
    for (int i = 0; i < kMaxSlots; ++i) g.depth[i] = topo.depth[i];
    MSD_HIP(launch_gemm(EPI_QKV, g, stream, prof_events(m, MSD_K_QKV, l)));

    AttnArgs aa{};
    aa.q_img = q_img;
    aa.k_cache = kc;
    aa.v_cache = vc;
    aa.len = kv->len;
    aa.status = kv->status;
    aa.out_img = img_attn;
    aa.MT = L.MT;
    aa.counters = counters + L.n_gemm_counters;
    aa.part_o = reinterpret_cast<float*>(w + L.part_o);
    aa.part_ml = reinterpret_cast<float*>(w + L.part_ml);
    aa.batch = blk->batch;
    aa.n_heads = c.n_heads;
    aa.n_kv_heads = c.n_kv_heads;
    aa.capacity = kv->capacity;
    aa.n_slots = blk->n_slots;
    aa.max_chunks = L.max_chunks;
    const AttnShape ash = attn_shape(m, L.max_chunks, c.n_kv_heads, blk->batch, q_tiles, c.head_dim);
    aa.q_per_wg = ash.q_per_wg;
    aa.nb = ash.nb;
    aa.ring = ash.ring ? 1 : 0;
    aa.scale = 1.0f / std::sqrt((float)c.head_dim);
    aa.topo = topo;
    aa.defer = attn_defer(m, L.max_chunks, ash.nb) ? 1 : 0;
    MSD_HIP(prof_mark(m, MSD_K_ATTN, l, true, stream));
    MSD_HIP(launch_attention(c.head_dim, aa, stream));
    if (aa.defer) MSD_HIP(launch_attention_merge(c.head_dim, aa, stream));
    MSD_HIP(prof_mark(m, MSD_K_ATTN, l, false, stream));

    g = gemm_base(m, L, w, M, s.o, d);
    g.a_img = img_attn;
    g.map = MAP_PLAIN;
    g.w0 = LT(m, l, MSD_L_WO);
    g.b0 = LT(m, l, MSD_L_BO);
    g.x = x;
    g.stats_out = stats;
    g.img_out[0] = ImageOut{img_h, LT(m, l, MSD_L_MLP_G)};
    MSD_HIP(launch_gemm(EPI_RESID, g, stream, prof_events(m, MSD_K_OPROJ, l)));

    g = gemm_base(m, L, w, M, s.up, c.act == MSD_ACT_SWIGLU ? 2 * c.d_ffn : c.d_ffn);
    g.a_img = img_h;
    g.norm = prenorm(m, stats, m->up_c[l], m->up_e[l]);
    g.act_img = img_act;
    if (c.act == MSD_ACT_SWIGLU) {
      g.map = MAP_GATEUP;
      g.w0 = LT(m, l, MSD_L_W_GATE);
      g.w1 = LT(m, l, MSD_L_W_UP);
      MSD_HIP(launch_gemm(EPI_SWIGLU, g, stream, prof_events(m, MSD_K_FFN_UP, l)));
    } else {
      g.map = MAP_PLAIN;
      g.w0 = LT(m, l, MSD_L_W_UP);
      g.b0 = LT(m, l, MSD_L_B_UP);
      MSD_HIP(launch_gemm(EPI_RELU, g, stream, prof_events(m, MSD_K_FFN_UP, l)));
    }

    const bool ee_here = ee && l + 1 == ee->layer;
    g = gemm_base(m, L, w, M, s.down, d);
    g.a_img = img_act;
    g.map = MAP_PLAIN;
    g.w0 = LT(m, l, MSD_L_W_DOWN);
    g.b0 = LT(m, l, MSD_L_B_DOWN);
    g.x = x;
    g.stats_out = stats;
    if (l + 1 < c.n_layers) g.img_out[0] = ImageOut{img_x, LT(m, l + 1, MSD_L_ATTN_G)};
    if (ee_here || l + 1 == c.n_layers) g.img_out[1] = ImageOut{img_f, T(m, MSD_T_FINAL_G)};
    MSD_HIP(launch_gemm(EPI_RESID, g, stream, prof_events(m, MSD_K_FFN_DOWN, l)));

    if (ee_here) {
      st = run_head(m, s, L, w, M, stats, ee->kappa, nullptr, ee->ids, ee->logp, nullptr, nullptr,
                    stream);
      if (st != MSD_OK) return st;
      if (ee->ready) MSD_HIP(hipEventRecord(ee->ready, stream));
    }
  }
  return run_head(m, s, L, w, M, stats, 1, logits, nullptr, nullptr, argmax, lse, stream);
}

}  // namespace

extern "C" {

msd_status msd_early_exit_topk(const msd_model* m, const float* hidden, int32_t M, int32_t kappa,
                               int32_t* ids, float* logp, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  if (!m || !hidden || !ids || !logp) return fail(MSD_ERR_INVALID_ARG, "null argument");
  if (M < 1 || M > kMaxMT * 16) return fail(MSD_ERR_SHAPE, "M must lie in [1, 144]");
  if (kappa < 1 || kappa > kMaxKappa) return fail(MSD_ERR_INVALID_ARG, "kappa out of [1, 32]");
  if (!aligned16(hidden)) return fail(MSD_ERR_INVALID_ARG, "hidden must be 16-byte aligned");
  const Layout L = layout(m, 1, M, kappa, 1);
  if (!ws || ws_bytes < L.total) return fail(MSD_ERR_WORKSPACE, "workspace too small");
  const Shapes s = shapes(m, M);
  char* w = static_cast<char*>(ws);
  float2* stats = reinterpret_cast<float2*>(w + L.stats);
  // statistics and final-norm image of the given rows; clears the head
  // GEMM's split-K counters (a kernel, not a memset node, so the call stays
  // safe under graph capture)
  RowsArgs ra{};
  ra.hidden = hidden;
  ra.M = M;
  ra.MT = L.MT;
  ra.d = m->cfg.d_model;
  ra.n_slots = M;
  ra.vocab = m->cfg.vocab;
  ra.stats = stats;
  ra.img = ImageOut{reinterpret_cast<uint16_t*>(w + L.img_f), T(m, MSD_T_FINAL_G)};
  ra.zero_i32 = reinterpret_cast<int32_t*>(w + L.counters);
  ra.n_zero = L.n_counters;
  MSD_HIP(launch_rows(ra, stream));
  return run_head(m, s, L, w, M, stats, kappa, nullptr, ids, logp, nullptr, nullptr, stream);
}

msd_status msd_accept(const msd_model* m, const msd_block* blk, const float* logits,
                      const int32_t* argmax, const msd_sampling* smp, int32_t* acc_len,
                      int32_t* next_tok, int32_t* path, uint8_t* near_tie, uint32_t* status,
                      void* ws, size_t ws_bytes, hipStream_t stream) {
  msd_status st = check_block(m, blk, false);
  if (st != MSD_OK) return st;
  if (!acc_len || !next_tok || !path) return fail(MSD_ERR_INVALID_ARG, "null output");
  Topo topo;
  st = make_topo(blk, &topo);
  if (st != MSD_OK) return st;
  AcceptArgs a{};
  a.mode = smp ? smp->mode : MSD_GREEDY;
  if (a.mode == MSD_GREEDY) {
    if (!argmax) return fail(MSD_ERR_INVALID_ARG, "GREEDY needs argmax");
  } else if (a.mode == MSD_REJECTION || a.mode == MSD_MATCH) {
    if (!logits) return fail(MSD_ERR_INVALID_ARG, "stochastic acceptance needs logits");
    if (!(smp->temperature > 0.0f)) return fail(MSD_ERR_INVALID_ARG, "temperature must be > 0");
    if (!smp->u_sample) return fail(MSD_ERR_INVALID_ARG, "null u_sample");
    if (a.mode == MSD_REJECTION) {
      if (smp->n_cand < 1 || smp->n_cand > 64) return fail(MSD_ERR_INVALID_ARG, "n_cand out of [1, 64]");
      if (!smp->cand_ids || !smp->cand_q || !smp->u_accept)
        return fail(MSD_ERR_INVALID_ARG, "REJECTION needs cand_ids, cand_q and u_accept");
    }
  } else {
    return fail(MSD_ERR_UNSUPPORTED, "unknown acceptance mode");
  }
  const float tol = smp ? smp->tol_logit : 0.0f;
  if (!(tol >= 0.0f) || !std::isfinite(tol)) return fail(MSD_ERR_INVALID_ARG, "tol_logit must be finite and >= 0");
  if (near_tie && !logits) return fail(MSD_ERR_INVALID_ARG, "near-tie flags need logits");
  a.near_tie = near_tie;
  a.tol_logit = tol;
  a.temperature = smp ? smp->temperature : 1.0f;
  a.batch = blk->batch;
  a.n_slots = blk->n_slots;
  a.vocab = m->cfg.vocab;
  a.n_cand = smp ? smp->n_cand : 0;
  a.tokens = blk->tokens;
  a.logits = logits;
  a.argmax = argmax;
  a.cand_ids = smp ? smp->cand_ids : nullptr;
  a.cand_q = smp ? smp->cand_q : nullptr;
  a.u_accept = smp ? smp->u_accept : nullptr;
  a.u_sample = smp ? smp->u_sample : nullptr;
  a.acc_len = acc_len;
  a.next_tok = next_tok;
  a.path = path;
  a.status = status;
  a.topo = topo;
  if (a.mode == MSD_REJECTION && !status) return fail(MSD_ERR_INVALID_ARG, "REJECTION needs a status word");
  // the stochastic modes' vocabulary statistics in the caller's workspace
  // when it holds them (16-byte aligned); otherwise the walk's own passes
  const size_t stat_bytes = (size_t)blk->batch * blk->n_slots * kAcceptStatChunks * sizeof(double2);
  if (a.mode != MSD_GREEDY && ws && ws_bytes >= stat_bytes && ((uintptr_t)ws & 15) == 0)
    a.stats = reinterpret_cast<double2*>(ws);
  MSD_HIP(launch_accept(a, stream));
  return MSD_OK;
}

msd_status msd_kv_commit(const msd_model* m, msd_kv_cache* kv, const msd_block* blk,
                         const int32_t* acc_len, const int32_t* path, hipStream_t stream) {
  msd_status st = check_block(m, blk, false);
  if (st != MSD_OK) return st;
  if (!kv || !kv->k || !kv->v || !kv->len) return fail(MSD_ERR_INVALID_ARG, "null kv cache field");
  if (!acc_len || !path) return fail(MSD_ERR_INVALID_ARG, "null acc_len or path");
  if (blk->batch > kv->batch_cap) return fail(MSD_ERR_SHAPE, "batch exceeds the cache's batch_cap");
  Topo topo;
  st = make_topo(blk, &topo);
  if (st != MSD_OK) return st;
  bool chain = true;
  for (int i = 1; i < blk->n_slots; ++i) chain = chain && topo.parent[i] == i - 1;
  CommitArgs a{};
  a.k_cache = static_cast<uint16_t*>(kv->k);
  a.v_cache = static_cast<uint16_t*>(kv->v);
  a.len = kv->len;
  a.acc_len = acc_len;
  a.path = path;
  a.n_layers = m->cfg.n_layers;
  a.batch = blk->batch;
  a.batch_cap = kv->batch_cap;
  a.n_kv_heads = m->cfg.n_kv_heads;
  a.capacity = kv->capacity;
  a.head_dim = m->cfg.head_dim;
  a.n_slots = blk->n_slots;
  a.copy_rows = chain ? 0 : 1;
  if (blk->n_slots < 2) a.copy_rows = 0;
  MSD_HIP(launch_commit(a, stream));
  return MSD_OK;
}

msd_status msd_reuse_select(const msd_model* m, const msd_block* blk, const int32_t* acc_len,
                            const int32_t* next_tok, const int32_t* path, const msd_hyp_tree* tree,
                            const float* logits, const float* lse, const int32_t* ee_ids,
                            int32_t kappa, int32_t* next_case, int32_t* next_node, float* omega,
                            msd_reuse_stats* stats, hipStream_t stream) {
  msd_status st = check_block(m, blk);
  if (st != MSD_OK) return st;
  if (!acc_len || !next_tok || !path || !next_case || !next_node)
    return fail(MSD_ERR_INVALID_ARG, "null accept outputs or selection outputs");
  if (!tree || !tree->parent || !tree->tokens) return fail(MSD_ERR_INVALID_ARG, "null hypothesis tree");
  if (tree->n_nodes < 1 || tree->n_nodes > kMaxTreeNodes)
    return fail(MSD_ERR_SHAPE, "hypothesis tree n_nodes must lie in [1, 256]");
  const bool om = logits || lse || ee_ids;
  if (om && !(logits && lse && ee_ids)) return fail(MSD_ERR_INVALID_ARG, "Omega needs logits, lse and ee_ids");
  if (om && (kappa < 1 || kappa > kMaxKappa)) return fail(MSD_ERR_INVALID_ARG, "kappa out of [1, 32]");
  ReuseArgs a{};
  a.tree.n_nodes = tree->n_nodes;
  for (int i = 0; i < tree->n_nodes; ++i) {
    const int p = tree->parent[i];
    if (p != -1 && (p < 0 || p >= i)) return fail(MSD_ERR_SHAPE, "tree parent[i] must be -1 or lie in [0, i)");
    const int d = p < 0 ? 1 : a.tree.depth[p] + 1;
    a.tree.parent[i] = (int16_t)p;
    a.tree.depth[i] = (uint8_t)(d < 255 ? d : 255);  // deeper than any block never matches
  }
  a.batch = blk->batch;
  a.n_slots = blk->n_slots;
  a.tokens = blk->tokens;
  a.acc_len = acc_len;
  a.next_tok = next_tok;
  a.path = path;
  a.tree_tokens = tree->tokens;
  a.logits = om ? logits : nullptr;
  a.lse = lse;
  a.ee_ids = ee_ids;
  a.kappa = kappa;
  a.vocab = m->cfg.vocab;
  a.next_case = next_case;
  a.next_node = next_node;
  a.omega = omega;
  a.stats = reinterpret_cast<ReuseStats*>(stats);
  MSD_HIP(launch_reuse(a, stream));
  return MSD_OK;
}

msd_status msd_set_profile(msd_model* m, int32_t kclass, hipEvent_t* begin, hipEvent_t* end,
                           int32_t n) {
  if (!m) return fail(MSD_ERR_INVALID_ARG, "null model");
  m->prof_begin.clear();
  m->prof_end.clear();
  m->prof_class = -1;
  if (n <= 0) return MSD_OK;
  if (!begin || !end) return fail(MSD_ERR_INVALID_ARG, "null event arrays");
  if (kclass < MSD_K_QKV || kclass > MSD_K_FFN_DOWN) return fail(MSD_ERR_INVALID_ARG, "kernel class");
  m->prof_begin.assign(begin, begin + n);
  m->prof_end.assign(end, end + n);
  m->prof_class = kclass;
  return MSD_OK;
}

}  // extern "C"
