// kernels.hpp -- argument blocks and launchers of the libdustin kernels (internal).
#pragma once

#include "common.hpp"

namespace dustin {

// ---- verification attention (attn.hip) ----
constexpr int kAttnMaxSplits = 32;  // token splits per (b, g)

struct AttnArgs {
  const uint16_t* q;
  int64_t q_sb, q_st, q_sh;
  uint16_t* out;
  int64_t o_sb, o_st, o_sh;
  KvView k, v;          // paged K and V share one page table and page size
  SeqDims dims;
  const int32_t* idx;   // NULL: dense (every committed position)
  int64_t idx_sb, idx_sg;
  const int32_t* count;
  int32_t groups;
  int32_t num_kv_heads, group_size;
  int32_t pairs;        // B * num_kv_heads
  float scale_log2;
  int32_t splits;           // unit slots per (b, g) on average: the grid holds pairs * splits
  int32_t split_steps;      // 32-token steps per split when every pair is as long as the longest
  int32_t min_split_steps;  // smallest split the kernel's balancing may choose
  int32_t rows_pad;
  float* part_acc;          // [pairs * splits, rows_pad, 128], by unit  (splits > 1 only)
  float* part_ml;           // [pairs * splits, rows_pad, 2]
  int32_t* counters;        // [pairs], zero between calls
};

// Row tiles (16 query rows each) up to which the attention kernel gives the verification
// window's tokens a step of their own; beyond that they share the last step with the
// selected (or committed) positions.
constexpr int kAttnSepMaxRT = 3;

// Pairs the attention kernel's split balancing handles (four per lane of one wave); with
// more pairs there is one workgroup per pair.
constexpr int kAttnBalancePairs = 256;

hipError_t launch_verify_attn(const AttnArgs& a, int rt, bool sparse, bool paged, hipStream_t stream);

// ---- scoring-head importance (score.hip) ----
constexpr int kScoreWaves = 4;
constexpr int kScoreChunk = 1024;        // positions per pass-1 workgroup (256 pages in page mode)
constexpr int kScorePageChunk = 256;
constexpr int kScoreFinishChunk = 1024;  // positions per pass-2 workgroup (4 per thread)
constexpr int kScoreFinishPages = 64;    // pages per pass-2 workgroup in page mode
constexpr int kScoreMaxHeads = 64;
constexpr int kScoreMaxEntries = 64;     // pass-1 column tiles: (KV head, up to 16 pairs)
constexpr int kScoreGroupTiles = 3;      // column tiles of one KV head per pass-1 workgroup
constexpr int kScoreMaxLayers = 32;
constexpr int kScoreMaxPairs = 1024;     // (layer, head, query) rows one output sums
// Single-pass form (score_sync.hip): the workspace starts with kScoreSyncBytes of
// per-sequence counters (zero between calls) and a timeout flag; every form of the score
// keeps its logits and statistics after them.
constexpr int kSyncWaves = 16;             // waves per single-pass workgroup
constexpr int kScoreSyncMaxBatch = 2048;   // sequences the counters cover
constexpr int kScoreSyncMaxChunks = 128;   // chunks of one sequence (far below the chip's CUs)
constexpr int kScoreSyncCUs = 256;         // MI355X compute units: one single-pass workgroup each
constexpr size_t kScoreSyncBytes = 16896;  // 2 * kScoreSyncMaxBatch counters + the flag, 256-aligned
static_assert(kScoreSyncBytes >= (2 * kScoreSyncMaxBatch + 1) * 4 && kScoreSyncBytes % 256 == 0, "sync region");
static_assert(kScoreSyncBytes == DUSTIN_SCORE_SYNC_BYTES && 2 * kScoreSyncMaxBatch * 4 == DUSTIN_SCORE_SYNC_FLAG_OFFSET,
              "the workspace layout the header documents");

// Eq. 5 over the positions of a cache, or (page mode) over the pages of a page-statistics
// array, whose rows [max | min] of length 2d meet the sign-split query [q+ | q-].
struct ScoreArgs {
  const uint16_t* q_layers[kScoreMaxLayers];  // queries of each scored layer (same strides)
  int64_t q_sb, q_sj, q_sh;
  KvView k;                                  // K view shared by the layers, but for its data
  const uint16_t* k_layers[kScoreMaxLayers];
  int32_t n_layers, batch;
  SeqDims dims;
  int32_t page_mode;   // 0: rows of k are positions; 1: rows are pages of page statistics
  int32_t page_shift;  // page mode: log2 of the page size (0 otherwise)
  int32_t chunk;       // rows per pass-1 workgroup
  int32_t heads[kScoreMaxHeads];
  int32_t n_heads;
  int32_t used_kv[kScoreMaxEntries];       // KV head of each pass-1 column tile
  int32_t pairs_per_kv[kScoreMaxEntries];  // (head, query) pairs of that tile
  uint8_t tile_first[kScoreMaxEntries];    // pass-1 workgroup x: its first tile
  uint8_t tile_count[kScoreMaxEntries];    // and its tile count (same KV head)
  uint8_t pair_head[kScoreMaxEntries * 16];   // head slot of pair i of tile u
  uint8_t pair_query[kScoreMaxEntries * 16];  // query of that pair
  int32_t group_size, groups;
  float scale_log2;
  const float* init;
  int64_t init_sb, init_sg;
  float* out;
  int64_t out_sb, out_sg;
  int32_t per_layer;  // 1: layer l writes out + l * out_sl (no init); 0: layers summed
  int64_t out_sl;
  float* logits;  // [n_layers, B, n_heads, nq_max, ld]  scaled logits, log2 domain
  float* stats;   // [n_layers, B, n_heads, nq_max, n_chunks, 2]  (max, sum of exp2) per chunk
  int64_t ld;
  int32_t nq_max, n_chunks;
  // optional: one count per written position added to hist[(b groups + go) kDigitBins +
  // order_key(out) >> 20] (summed outputs only)
  uint32_t* hist;
};
static_assert(sizeof(ScoreArgs) <= 4096, "kernel arguments stay within 4 KiB");

// n_groups pass-1 workgroups along x (tile_first / tile_count), max_group the largest
// tile count; row_dim: length of a K row (head_dim, or 2 * head_dim for page statistics)
hipError_t launch_score(const ScoreArgs& a, int B, int n_groups, int max_group, int row_dim, hipStream_t stream);

// One call of the single-pass form (score_sync.hip): columns 0 .. np - 1 are (query head
// col_head, query col_query) pairs on used KV head kv[col_u]; chunks of 256 tw positions,
// `chunks` per sequence, a sequence's chunks on one XCD when `local`.
struct SyncCall {
  const uint16_t* q_layers[kScoreMaxLayers];
  const uint16_t* k_layers[kScoreMaxLayers];
  int64_t q_sb, q_sj, q_sh;
  KvView k;
  SeqDims dims;
  const float* init;
  int64_t init_sb;
  float* out;
  int64_t out_sb;
  float* stats;   // [n_layers, batch, chunks, 16] (max, sum of exp2) per chunk and column
  int32_t* sync;  // the workspace's counter region (zero between calls) and timeout flag
  float scale_log2;
  int32_t batch, n_layers, head_dim, nu, tw, np, chunks, local;
  int32_t extent;  // bytes of K rows one buffer resource covers (a sequence, or the page pool)
  int32_t kv[4];
  int32_t col_head[16];
  uint8_t col_query[16], col_u[16];
  uint32_t* hist;  // optional: as ScoreArgs::hist (one output row per sequence)
};

struct SyncArgs {
  SyncCall call[2];
  int32_t blocks0;  // blocks of call 0 (set by the launcher)
};
static_assert(sizeof(SyncArgs) <= 4096, "kernel arguments stay within 4 KiB");

// the single-pass form of one call; and of two calls in one launch, for the pairs of
// shapes score_sync_pair_supported accepts
hipError_t launch_score_sync(const SyncArgs& a, hipStream_t stream);
bool score_sync_pair_supported(const SyncCall& c0, const SyncCall& c1);
hipError_t launch_score_sync_pair(const SyncArgs& a, hipStream_t stream);

// ---- attention recovery rate (arr.hip) ----
struct ArrArgs {
  const float* s;  // Eq. 5 score over the served heads and the window's queries
  int64_t s_sb, s_sg;
  const int32_t* idx;
  int64_t idx_sb, idx_sg;
  const int32_t* count;
  SeqDims dims;    // seq_lens (N_b), n_query (w_b), k_max
  int32_t groups, heads_per_group;
  double* arr;     // [B, groups]
};

hipError_t launch_arr(const ArrArgs& a, int B, hipStream_t stream);

// ---- page statistics for the page estimator (page.hip) ----
constexpr int kMaxPageSize = 4096;
struct PageMetaArgs {
  KvView k;
  SeqDims dims;
  const int32_t* from;  // device [B]: first position that changed, or NULL (= 0)
  uint16_t* meta;       // [B, pages, Hkv, 2 d]: per page, channel max then min
  int64_t m_sb, m_sp;
  int32_t num_kv_heads, page_shift, span_pages;
};

hipError_t launch_page_meta(const PageMetaArgs& a, int B, int head_dim, hipStream_t stream);

// ---- tiered selection (topk.hip) ----
struct TopkArgs {
  const float* s_draft;
  int64_t d_sb, d_sg;
  const float* s_target;
  int64_t t_sb, t_sg;
  SeqDims dims;
  int32_t groups, n_sink, n_window;
  int32_t* idx;
  int64_t idx_sb, idx_sg;
  int32_t* count;
  // hand-off between the two tiers of a row (both score arrays given): per (b, go) an
  // arrival counter (zero between calls) and two chosen-set bitmaps of `words` words
  uint32_t* counters;  // [B * groups]
  uint32_t* bitmaps;   // [B * groups][2][words]
  int32_t words;
  // optional (groups = 1): per sequence the top-digit histogram of the whole row of S_D /
  // S_T, which replaces the tier's first pass and is returned to zero
  uint32_t* hist_d;
  uint32_t* hist_t;
};

hipError_t launch_topk(const TopkArgs& a, int B, hipStream_t stream);

// ---- verification window K/V into the caches, and the commit of accepted tokens (kv.hip) ----
struct KvAppendArgs {
  const uint16_t* k_new;
  int64_t k_sb, k_st, k_sh;
  const uint16_t* v_new;
  int64_t v_sb, v_st, v_sh;
  KvView k, v;   // the caches (written)
  SeqDims dims;  // seq_lens (N_b), n_query (T_b), max_len, nq_max
  int32_t batch, num_kv_heads, head_dim;
};

hipError_t launch_kv_append(const KvAppendArgs& a, hipStream_t stream);
hipError_t launch_kv_commit(int32_t* seq_lens, const int32_t* accepted, const int32_t* n_query, int nq_max,
                            int batch, hipStream_t stream);

}  // namespace dustin
