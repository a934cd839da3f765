// api.hip -- the extern "C" boundary of libdustin: argument validation, workspace
// layout, launch configuration.  Validation happens before any HIP call, so a rejected
// call touches neither the device nor any output.
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include "kernels.hpp"
#include "probe.hpp"

using namespace dustin;

namespace {

constexpr size_t kAlign = 256;
constexpr int kTopkMaxLen = 1 << 19;

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

bool rows_aligned(const void* p, int64_t s0, int64_t s1, int64_t s2) {
  // bf16 rows read or written 16 bytes at a time
  return aligned(p, 16) && s0 % 8 == 0 && s1 % 8 == 0 && s2 % 8 == 0;
}

int env_int(const char* name, int fallback) {
  const char* v = getenv(name);
  if (!v || !*v) return fallback;
  const int x = atoi(v);
  return x > 0 ? x : fallback;
}

bool batch_ok(const dustin_batch* bt) {
  if (!bt || bt->batch < 0 || bt->max_len < 0 || bt->nq_max < 0 || bt->k_max < 0) return false;
  if (bt->batch > 0 && !bt->seq_lens) return false;
  return true;
}

SeqDims dims_of(const dustin_batch* bt) {
  SeqDims d;
  d.seq_lens = bt->seq_lens;
  d.n_query = bt->n_query;
  d.budget = bt->budget;
  d.m = bt->m;
  d.max_len = bt->max_len;
  d.nq_max = bt->nq_max;
  d.k_max = bt->k_max;
  d.m_scalar = bt->m_scalar;
  return d;
}

// Validates a cache view for `need` addressable positions per sequence.
dustin_status kv_of(const dustin_kv* kv, int head_dim, int64_t need, KvView* out) {
  if (!kv || !kv->data || kv->num_kv_heads <= 0) return DUSTIN_ERR_INVALID_ARG;
  if (kv->head_dim != head_dim) return DUSTIN_ERR_INVALID_ARG;
  if (!aligned(kv->data, 16) || kv->stride_n % 8 || kv->stride_h % 8 || kv->stride_b % 8 ||
      kv->stride_page % 8)
    return DUSTIN_ERR_INVALID_ARG;
  if (kv->stride_n <= 0 || kv->stride_h < 0 || kv->stride_b < 0) return DUSTIN_ERR_INVALID_ARG;
  memset(out, 0, sizeof *out);
  out->data = static_cast<const uint16_t*>(kv->data);
  out->stride_b = kv->stride_b;
  out->stride_n = kv->stride_n;
  out->stride_h = kv->stride_h;
  if (kv->page_table) {
    const int ps = kv->page_size;
    if (ps <= 0 || (ps & (ps - 1)) || kv->max_pages <= 0 || kv->num_pages <= 0 ||
        kv->stride_page <= 0)
      return DUSTIN_ERR_INVALID_ARG;
    if (!aligned(kv->page_table, 4)) return DUSTIN_ERR_INVALID_ARG;
    int shift = 0;
    while ((1 << shift) < ps) ++shift;
    out->page_table = kv->page_table;
    out->page_shift = shift;
    out->max_pages = kv->max_pages;
    out->num_pages = kv->num_pages;
    out->stride_page = kv->stride_page;
    out->capacity = (int64_t)kv->max_pages * ps;
    if (((int64_t)kv->num_pages << shift) > INT32_MAX) return DUSTIN_ERR_UNSUPPORTED;
  } else {
    out->capacity = kv->capacity;
  }
  if (out->capacity < need || out->capacity <= 0) return DUSTIN_ERR_INVALID_ARG;
  if (!kv->page_table && out->capacity > INT32_MAX) return DUSTIN_ERR_UNSUPPORTED;
  return DUSTIN_OK;
}

int attn_row_tiles(int nq_max, int group_size) {
  const int rows = nq_max * group_size;
  int rt = (rows + 15) / 16;
  if (rt == 7) rt = 8;  // instantiated tile counts: 1..6 and 8
  return rt < 1 ? 1 : rt;
}

// Unit slots per (b, g): enough workgroups for one per CU (256 CUs, one workgroup of four
// waves each), each split at least 8 steps of 32 tokens (two per wave) for the longest
// pair.  The kernel then sizes the splits from the actual per-pair lengths, so that longer
// pairs take more of the slots; beyond kAttnBalancePairs pairs each pair is one workgroup.
int attn_splits(int batch, int num_kv_heads, int64_t tokens_per_pair) {
  const int64_t pairs = (int64_t)batch * num_kv_heads;
  if (pairs <= 0) return 1;
  const int64_t steps = (tokens_per_pair + 31) / 32;
  int64_t s;
  const int forced = env_int("DUSTIN_ATTN_SPLITS", 0);
  if (pairs > kAttnBalancePairs) return 1;
  if (forced > 0) {
    s = forced;
  } else {
    s = (256 + pairs - 1) / pairs;
    if (s > steps / 8) s = steps / 8;
  }
  if (s > kAttnMaxSplits) s = kAttnMaxSplits;
  if (s > steps) s = steps;
  return s < 1 ? 1 : (int)s;
}

// Split workspace: a fixed counter region first (one int32 per (b, g) for up to
// kAttnMaxPairs pairs, zero between calls whatever shape used it last), then the partials.
constexpr int64_t kAttnMaxPairs = 65536;

struct AttnWs {
  size_t counters, acc, ml, total;
};

AttnWs attn_ws_layout(int batch, int num_kv_heads, int rows_pad, int splits) {
  AttnWs w{0, 0, 0, 0};
  if (splits <= 1) return w;
  const size_t pairs = (size_t)batch * num_kv_heads;
  w.counters = kAttnMaxPairs * sizeof(int32_t);
  w.acc = round_up(pairs * splits * rows_pad * 128 * sizeof(float), kAlign);
  w.ml = round_up(pairs * splits * rows_pad * 2 * sizeof(float), kAlign);
  w.total = w.counters + w.acc + w.ml;
  return w;
}

size_t attn_ws_bytes(int batch, int num_q_heads, int num_kv_heads, int nq_max, int64_t tokens) {
  if (batch <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads) return 0;
  const int rt = attn_row_tiles(nq_max, num_q_heads / num_kv_heads);
  const int splits = attn_splits(batch, num_kv_heads, tokens + nq_max);
  return attn_ws_layout(batch, num_kv_heads, rt * 16, splits).total;
}

// A validated attention call: its kernel arguments (workspace fields still unset), the row
// tiles and cache kind that pick the kernel, and the workspace it needs.  `empty` marks a
// valid call with nothing to compute.
struct AttnCall {
  AttnArgs a;
  int rt;
  bool paged, empty;
  size_t need_ws;
};

dustin_status prepare_attention(bool sparse, const void* q, int64_t q_sb, int64_t q_st, int64_t q_sh,
                                int32_t num_q_heads, const dustin_kv* k, const dustin_kv* v,
                                const dustin_batch* bt, const int32_t* idx, int64_t idx_sb,
                                int64_t idx_sg, const int32_t* count, int32_t groups, float scale,
                                void* out, int64_t o_sb, int64_t o_st, int64_t o_sh, AttnCall* call) {
  memset(call, 0, sizeof *call);
  if (!batch_ok(bt) || !q || !out || !k || !v) return DUSTIN_ERR_INVALID_ARG;
  if (!isfinite(scale) || !(scale > 0.f)) return DUSTIN_ERR_INVALID_ARG;
  const int Hkv = k->num_kv_heads;
  if (num_q_heads <= 0 || Hkv <= 0 || num_q_heads % Hkv || v->num_kv_heads != Hkv)
    return DUSTIN_ERR_INVALID_ARG;
  if (k->head_dim != 128 || v->head_dim != 128) return DUSTIN_ERR_UNSUPPORTED;
  if (bt->max_len > INT32_MAX - 64) return DUSTIN_ERR_UNSUPPORTED;  // positions N_b + t are int32
  if (k->page_table != v->page_table) return DUSTIN_ERR_INVALID_ARG;  // one table for K and V
  if (k->page_table && (k->page_size != v->page_size || k->max_pages != v->max_pages ||
                        k->num_pages != v->num_pages))
    return DUSTIN_ERR_INVALID_ARG;
  if (!rows_aligned(q, q_sb, q_st, q_sh) || !rows_aligned(out, o_sb, o_st, o_sh))
    return DUSTIN_ERR_INVALID_ARG;
  const int gs = num_q_heads / Hkv;
  if ((int64_t)bt->nq_max * gs > 128) return DUSTIN_ERR_UNSUPPORTED;
  if ((int64_t)bt->batch * Hkv > kAttnMaxPairs) return DUSTIN_ERR_UNSUPPORTED;
  if (sparse) {
    if (!idx || !count || (groups != 1 && groups != Hkv)) return DUSTIN_ERR_INVALID_ARG;
    if (!aligned(idx, 4) || !aligned(count, 4) || idx_sb < 0 || idx_sg < 0)
      return DUSTIN_ERR_INVALID_ARG;
  }
  const int64_t need = (int64_t)bt->max_len + bt->nq_max;
  KvView kv, vv;
  dustin_status st = kv_of(k, 128, need, &kv);
  if (st != DUSTIN_OK) return st;
  st = kv_of(v, 128, need, &vv);
  if (st != DUSTIN_OK) return st;
  // the attention kernels address a row as base + 32-bit byte offset (row * stride_n * 2),
  // with row = page * page_size + slot for a paged cache: pages must be packed back to back
  for (const KvView* c : {&kv, &vv}) {
    if (c->page_table && c->stride_page != ((int64_t)1 << c->page_shift) * c->stride_n)
      return DUSTIN_ERR_UNSUPPORTED;
    const int64_t rows = c->page_table ? ((int64_t)c->num_pages << c->page_shift) : c->capacity;
    if ((rows - 1) * c->stride_n * 2 + 256 > (int64_t)UINT32_MAX) return DUSTIN_ERR_UNSUPPORTED;
  }
  const int B = bt->batch;
  if (B == 0 || bt->nq_max == 0) {
    call->empty = true;
    return DUSTIN_OK;
  }
  const int64_t tokens = sparse ? (int64_t)bt->k_max : (int64_t)bt->max_len;
  call->need_ws = attn_ws_bytes(B, num_q_heads, Hkv, bt->nq_max, tokens);

  AttnArgs& a = call->a;
  a.q = static_cast<const uint16_t*>(q);
  a.q_sb = q_sb;
  a.q_st = q_st;
  a.q_sh = q_sh;
  a.out = static_cast<uint16_t*>(out);
  a.o_sb = o_sb;
  a.o_st = o_st;
  a.o_sh = o_sh;
  a.k = kv;
  a.v = vv;
  a.dims = dims_of(bt);
  a.idx = idx;
  a.idx_sb = idx_sb;
  a.idx_sg = idx_sg;
  a.count = count;
  a.groups = sparse ? groups : 1;
  a.num_kv_heads = Hkv;
  a.group_size = gs;
  a.pairs = B * Hkv;
  a.scale_log2 = scale * kLog2e;
  const int rt = attn_row_tiles(bt->nq_max, gs);
  a.rows_pad = rt * 16;
  const int64_t tokens_max = tokens + bt->nq_max;
  a.splits = attn_splits(B, Hkv, tokens_max);
  const bool sep = rt <= kAttnSepMaxRT;  // the kernels give the window a step of its own there
  // 32-token steps of the longest pair that the splits share: its selected (or committed)
  // tokens, with the window's tokens as a step of their own when sep is set
  const int64_t steps_max = sep ? (tokens > 0 ? (tokens + 31) / 32 : 1) : (tokens_max + 31) / 32;
  a.split_steps = (int)((steps_max + a.splits - 1) / a.splits);
  a.min_split_steps = env_int("DUSTIN_ATTN_SPLITS", 0) > 0 ? 1 : 8;
  call->rt = rt;
  call->paged = kv.page_table != nullptr;
  return DUSTIN_OK;
}

// Points the split fields at a workspace of at least call.need_ws bytes and launches.
dustin_status launch_attention(AttnCall& call, bool sparse, void* ws, void* stream) {
  AttnArgs& a = call.a;
  if (a.splits > 1) {
    const AttnWs w = attn_ws_layout(a.pairs / a.num_kv_heads, a.num_kv_heads, a.rows_pad, a.splits);
    char* base = static_cast<char*>(ws);
    a.counters = reinterpret_cast<int32_t*>(base);
    a.part_acc = reinterpret_cast<float*>(base + w.counters);
    a.part_ml = reinterpret_cast<float*>(base + w.counters + w.acc);
  }
  const hipError_t e = launch_verify_attn(a, call.rt, sparse, call.paged, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DUSTIN_OK : DUSTIN_ERR_LAUNCH;
}

dustin_status run_attention(bool sparse, const void* q, int64_t q_sb, int64_t q_st, int64_t q_sh,
                            int32_t num_q_heads, const dustin_kv* k, const dustin_kv* v,
                            const dustin_batch* bt, const int32_t* idx, int64_t idx_sb,
                            int64_t idx_sg, const int32_t* count, int32_t groups, float scale,
                            void* out, int64_t o_sb, int64_t o_st, int64_t o_sh, void* ws,
                            size_t ws_bytes, void* stream) {
  AttnCall call;
  const dustin_status st = prepare_attention(sparse, q, q_sb, q_st, q_sh, num_q_heads, k, v, bt, idx, idx_sb,
                                             idx_sg, count, groups, scale, out, o_sb, o_st, o_sh, &call);
  if (st != DUSTIN_OK || call.empty) return st;
  if (call.need_ws && (!ws || ws_bytes < call.need_ws || !aligned(ws, kAlign))) return DUSTIN_ERR_WORKSPACE;
  return launch_attention(call, sparse, ws, stream);
}

}  // namespace

extern "C" {

const char* dustin_status_string(int32_t status) {
  switch (status) {
    case DUSTIN_OK: return "ok";
    case DUSTIN_ERR_INVALID_ARG: return "invalid argument";
    case DUSTIN_ERR_UNSUPPORTED: return "unsupported configuration";
    case DUSTIN_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case DUSTIN_ERR_LAUNCH: return "kernel launch failed";
    case DUSTIN_ERR_SCRATCH_LIMIT:
      return "the call needs more split scratch than the no-allocation entry point's fixed array holds";
  }
  return "unknown status";
}

int32_t dustin_version(void) { return (1 << 16) | 0; }

// ------------------------------------------------------------------ score

namespace {

// workspace of one score call: the single-pass form's counters (kScoreSyncBytes, zero
// between calls, at the start whatever form a call takes), then fp32 logits rows of `cols`
// entries (a multiple of 64) and per-chunk statistics, for `rows` (layer, sequence, head,
// query) rows.  The single-pass form keeps its per-chunk statistics where the logits go.
size_t score_ws_bytes(size_t rows, size_t cols, size_t chunk) {
  const size_t ld = round_up(cols, 64);
  const size_t n_chunks = (cols + chunk - 1) / chunk;
  return kScoreSyncBytes + round_up(rows * ld * sizeof(float), kAlign) +
         round_up(rows * n_chunks * 2 * sizeof(float), kAlign);
}

// The single-pass form (score_sync.hip) for a call with at most 16 (head, query) pairs over
// at most 4 KV heads, one output group and one output (a's heads, layers, cache view, dims,
// output and workspace fields set): fills sc and returns true, or false when the call
// takes the two-pass form.
bool score_sync_plan(const ScoreArgs& a, int32_t n_heads, int32_t nq_max, int row_dim, int B, int64_t max_len,
                     int32_t groups, int32_t* sync_region, size_t logits_bytes, SyncCall& sc) {
  if (a.page_mode || a.per_layer || groups != 1 || B > kScoreSyncMaxBatch) return false;
  if (row_dim != 64 && row_dim != 128) return false;
  if ((int64_t)n_heads * nq_max > 16) return false;
  memset(&sc, 0, sizeof sc);
  // used KV heads in ascending order; columns KV head by KV head, then head slot, then query
  int nu = 0;
  for (int i = 0; i < n_heads; ++i) {
    const int g = a.heads[i] / a.group_size;
    int at = 0;
    while (at < nu && sc.kv[at] < g) ++at;
    if (at < nu && sc.kv[at] == g) continue;
    if (nu == 4) return false;
    for (int v = nu; v > at; --v) sc.kv[v] = sc.kv[v - 1];
    sc.kv[at] = g;
    ++nu;
  }
  if (nu == 0) return false;
  int np = 0;
  for (int u = 0; u < nu; ++u)
    for (int i = 0; i < n_heads; ++i) {
      if (a.heads[i] / a.group_size != sc.kv[u]) continue;
      for (int jq = 0; jq < nq_max; ++jq) {
        sc.col_head[np] = a.heads[i];
        sc.col_query[np] = (uint8_t)jq;
        sc.col_u[np] = (uint8_t)u;
        ++np;
      }
    }
  // Chunks of 256 tw positions: eight tiles per wave once the batch fills the chip with
  // them.  The form keeps one workgroup on a CU for the whole call, so it is taken only
  // when every chunk the sizes allow gets a CU at once (beyond that, the two-pass form's
  // many small workgroups balance the load better).
  int tw = (int64_t)B * max_len >= (int64_t)192 * 2048 ? 8 : 2;
  int64_t chunks = (max_len + 256 * tw - 1) / (256 * tw);
  if (chunks > kScoreSyncMaxChunks && tw == 2) {  // long sequences of a small batch
    tw = 8;
    chunks = (max_len + 256 * tw - 1) / (256 * tw);
  }
  if (chunks > kScoreSyncMaxChunks || (int64_t)B * chunks > kScoreSyncCUs) return false;
  if ((size_t)a.n_layers * B * chunks * 16 * 2 * sizeof(float) > logits_bytes) return false;
  // every K row the kernel reads lies within 2^31 bytes of its buffer resource's base (a
  // sequence's rows, or the page pool)
  const int64_t rows_bytes = a.k.page_table
                                 ? (int64_t)(a.k.num_pages - 1) * a.k.stride_page * 2 +
                                       (int64_t)((1 << a.k.page_shift) - 1) * a.k.stride_n * 2
                                 : (a.k.capacity - 1) * a.k.stride_n * 2;
  const int64_t extent = rows_bytes + (int64_t)sc.kv[nu - 1] * a.k.stride_h * 2 + (int64_t)row_dim * 2;
  if (rows_bytes < 0 || extent > INT32_MAX) return false;
  for (int l = 0; l < a.n_layers; ++l) {
    sc.q_layers[l] = a.q_layers[l];
    sc.k_layers[l] = a.k_layers[l];
  }
  sc.q_sb = a.q_sb;
  sc.q_sj = a.q_sj;
  sc.q_sh = a.q_sh;
  sc.k = a.k;
  sc.dims = a.dims;
  sc.init = a.init;
  sc.init_sb = a.init_sb;
  sc.out = a.out;
  sc.out_sb = a.out_sb;
  sc.stats = a.logits;  // the per-chunk statistics go where the two-pass form's logits do
  sc.sync = sync_region;
  sc.scale_log2 = a.scale_log2;
  sc.batch = B;
  sc.n_layers = a.n_layers;
  sc.head_dim = row_dim;
  sc.nu = nu;
  sc.tw = tw;
  sc.np = np;
  sc.chunks = (int32_t)chunks;
  // a sequence's chunks on one XCD when they fit there with the other sequences of that XCD
  sc.local = (B + 7) / 8 * chunks <= kScoreSyncCUs / 8 ? 1 : 0;
  sc.extent = (int32_t)extent;
  return true;
}

int log2_exact(int x) {
  int s = 0;
  while ((1 << s) < x) ++s;
  return s;
}

// The scoring heads and their pass-1 column tiles: every (head, query) pair, KV head by
// KV head, at most 16 pairs per tile; then the pass-1 workgroups, each up to
// kScoreGroupTiles consecutive tiles of one KV head (its rows are read once for all).
dustin_status score_pairs(ScoreArgs& a, const int32_t* heads_host, int32_t n_heads, int32_t num_q_heads,
                          int32_t gs, int32_t nq_max, int* n_groups, int* max_group) {
  for (int i = 0; i < n_heads; ++i) {
    const int h = heads_host[i];
    if (h < 0 || h >= num_q_heads) return DUSTIN_ERR_INVALID_ARG;
    for (int j = 0; j < i; ++j)
      if (heads_host[j] == h) return DUSTIN_ERR_INVALID_ARG;
    a.heads[i] = h;
  }
  int nt = 0;
  for (int g = 0; g < num_q_heads / gs; ++g) {
    int u = -1;  // the open tile of KV head g
    for (int i = 0; i < n_heads; ++i) {
      if (heads_host[i] / gs != g) continue;
      for (int jq = 0; jq < nq_max; ++jq) {
        if (u < 0 || a.pairs_per_kv[u] == 16) {
          if (nt == kScoreMaxEntries) return DUSTIN_ERR_UNSUPPORTED;
          u = nt++;
          a.used_kv[u] = g;
        }
        a.pair_head[u * 16 + a.pairs_per_kv[u]] = (uint8_t)i;
        a.pair_query[u * 16 + a.pairs_per_kv[u]] = (uint8_t)jq;
        a.pairs_per_kv[u]++;
      }
    }
  }
  int ng = 0, mg = 0;
  for (int u = 0; u < nt; ++u) {
    if (ng > 0 && a.used_kv[a.tile_first[ng - 1]] == a.used_kv[u] && a.tile_count[ng - 1] < kScoreGroupTiles) {
      a.tile_count[ng - 1]++;
    } else {
      a.tile_first[ng] = (uint8_t)u;
      a.tile_count[ng] = 1;
      ++ng;
    }
    if (a.tile_count[ng - 1] > mg) mg = a.tile_count[ng - 1];
  }
  *n_groups = ng;
  *max_group = mg;
  return DUSTIN_OK;
}

bool score_io_ok(const float* init, int64_t init_sb, int64_t init_sg, const float* out, int64_t out_sb,
                 int64_t out_sg) {
  if (!out || !aligned(out, 4) || out_sb < 0 || out_sg < 0) return false;
  return !init || (aligned(init, 4) && init_sb >= 0 && init_sg >= 0);
}

// A validated score call, ready to launch: the two-pass arguments, and the single-pass
// form's when the call takes it.
struct ScorePrep {
  ScoreArgs a;
  int n_groups = 0, max_group = 0, row_dim = 0, B = 0;
  bool empty = false;  // nothing to compute
  bool sync = false;
  SyncCall sc;
};

// Fills the output, size and workspace fields of P.a (heads, layers, k view, dims already
// set) for `cols` rows per sequence at most, and plans the single-pass form.
dustin_status score_fill(ScorePrep& P, int row_dim, int B, int32_t nq_max, int64_t cols, float scale,
                         int32_t groups, const float* init, int64_t init_sb, int64_t init_sg, float* out,
                         int64_t out_sb, int64_t out_sg, void* workspace, size_t workspace_bytes) {
  ScoreArgs& a = P.a;
  const size_t rows = (size_t)a.n_layers * B * a.n_heads * nq_max;
  const size_t need_ws = score_ws_bytes(rows, (size_t)cols, (size_t)a.chunk);
  if (!workspace || workspace_bytes < need_ws || !aligned(workspace, kAlign)) return DUSTIN_ERR_WORKSPACE;
  a.batch = B;
  a.groups = groups;
  a.scale_log2 = scale * kLog2e;
  a.init = init;
  a.init_sb = init_sb;
  a.init_sg = init_sg;
  a.out = out;
  a.out_sb = out_sb;
  a.out_sg = out_sg;
  a.nq_max = nq_max;
  a.ld = (int64_t)round_up((size_t)cols, 64);
  a.n_chunks = (int32_t)((cols + a.chunk - 1) / a.chunk);
  char* const base = static_cast<char*>(workspace);
  a.logits = reinterpret_cast<float*>(base + kScoreSyncBytes);
  const size_t logits_bytes = round_up(rows * a.ld * sizeof(float), kAlign);
  a.stats = reinterpret_cast<float*>(base + kScoreSyncBytes + logits_bytes);
  P.row_dim = row_dim;
  P.B = B;
  P.sync = score_sync_plan(a, a.n_heads, nq_max, row_dim, B, cols, groups, reinterpret_cast<int32_t*>(base),
                           logits_bytes, P.sc);
  return DUSTIN_OK;
}

dustin_status score_run(const ScorePrep& P, void* stream) {
  if (P.empty) return DUSTIN_OK;
  hipError_t e;
  if (P.sync) {
    SyncArgs sa;
    memset(&sa, 0, sizeof sa);
    sa.call[0] = P.sc;
    e = launch_score_sync(sa, static_cast<hipStream_t>(stream));
  } else {
    e = launch_score(P.a, P.B, P.n_groups, P.max_group, P.row_dim, static_cast<hipStream_t>(stream));
  }
  return e == hipSuccess ? DUSTIN_OK : DUSTIN_ERR_LAUNCH;
}

// Validates Eq. 5 for n_layers layers that share shapes, summed into one output (or each
// layer into its own with per_layer), and fills P.
dustin_status prepare_score(ScorePrep& P, int32_t n_layers, const void* const* q_layers, int64_t q_sb,
                            int64_t q_sj, int64_t q_sh, int32_t num_q_heads, const int32_t* heads_host,
                            int32_t n_heads, const dustin_kv* k_layers, const dustin_batch* bt, float scale,
                            int32_t groups, const float* init, int64_t init_sb, int64_t init_sg, float* out,
                            int64_t out_sb, int64_t out_sg, void* workspace, size_t workspace_bytes,
                            bool per_layer = false, int64_t out_sl = 0) {
  if (!batch_ok(bt) || !q_layers || !k_layers || !out || !heads_host) return DUSTIN_ERR_INVALID_ARG;
  if (n_layers < 1 || n_layers > kScoreMaxLayers) return DUSTIN_ERR_UNSUPPORTED;
  if (!isfinite(scale)) return DUSTIN_ERR_INVALID_ARG;
  if (n_heads < 1 || n_heads > kScoreMaxHeads) return DUSTIN_ERR_UNSUPPORTED;
  const dustin_kv* k = &k_layers[0];
  const int Hkv = k->num_kv_heads;
  if (num_q_heads <= 0 || Hkv <= 0 || num_q_heads % Hkv) return DUSTIN_ERR_INVALID_ARG;
  if (k->head_dim != 64 && k->head_dim != 128) return DUSTIN_ERR_UNSUPPORTED;
  if (groups != 1 && groups != Hkv) return DUSTIN_ERR_INVALID_ARG;
  if (bt->nq_max < 1 || bt->nq_max > 16) return DUSTIN_ERR_UNSUPPORTED;
  if ((int64_t)(per_layer ? 1 : n_layers) * n_heads * bt->nq_max > kScoreMaxPairs) return DUSTIN_ERR_UNSUPPORTED;
  if (per_layer && (init || out_sl < 0)) return DUSTIN_ERR_INVALID_ARG;
  for (int l = 0; l < n_layers; ++l) {
    if (!q_layers[l] || !rows_aligned(q_layers[l], q_sb, q_sj, q_sh)) return DUSTIN_ERR_INVALID_ARG;
    const dustin_kv* kl = &k_layers[l];
    // the layers' caches differ only in where they start
    if (!kl->data || kl->num_kv_heads != Hkv || kl->head_dim != k->head_dim || kl->stride_b != k->stride_b ||
        kl->stride_n != k->stride_n || kl->stride_h != k->stride_h || kl->capacity != k->capacity ||
        kl->page_table != k->page_table || kl->page_size != k->page_size || kl->max_pages != k->max_pages ||
        kl->num_pages != k->num_pages || kl->stride_page != k->stride_page)
      return DUSTIN_ERR_INVALID_ARG;
    if (!aligned(kl->data, 16)) return DUSTIN_ERR_INVALID_ARG;
  }
  if (!score_io_ok(init, init_sb, init_sg, out, out_sb, out_sg)) return DUSTIN_ERR_INVALID_ARG;

  ScoreArgs& a = P.a;
  memset(&a, 0, sizeof a);
  a.n_heads = n_heads;
  a.group_size = num_q_heads / Hkv;
  dustin_status st =
      score_pairs(a, heads_host, n_heads, num_q_heads, a.group_size, bt->nq_max, &P.n_groups, &P.max_group);
  if (st != DUSTIN_OK) return st;
  KvView kv;
  st = kv_of(k, k->head_dim, bt->max_len, &kv);
  if (st != DUSTIN_OK) return st;
  const int B = bt->batch;
  if (B == 0 || bt->max_len == 0) {
    P.empty = true;
    return DUSTIN_OK;
  }
  if ((int64_t)B * n_layers > 65535) return DUSTIN_ERR_UNSUPPORTED;
  for (int l = 0; l < n_layers; ++l) {
    a.q_layers[l] = static_cast<const uint16_t*>(q_layers[l]);
    a.k_layers[l] = static_cast<const uint16_t*>(k_layers[l].data);
  }
  a.n_layers = n_layers;
  a.q_sb = q_sb;
  a.q_sj = q_sj;
  a.q_sh = q_sh;
  a.k = kv;
  a.dims = dims_of(bt);
  a.chunk = kScoreChunk;
  a.per_layer = per_layer ? 1 : 0;
  a.out_sl = out_sl;
  if ((int64_t)groups * (per_layer ? n_layers : 1) > 65535) return DUSTIN_ERR_UNSUPPORTED;
  return score_fill(P, k->head_dim, B, bt->nq_max, bt->max_len, scale, groups, init, init_sb, init_sg, out, out_sb,
                    out_sg, workspace, workspace_bytes);
}

dustin_status run_score(int32_t n_layers, const void* const* q_layers, int64_t q_sb, int64_t q_sj,
                        int64_t q_sh, int32_t num_q_heads, const int32_t* heads_host, int32_t n_heads,
                        const dustin_kv* k_layers, const dustin_batch* bt, float scale, int32_t groups,
                        const float* init, int64_t init_sb, int64_t init_sg, float* out, int64_t out_sb,
                        int64_t out_sg, void* workspace, size_t workspace_bytes, void* stream,
                        bool per_layer = false, int64_t out_sl = 0) {
  ScorePrep P;
  const dustin_status st =
      prepare_score(P, n_layers, q_layers, q_sb, q_sj, q_sh, num_q_heads, heads_host, n_heads, k_layers, bt, scale,
                    groups, init, init_sb, init_sg, out, out_sb, out_sg, workspace, workspace_bytes, per_layer, out_sl);
  return st != DUSTIN_OK ? st : score_run(P, stream);
}

}  // namespace

size_t dustin_score_workspace(int32_t batch, int32_t max_len, int32_t nq_max, int32_t n_heads) {
  if (batch <= 0 || max_len <= 0 || nq_max <= 0 || n_heads <= 0) return 0;
  return score_ws_bytes((size_t)batch * n_heads * nq_max, (size_t)max_len, kScoreChunk);
}

dustin_status dustin_score(const void* q, int64_t q_sb, int64_t q_sj, int64_t q_sh,
                           int32_t num_q_heads, const int32_t* heads_host, int32_t n_heads,
                           const dustin_kv* k, const dustin_batch* bt, float scale,
                           int32_t groups, const float* init, int64_t init_sb, int64_t init_sg,
                           float* out, int64_t out_sb, int64_t out_sg, void* workspace,
                           size_t workspace_bytes, void* stream) {
  if (!q || !k) return DUSTIN_ERR_INVALID_ARG;
  const void* qs[1] = {q};
  return run_score(1, qs, q_sb, q_sj, q_sh, num_q_heads, heads_host, n_heads, k, bt, scale, groups, init,
                   init_sb, init_sg, out, out_sb, out_sg, workspace, workspace_bytes, stream);
}

dustin_status dustin_score_layers(int32_t n_layers, const void* const* q_layers_host, int64_t q_sb,
                                  int64_t q_sj, int64_t q_sh, int32_t num_q_heads,
                                  const int32_t* heads_host, int32_t n_heads,
                                  const dustin_kv* k_layers_host, const dustin_batch* bt, float scale,
                                  int32_t groups, const float* init, int64_t init_sb, int64_t init_sg,
                                  float* out, int64_t out_sb, int64_t out_sg, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  return run_score(n_layers, q_layers_host, q_sb, q_sj, q_sh, num_q_heads, heads_host, n_heads, k_layers_host,
                   bt, scale, groups, init, init_sb, init_sg, out, out_sb, out_sg, workspace, workspace_bytes,
                   stream);
}

dustin_status dustin_score_per_layer(int32_t n_layers, const void* const* q_layers_host, int64_t q_sb,
                                     int64_t q_sj, int64_t q_sh, int32_t num_q_heads,
                                     const int32_t* heads_host, int32_t n_heads,
                                     const dustin_kv* k_layers_host, const dustin_batch* bt, float scale,
                                     int32_t groups, float* out, int64_t out_sl, int64_t out_sb,
                                     int64_t out_sg, void* workspace, size_t workspace_bytes, void* stream) {
  return run_score(n_layers, q_layers_host, q_sb, q_sj, q_sh, num_q_heads, heads_host, n_heads, k_layers_host,
                   bt, scale, groups, nullptr, 0, 0, out, out_sb, out_sg, workspace, workspace_bytes, stream,
                   true, out_sl);
}

dustin_status dustin_score_calls(int32_t n_calls, const dustin_score_call* calls, void* stream) {
  if (n_calls < 1 || n_calls > 2 || !calls) return DUSTIN_ERR_INVALID_ARG;
  ScorePrep P[2];
  for (int i = 0; i < n_calls; ++i) {
    const dustin_score_call& c = calls[i];
    const dustin_status st =
        prepare_score(P[i], c.n_layers, c.q_layers_host, c.q_sb, c.q_sj, c.q_sh, c.num_q_heads, c.heads_host,
                      c.n_heads, c.k_layers_host, c.bt, c.scale, c.groups, c.init, c.init_sb, c.init_sg, c.out,
                      c.out_sb, c.out_sg, c.workspace, c.workspace_bytes);
    if (st != DUSTIN_OK) return st;
    if (c.digit_hist && !aligned(c.digit_hist, 16)) return DUSTIN_ERR_INVALID_ARG;
    P[i].a.hist = c.digit_hist;
    P[i].sc.hist = c.digit_hist;
  }
  if (n_calls == 2 && calls[0].digit_hist && calls[0].digit_hist == calls[1].digit_hist) return DUSTIN_ERR_INVALID_ARG;
  if (n_calls == 2 && calls[0].workspace == calls[1].workspace) return DUSTIN_ERR_WORKSPACE;
  if (n_calls == 2 && P[0].sync && P[1].sync && !P[0].empty && !P[1].empty &&
      score_sync_pair_supported(P[0].sc, P[1].sc)) {
    SyncArgs sa;
    memset(&sa, 0, sizeof sa);
    sa.call[0] = P[0].sc;
    sa.call[1] = P[1].sc;
    return launch_score_sync_pair(sa, static_cast<hipStream_t>(stream)) == hipSuccess ? DUSTIN_OK
                                                                                      : DUSTIN_ERR_LAUNCH;
  }
  for (int i = 0; i < n_calls; ++i) {
    const dustin_status st = score_run(P[i], stream);
    if (st != DUSTIN_OK) return st;
  }
  return DUSTIN_OK;
}

// ------------------------------------------------------------------ page estimator

namespace {

bool page_size_ok(int32_t page_size) {
  return page_size >= 1 && page_size <= kMaxPageSize && (page_size & (page_size - 1)) == 0;
}

int32_t pages_of(int32_t n, int32_t page_size) { return (int32_t)(((int64_t)n + page_size - 1) / page_size); }

// a page-statistics array as a K view whose rows (pages) hold 2 * head_dim values
dustin_status meta_view(const void* meta, int64_t meta_sb, int64_t meta_sp, int32_t meta_pages, int32_t Hkv,
                        int32_t head_dim, int32_t need_pages, KvView* out) {
  if (!meta || !aligned(meta, 16) || meta_sb < 0 || meta_sb % 8 || meta_sp % 8) return DUSTIN_ERR_INVALID_ARG;
  if (meta_sp < (int64_t)Hkv * 2 * head_dim || meta_pages < need_pages) return DUSTIN_ERR_INVALID_ARG;
  if (meta_pages <= 0) return DUSTIN_ERR_INVALID_ARG;
  memset(out, 0, sizeof *out);
  out->data = static_cast<const uint16_t*>(meta);
  out->stride_b = meta_sb;
  out->stride_n = meta_sp;
  out->stride_h = 2 * head_dim;
  out->capacity = meta_pages;
  return DUSTIN_OK;
}

}  // namespace

dustin_status dustin_page_meta(const dustin_kv* k, const dustin_batch* bt, const int32_t* from, int32_t max_span,
                               int32_t page_size, void* meta, int64_t meta_sb, int64_t meta_sp,
                               int32_t meta_pages, void* stream) {
  if (!batch_ok(bt) || !k) return DUSTIN_ERR_INVALID_ARG;
  if (!page_size_ok(page_size)) return DUSTIN_ERR_INVALID_ARG;
  if (k->head_dim != 64 && k->head_dim != 128) return DUSTIN_ERR_UNSUPPORTED;
  if (k->num_kv_heads <= 0 || k->num_kv_heads > 65535) return DUSTIN_ERR_INVALID_ARG;
  if (max_span < 0 || max_span > bt->max_len) return DUSTIN_ERR_INVALID_ARG;
  if (from && !aligned(from, 4)) return DUSTIN_ERR_INVALID_ARG;
  KvView kv, mv;
  dustin_status st = kv_of(k, k->head_dim, bt->max_len, &kv);
  if (st != DUSTIN_OK) return st;
  const int32_t P = pages_of(bt->max_len, page_size);
  st = meta_view(meta, meta_sb, meta_sp, meta_pages, k->num_kv_heads, k->head_dim, P, &mv);
  if (st != DUSTIN_OK) return st;
  const int B = bt->batch;
  if (B > 65535) return DUSTIN_ERR_UNSUPPORTED;
  if (B == 0 || bt->max_len == 0 || max_span == 0) return DUSTIN_OK;
  PageMetaArgs a;
  memset(&a, 0, sizeof a);
  a.k = kv;
  a.dims = dims_of(bt);
  a.from = from;
  a.meta = static_cast<uint16_t*>(meta);
  a.m_sb = meta_sb;
  a.m_sp = meta_sp;
  a.num_kv_heads = k->num_kv_heads;
  a.page_shift = log2_exact(page_size);
  // the span's pages, plus the partly filled page it may start in
  const int32_t span = pages_of(max_span, page_size) + (from ? 1 : 0);
  a.span_pages = span < P ? span : P;
  const hipError_t e = launch_page_meta(a, B, k->head_dim, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DUSTIN_OK : DUSTIN_ERR_LAUNCH;
}

size_t dustin_page_score_workspace(int32_t batch, int32_t max_len, int32_t page_size, int32_t nq_max,
                                   int32_t n_heads) {
  if (batch <= 0 || max_len <= 0 || nq_max <= 0 || n_heads <= 0 || !page_size_ok(page_size)) return 0;
  return score_ws_bytes((size_t)batch * n_heads * nq_max, (size_t)pages_of(max_len, page_size), kScorePageChunk);
}

dustin_status dustin_page_score(const void* q, int64_t q_sb, int64_t q_sj, int64_t q_sh, int32_t num_q_heads,
                                const int32_t* heads_host, int32_t n_heads, const void* meta, int64_t meta_sb,
                                int64_t meta_sp, int32_t meta_pages, int32_t num_kv_heads, int32_t head_dim,
                                int32_t page_size, const dustin_batch* bt, float scale, int32_t groups,
                                const float* init, int64_t init_sb, int64_t init_sg, float* out, int64_t out_sb,
                                int64_t out_sg, void* workspace, size_t workspace_bytes, void* stream) {
  if (!batch_ok(bt) || !q || !heads_host) return DUSTIN_ERR_INVALID_ARG;
  if (!isfinite(scale) || !page_size_ok(page_size)) return DUSTIN_ERR_INVALID_ARG;
  if (n_heads < 1 || n_heads > kScoreMaxHeads) return DUSTIN_ERR_UNSUPPORTED;
  if (num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads) return DUSTIN_ERR_INVALID_ARG;
  if (head_dim != 64 && head_dim != 128) return DUSTIN_ERR_UNSUPPORTED;
  if (groups != 1 && groups != num_kv_heads) return DUSTIN_ERR_INVALID_ARG;
  if (bt->nq_max < 1 || bt->nq_max > 16) return DUSTIN_ERR_UNSUPPORTED;
  if ((int64_t)n_heads * bt->nq_max > kScoreMaxPairs) return DUSTIN_ERR_UNSUPPORTED;
  if (!rows_aligned(q, q_sb, q_sj, q_sh)) return DUSTIN_ERR_INVALID_ARG;
  if (!score_io_ok(init, init_sb, init_sg, out, out_sb, out_sg)) return DUSTIN_ERR_INVALID_ARG;
  const int32_t P = pages_of(bt->max_len, page_size);
  ScorePrep sp;
  ScoreArgs& a = sp.a;
  memset(&a, 0, sizeof a);
  dustin_status st = meta_view(meta, meta_sb, meta_sp, meta_pages, num_kv_heads, head_dim, P, &a.k);
  if (st != DUSTIN_OK) return st;
  a.n_heads = n_heads;
  a.group_size = num_q_heads / num_kv_heads;
  int n_groups = 0, max_group = 0;
  st = score_pairs(a, heads_host, n_heads, num_q_heads, a.group_size, bt->nq_max, &n_groups, &max_group);
  if (st != DUSTIN_OK) return st;
  const int B = bt->batch;
  if (B > 65535) return DUSTIN_ERR_UNSUPPORTED;
  if (B == 0 || bt->max_len == 0) return DUSTIN_OK;
  a.q_layers[0] = static_cast<const uint16_t*>(q);
  a.k_layers[0] = a.k.data;
  a.n_layers = 1;
  a.q_sb = q_sb;
  a.q_sj = q_sj;
  a.q_sh = q_sh;
  a.dims = dims_of(bt);
  a.page_mode = 1;
  a.page_shift = log2_exact(page_size);
  a.chunk = kScorePageChunk;
  sp.n_groups = n_groups;
  sp.max_group = max_group;
  st = score_fill(sp, 2 * head_dim, B, bt->nq_max, P, scale, groups, init, init_sb, init_sg, out, out_sb, out_sg,
                  workspace, workspace_bytes);
  return st != DUSTIN_OK ? st : score_run(sp, stream);
}

// ------------------------------------------------------------------ attention recovery rate

dustin_status dustin_arr(const float* s, int64_t s_sb, int64_t s_sg, const int32_t* idx, int64_t idx_sb,
                         int64_t idx_sg, const int32_t* count, const dustin_batch* bt, int32_t groups,
                         int32_t heads_per_group, double* arr, void* stream) {
  if (!batch_ok(bt) || !s || !idx || !count || !arr) return DUSTIN_ERR_INVALID_ARG;
  if (groups < 1 || groups > 65535 || heads_per_group < 1) return DUSTIN_ERR_INVALID_ARG;
  if (!aligned(s, 4) || !aligned(idx, 4) || !aligned(count, 4) || !aligned(arr, 8)) return DUSTIN_ERR_INVALID_ARG;
  if (s_sb < 0 || s_sg < 0 || idx_sb < 0 || idx_sg < 0) return DUSTIN_ERR_INVALID_ARG;
  const int B = bt->batch;
  if (B > 65535) return DUSTIN_ERR_UNSUPPORTED;
  if (B == 0) return DUSTIN_OK;
  ArrArgs a;
  memset(&a, 0, sizeof a);
  a.s = s;
  a.s_sb = s_sb;
  a.s_sg = s_sg;
  a.idx = idx;
  a.idx_sb = idx_sb;
  a.idx_sg = idx_sg;
  a.count = count;
  a.dims = dims_of(bt);
  a.groups = groups;
  a.heads_per_group = heads_per_group;
  a.arr = arr;
  const hipError_t e = launch_arr(a, B, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DUSTIN_OK : DUSTIN_ERR_LAUNCH;
}

// ------------------------------------------------------------------ top-k

namespace {

// Top-k workspace: an arrival counter per (b, go) in a region of fixed size (kTopkMaxRows
// counters, whatever the call's shape, so that a buffer that served a call of another shape
// still reads zero there), then two bitmaps of the row's positions per (b, go) for the
// hand-off between its two tiers.  Beyond kTopkMaxRows rows there is no hand-off (and no
// workspace): the tiers of a row run one after the other in one workgroup.
constexpr int64_t kTopkMaxRows = 4096;

struct TopkWs {
  size_t counters, bitmaps, total;
  int32_t words;
};

TopkWs topk_ws_layout(int32_t batch, int32_t groups, int32_t max_len) {
  TopkWs w{0, 0, 0, 0};
  if (batch <= 0 || groups <= 0 || max_len <= 0) return w;
  const size_t rows = (size_t)batch * groups;
  if (rows > (size_t)kTopkMaxRows) return w;
  w.words = (max_len + 31) / 32;
  w.counters = kTopkMaxRows * sizeof(uint32_t);
  w.bitmaps = round_up(rows * 2 * (size_t)w.words * sizeof(uint32_t), kAlign);
  w.total = w.counters + w.bitmaps;
  return w;
}

}  // namespace

size_t dustin_topk_workspace(int32_t batch, int32_t groups, int32_t max_len) {
  return topk_ws_layout(batch, groups, max_len).total;
}

dustin_status dustin_topk(const float* s_draft, int64_t d_sb, int64_t d_sg,
                          const float* s_target, int64_t t_sb, int64_t t_sg,
                          const dustin_batch* bt, int32_t groups, int32_t n_sink,
                          int32_t n_window, int32_t* idx, int64_t idx_sb, int64_t idx_sg,
                          int32_t* count, uint32_t* hist_draft, uint32_t* hist_target, void* workspace,
                          size_t workspace_bytes, void* stream) {
  if (!batch_ok(bt) || !idx || !count) return DUSTIN_ERR_INVALID_ARG;
  if ((hist_draft && (!s_draft || !aligned(hist_draft, 16))) || (hist_target && (!s_target || !aligned(hist_target, 16))))
    return DUSTIN_ERR_INVALID_ARG;
  if ((hist_draft || hist_target) && groups != 1) return DUSTIN_ERR_INVALID_ARG;
  if (hist_draft && hist_draft == hist_target) return DUSTIN_ERR_INVALID_ARG;
  if (!s_draft && !s_target) return DUSTIN_ERR_INVALID_ARG;
  if (groups < 1 || groups > 65535 || n_sink < 0 || n_window < 0) return DUSTIN_ERR_INVALID_ARG;
  if (bt->max_len > kTopkMaxLen) return DUSTIN_ERR_UNSUPPORTED;
  const int P = n_sink + n_window;
  if (bt->k_max < P) return DUSTIN_ERR_INVALID_ARG;
  if (!bt->m && (bt->m_scalar < 0 || bt->m_scalar > bt->k_max - P)) return DUSTIN_ERR_INVALID_ARG;
  if (!s_draft && !bt->m && bt->m_scalar != 0) return DUSTIN_ERR_INVALID_ARG;
  if (!s_target && !bt->m && !bt->budget && bt->m_scalar != bt->k_max - P) return DUSTIN_ERR_INVALID_ARG;
  if (!aligned(idx, 4) || !aligned(count, 4) || idx_sb < 0 || idx_sg < 0) return DUSTIN_ERR_INVALID_ARG;
  if ((s_draft && (!aligned(s_draft, 4) || d_sb < 0 || d_sg < 0)) ||
      (s_target && (!aligned(s_target, 4) || t_sb < 0 || t_sg < 0)))
    return DUSTIN_ERR_INVALID_ARG;
  const int B = bt->batch;
  if (B == 0) return DUSTIN_OK;
  // with both score arrays the two tiers of a row run side by side and hand off through
  // the workspace
  const TopkWs w = topk_ws_layout(B, groups, bt->max_len);
  const bool hand_off = s_draft && s_target && w.total > 0;
  if (hand_off && (!workspace || workspace_bytes < w.total || !aligned(workspace, kAlign)))
    return DUSTIN_ERR_WORKSPACE;
  TopkArgs a;
  memset(&a, 0, sizeof a);
  if (hand_off) {
    a.counters = static_cast<uint32_t*>(workspace);
    a.bitmaps = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + w.counters);
    a.words = w.words;
  }
  a.s_draft = s_draft;
  a.d_sb = d_sb;
  a.d_sg = d_sg;
  a.s_target = s_target;
  a.t_sb = t_sb;
  a.t_sg = t_sg;
  a.dims = dims_of(bt);
  a.groups = groups;
  a.n_sink = n_sink;
  a.n_window = n_window;
  a.idx = idx;
  a.idx_sb = idx_sb;
  a.idx_sg = idx_sg;
  a.count = count;
  a.hist_d = hist_draft;
  a.hist_t = hist_target;
  const hipError_t e = launch_topk(a, B, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DUSTIN_OK : DUSTIN_ERR_LAUNCH;
}

// ------------------------------------------------------------------ KV append / commit

dustin_status dustin_kv_append(const void* k_new, int64_t k_sb, int64_t k_st, int64_t k_sh,
                               const void* v_new, int64_t v_sb, int64_t v_st, int64_t v_sh,
                               const dustin_kv* k, const dustin_kv* v, const dustin_batch* bt,
                               void* stream) {
  if (!batch_ok(bt) || !k_new || !v_new || !k || !v) return DUSTIN_ERR_INVALID_ARG;
  if (bt->batch == 0 || bt->nq_max == 0) return DUSTIN_OK;
  const int d = k->head_dim, H = k->num_kv_heads;
  if (d <= 0 || d % 8 || v->head_dim != d || v->num_kv_heads != H || H <= 0) return DUSTIN_ERR_INVALID_ARG;
  if (k->page_table != v->page_table) return DUSTIN_ERR_INVALID_ARG;
  if (!rows_aligned(k_new, k_sb, k_st, k_sh) || !rows_aligned(v_new, v_sb, v_st, v_sh))
    return DUSTIN_ERR_INVALID_ARG;
  if (k_sb < 0 || k_st < 0 || k_sh < 0 || v_sb < 0 || v_st < 0 || v_sh < 0) return DUSTIN_ERR_INVALID_ARG;
  KvAppendArgs a;
  memset(&a, 0, sizeof a);
  const int64_t need = (int64_t)bt->max_len + bt->nq_max;
  dustin_status st = kv_of(k, d, need, &a.k);
  if (st != DUSTIN_OK) return st;
  st = kv_of(v, d, need, &a.v);
  if (st != DUSTIN_OK) return st;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.k_sb = k_sb;
  a.k_st = k_st;
  a.k_sh = k_sh;
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.v_sb = v_sb;
  a.v_st = v_st;
  a.v_sh = v_sh;
  a.dims = dims_of(bt);
  a.batch = bt->batch;
  a.num_kv_heads = H;
  a.head_dim = d;
  const hipError_t e = launch_kv_append(a, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DUSTIN_OK : DUSTIN_ERR_LAUNCH;
}

dustin_status dustin_kv_commit(int32_t* seq_lens, const int32_t* accepted, const int32_t* n_query,
                               int32_t batch, int32_t nq_max, void* stream) {
  if (batch < 0 || nq_max < 0) return DUSTIN_ERR_INVALID_ARG;
  if (batch == 0) return DUSTIN_OK;
  if (!seq_lens || !accepted || !aligned(seq_lens, 4) || !aligned(accepted, 4) ||
      (n_query && !aligned(n_query, 4)))
    return DUSTIN_ERR_INVALID_ARG;
  const hipError_t e =
      launch_kv_commit(seq_lens, accepted, n_query, nq_max, batch, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DUSTIN_OK : DUSTIN_ERR_LAUNCH;
}

// ------------------------------------------------------------------ attention

size_t dustin_attn_workspace(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                             int32_t nq_max, int32_t max_tokens, int32_t sparse) {
  (void)sparse;
  if (nq_max <= 0 || max_tokens < 0) return 0;
  return attn_ws_bytes(batch, num_q_heads, num_kv_heads, nq_max, max_tokens);
}

dustin_status dustin_sparse_verify_attn(const void* q, int64_t q_sb, int64_t q_st,
                                        int64_t q_sh, int32_t num_q_heads, const dustin_kv* k,
                                        const dustin_kv* v, const dustin_batch* bt,
                                        const int32_t* idx, int64_t idx_sb, int64_t idx_sg,
                                        const int32_t* count, int32_t groups, float scale,
                                        void* out, int64_t o_sb, int64_t o_st, int64_t o_sh,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  return run_attention(true, q, q_sb, q_st, q_sh, num_q_heads, k, v, bt, idx, idx_sb, idx_sg,
                       count, groups, scale, out, o_sb, o_st, o_sh, workspace, workspace_bytes,
                       stream);
}

dustin_status dense_verify_attn(const void* q, int64_t q_sb, int64_t q_st, int64_t q_sh,
                                int32_t num_q_heads, const dustin_kv* k, const dustin_kv* v,
                                const dustin_batch* bt, float scale, void* out, int64_t o_sb,
                                int64_t o_st, int64_t o_sh, void* workspace,
                                size_t workspace_bytes, void* stream) {
  return run_attention(false, q, q_sb, q_st, q_sh, num_q_heads, k, v, bt, nullptr, 0, 0, nullptr,
                       1, scale, out, o_sb, o_st, o_sh, workspace, workspace_bytes, stream);
}

}  // extern "C"

// ------------------------------------------------------------------ attention without allocation
//
// The split partials and counters of dustin_sparse_verify_attn_noalloc live in this fixed
// array, one copy per GPU that the library runs on, held until the process ends.  In host
// code its name is only a stand-in: its device address comes from hipGetSymbolAddress, once
// per device, and only that address is handed to kernels.

static __device__ __align__(256) unsigned char scratch[DUSTIN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device, once looked up

__global__ void zero_words_kernel(uint32_t* p, uint32_t n) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0u;
}

// The current device's scratch address.  At the first call on a device it is looked up and
// the counter region (which must read zero before the first split call) is cleared by a
// fill kernel on `stream`, ahead of the call's own launch.
dustin_status device_scratch(hipStream_t stream, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return DUSTIN_ERR_LAUNCH;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DUSTIN_ERR_LAUNCH;
    const uint32_t words = (uint32_t)(kAttnMaxPairs * sizeof(int32_t) / 4);
    hipLaunchKernelGGL(zero_words_kernel, dim3(64), dim3(256), 0, stream, static_cast<uint32_t*>(p), words);
    if (hipGetLastError() != hipSuccess) return DUSTIN_ERR_LAUNCH;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return DUSTIN_OK;
}

}  // namespace

extern "C" dustin_status dustin_sparse_verify_attn_noalloc(
    const void* q, int64_t q_sb, int64_t q_st, int64_t q_sh, int32_t num_q_heads, const dustin_kv* k,
    const dustin_kv* v, const dustin_batch* bt, const int32_t* idx, int64_t idx_sb, int64_t idx_sg,
    const int32_t* count, int32_t groups, float scale, void* out, int64_t o_sb, int64_t o_st, int64_t o_sh,
    void* stream) {
  AttnCall call;
  dustin_status st = prepare_attention(true, q, q_sb, q_st, q_sh, num_q_heads, k, v, bt, idx, idx_sb, idx_sg,
                                       count, groups, scale, out, o_sb, o_st, o_sh, &call);
  if (st != DUSTIN_OK || call.empty) return st;
  if (call.need_ws > (size_t)DUSTIN_NOALLOC_SCRATCH_BYTES) return DUSTIN_ERR_SCRATCH_LIMIT;
  void* ws = nullptr;
  if (call.need_ws) {
    st = device_scratch(static_cast<hipStream_t>(stream), &ws);
    if (st != DUSTIN_OK) return st;
  }
  return launch_attention(call, true, ws, stream);
}

// ------------------------------------------------------------------ streaming-read probe

dustin_status dustin_read_probe(const void* data, size_t bytes, uint32_t* block_sums, int32_t blocks,
                                void* stream) {
  if (!data || !block_sums || blocks < 1 || blocks > 65536) return DUSTIN_ERR_INVALID_ARG;
  if (!aligned(data, 16) || !aligned(block_sums, 4) || bytes % 16) return DUSTIN_ERR_INVALID_ARG;
  if (bytes / 16 / (size_t)blocks + 1 >= ((size_t)1 << 31) / 16) return DUSTIN_ERR_UNSUPPORTED;
  const hipError_t e = launch_read_probe(data, bytes, block_sums, blocks, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DUSTIN_OK : DUSTIN_ERR_LAUNCH;
}

