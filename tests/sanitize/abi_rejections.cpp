// The C ABI's host-side validation under AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Test infrastructure: built host-only together with csrc/api.hip, with the kernel
// launchers replaced by the stubs below (each returns an error, so a call that passes
// validation reports DUSTIN_ERR_LAUNCH and never touches a device).  Every call hands the
// library fake, aligned device addresses that validation must never dereference, and real
// host arrays where the ABI takes host memory.  Prints one line per failed expectation and
// exits non-zero if any failed.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../paper_2606_24957_amd/csrc/kernels.hpp"

namespace dustin {
hipError_t launch_verify_attn(const AttnArgs&, int, bool, bool, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_score(const ScoreArgs&, int, int, int, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_score_sync(const SyncArgs&, hipStream_t) { return hipErrorInvalidValue; }
bool score_sync_pair_supported(const SyncCall&, const SyncCall&) { return false; }
hipError_t launch_score_sync_pair(const SyncArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_arr(const ArrArgs&, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_page_meta(const PageMetaArgs&, int, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_topk(const TopkArgs&, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_kv_append(const KvAppendArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_kv_commit(int32_t*, const int32_t*, const int32_t*, int, int, hipStream_t) {
  return hipErrorInvalidValue;
}
hipError_t launch_read_probe(const void*, uint64_t, uint32_t*, int, hipStream_t) { return hipErrorInvalidValue; }
}  // namespace dustin

static int failures = 0;
#define EXPECT(call, want)                                                                    \
  do {                                                                                        \
    const int got_ = (int)(call);                                                             \
    if (got_ != (int)(want)) {                                                                \
      printf("FAIL line %d: %s -> %d, expected %d\n", __LINE__, #call, got_, (int)(want));    \
      ++failures;                                                                             \
    }                                                                                         \
  } while (0)

static void* const FAKE = reinterpret_cast<void*>(0x10000);
static void* fake(size_t off) { return reinterpret_cast<char*>(FAKE) + off; }

static dustin_batch batch(int B = 2, int max_len = 100, int nq = 4, int k_max = 40, int m = 10) {
  dustin_batch bt;
  memset(&bt, 0, sizeof bt);
  bt.batch = B;
  bt.max_len = max_len;
  bt.nq_max = nq;
  bt.k_max = k_max;
  bt.m_scalar = m;
  bt.seq_lens = static_cast<const int32_t*>(FAKE);
  return bt;
}

static dustin_kv kv(int Hkv = 2, int d = 128, int cap = 200) {
  dustin_kv k;
  memset(&k, 0, sizeof k);
  k.data = FAKE;
  k.num_kv_heads = Hkv;
  k.head_dim = d;
  k.stride_n = Hkv * d;
  k.stride_h = d;
  k.stride_b = (int64_t)cap * Hkv * d;
  k.capacity = cap;
  return k;
}

static int topk(const dustin_batch& bt, const void* sd = FAKE, const void* st = FAKE, int groups = 1,
                void* idx = FAKE, void* ws = FAKE, size_t ws_bytes = (size_t)1 << 30) {
  return dustin_topk(static_cast<const float*>(sd), 0, 0, static_cast<const float*>(st), 0, 0, &bt, groups, 4, 16,
                     static_cast<int32_t*>(idx), 0, 0, static_cast<int32_t*>(FAKE), nullptr, nullptr, ws, ws_bytes,
                     nullptr);
}

static int attn(int Hq = 8, dustin_kv k = kv(), dustin_kv v = kv(), dustin_batch bt = batch(), const void* q = FAKE,
                const void* idx = FAKE, int groups = 1, float scale = 0.1f, void* ws = nullptr, size_t ws_bytes = 0,
                int64_t q_sb = 800 * 8 * 128) {
  return dustin_sparse_verify_attn(q, q_sb, 8 * 128, 128, Hq, &k, &v, &bt, static_cast<const int32_t*>(idx), 0, 0,
                                   static_cast<const int32_t*>(FAKE), groups, scale, FAKE, 800 * 8 * 128, 8 * 128,
                                   128, ws, ws_bytes, nullptr);
}

static int score(const int* heads, int n_heads, int Hq = 8, dustin_kv k = kv(), dustin_batch bt = batch(),
                 int groups = 1, void* ws = FAKE, size_t ws_bytes = (size_t)1 << 30) {
  return dustin_score(FAKE, 800 * 8 * 128, 8 * 128, 128, Hq, heads, n_heads, &k, &bt, 0.1f, groups, nullptr, 0, 0,
                      static_cast<float*>(FAKE), 0, 0, ws, ws_bytes, nullptr);
}

int main() {
  // ---- status strings
  for (int s = 0; s <= 5; ++s)
    if (!dustin_status_string(s)[0] || !strcmp(dustin_status_string(s), "unknown status")) ++failures;
  if (strcmp(dustin_status_string(99), "unknown status") != 0 || strcmp(dustin_status_string(-1), "unknown status") != 0)
    ++failures;

  // ---- top-k
  EXPECT(topk(batch(2, 100, 4, 19)), DUSTIN_ERR_INVALID_ARG);  // k < sinks + window
  EXPECT(topk(batch(2, 100, 4, 40, 21)), DUSTIN_ERR_INVALID_ARG);
  EXPECT(topk(batch(2, 100, 4, 40, -1)), DUSTIN_ERR_INVALID_ARG);
  EXPECT(topk(batch(2, 100, 4, 40, 3), nullptr), DUSTIN_ERR_INVALID_ARG);
  EXPECT(topk(batch(2, 100, 4, 40, 3), FAKE, nullptr), DUSTIN_ERR_INVALID_ARG);
  EXPECT(topk(batch(), nullptr, nullptr), DUSTIN_ERR_INVALID_ARG);
  EXPECT(topk(batch(), FAKE, FAKE, 1, nullptr), DUSTIN_ERR_INVALID_ARG);
  EXPECT(topk(batch(), FAKE, FAKE, 0), DUSTIN_ERR_INVALID_ARG);
  EXPECT(topk(batch(2, (1 << 19) + 1)), DUSTIN_ERR_UNSUPPORTED);
  {
    dustin_batch bt = batch();
    bt.seq_lens = nullptr;
    EXPECT(topk(bt), DUSTIN_ERR_INVALID_ARG);
  }
  EXPECT(topk(batch(), FAKE, FAKE, 1, FAKE, nullptr, 0), DUSTIN_ERR_WORKSPACE);  // the tiers' hand-off
  EXPECT(topk(batch(), FAKE, FAKE, 1, FAKE, fake(4)), DUSTIN_ERR_WORKSPACE);
  EXPECT(topk(batch(2, 100, 4, 40, 0), nullptr, FAKE, 1, FAKE, nullptr, 0), DUSTIN_ERR_LAUNCH);  // one tier: none
  EXPECT(topk(batch()), DUSTIN_ERR_LAUNCH);  // valid: reaches the (stubbed) launch

  // ---- sparse and dense attention
  EXPECT(attn(8, kv(), kv(), batch(), nullptr), DUSTIN_ERR_INVALID_ARG);
  EXPECT(attn(8, kv(), kv(), batch(), FAKE, nullptr), DUSTIN_ERR_INVALID_ARG);
  EXPECT(attn(7), DUSTIN_ERR_INVALID_ARG);                                  // Hq % Hkv
  EXPECT(attn(8, kv(), kv(), batch(), FAKE, FAKE, 3), DUSTIN_ERR_INVALID_ARG);  // groups
  EXPECT(attn(8, kv(), kv(), batch(), fake(2)), DUSTIN_ERR_INVALID_ARG);   // 16-byte rows
  EXPECT(attn(8, kv(), kv(), batch(), FAKE, FAKE, 1, 0.1f, nullptr, 0, 4), DUSTIN_ERR_INVALID_ARG);
  EXPECT(attn(8, kv(), kv(), batch(), FAKE, FAKE, 1, __builtin_nanf("")), DUSTIN_ERR_INVALID_ARG);
  EXPECT(attn(8, kv(2, 64), kv(2, 64)), DUSTIN_ERR_UNSUPPORTED);          // head_dim 128 only
  EXPECT(attn(8, kv(2, 128, 103)), DUSTIN_ERR_INVALID_ARG);               // capacity < max_len + T
  EXPECT(attn(8, kv(), kv(4)), DUSTIN_ERR_INVALID_ARG);
  EXPECT(attn(64, kv(2), kv(2), batch(2, 100, 5)), DUSTIN_ERR_UNSUPPORTED);  // 160 rows per KV head
  {
    dustin_kv paged = kv();
    paged.page_table = static_cast<const int32_t*>(FAKE);
    paged.page_size = 12;
    paged.max_pages = 20;
    paged.num_pages = 40;
    paged.stride_page = 12 * 256;
    EXPECT(attn(8, paged, paged), DUSTIN_ERR_INVALID_ARG);  // page size not a power of two
    EXPECT(attn(8, paged, kv()), DUSTIN_ERR_INVALID_ARG);   // K paged, V not
  }
  const size_t need = dustin_attn_workspace(1, 8, 2, 4, 40, 1);
  if (need) {
    EXPECT(attn(8, kv(), kv(), batch(1)), DUSTIN_ERR_WORKSPACE);
    EXPECT(attn(8, kv(), kv(), batch(1), FAKE, FAKE, 1, 0.1f, fake(8), need), DUSTIN_ERR_WORKSPACE);
    EXPECT(attn(8, kv(), kv(), batch(1), FAKE, FAKE, 1, 0.1f, FAKE, need), DUSTIN_ERR_LAUNCH);
  }
  {
    dustin_kv k = kv();
    dustin_batch bt = batch();
    EXPECT(dense_verify_attn(nullptr, 800 * 8 * 128, 8 * 128, 128, 8, &k, &k, &bt, 0.1f, FAKE, 800 * 8 * 128,
                             8 * 128, 128, nullptr, 0, nullptr),
           DUSTIN_ERR_INVALID_ARG);
    EXPECT(dense_verify_attn(FAKE, 800 * 8 * 128, 8 * 128, 128, 8, &k, &k, nullptr, 0.1f, FAKE, 800 * 8 * 128,
                             8 * 128, 128, nullptr, 0, nullptr),
           DUSTIN_ERR_INVALID_ARG);
  }

  // ---- the no-allocation attention: validation, then the scratch limit, before any HIP call
  {
    dustin_kv k = kv(8, 128, 400);
    dustin_batch bt = batch(32, 300, 16, 256);
    setenv("DUSTIN_ATTN_SPLITS", "32", 1);
    EXPECT(dustin_sparse_verify_attn_noalloc(FAKE, 800 * 8 * 128, 8 * 128, 128, 64, &k, &k, &bt,
                                             static_cast<const int32_t*>(FAKE), 0, 0,
                                             static_cast<const int32_t*>(FAKE), 1, 0.1f, FAKE, 800 * 8 * 128,
                                             8 * 128, 128, nullptr),
           DUSTIN_ERR_SCRATCH_LIMIT);
    unsetenv("DUSTIN_ATTN_SPLITS");
    EXPECT(dustin_sparse_verify_attn_noalloc(nullptr, 800 * 8 * 128, 8 * 128, 128, 64, &k, &k, &bt,
                                             static_cast<const int32_t*>(FAKE), 0, 0,
                                             static_cast<const int32_t*>(FAKE), 1, 0.1f, FAKE, 800 * 8 * 128,
                                             8 * 128, 128, nullptr),
           DUSTIN_ERR_INVALID_ARG);
  }

  // ---- score
  {
    const int h_bad[2] = {0, 8}, h_dup[2] = {2, 2}, h_ok[2] = {0, 3};
    int h65[65];
    for (int i = 0; i < 65; ++i) h65[i] = i;
    EXPECT(score(h_bad, 2), DUSTIN_ERR_INVALID_ARG);
    EXPECT(score(h_dup, 2), DUSTIN_ERR_INVALID_ARG);
    EXPECT(score(h_ok, 0), DUSTIN_ERR_UNSUPPORTED);
    EXPECT(score(h65, 65, 128), DUSTIN_ERR_UNSUPPORTED);
    EXPECT(score(h_ok, 2, 8, kv(), batch(), 3), DUSTIN_ERR_INVALID_ARG);
    EXPECT(score(h_ok, 2, 8, kv(2, 96)), DUSTIN_ERR_UNSUPPORTED);
    EXPECT(score(h_ok, 2, 8, kv(), batch(2, 100, 17)), DUSTIN_ERR_UNSUPPORTED);
    EXPECT(score(h_ok, 2, 8, kv(), batch(), 1, nullptr, 0), DUSTIN_ERR_WORKSPACE);
    EXPECT(score(h_ok, 2, 8, kv(), batch(), 1, fake(4)), DUSTIN_ERR_WORKSPACE);
    EXPECT(score(h_ok, 2, 8, kv(), batch(), 1, FAKE, 16), DUSTIN_ERR_WORKSPACE);
    EXPECT(score(h_ok, 2), DUSTIN_ERR_LAUNCH);
    // per-layer and multi-layer forms over host arrays of layers
    dustin_kv ks[2] = {kv(), kv()}, mixed[2] = {kv(), kv(2, 128, 300)};
    const void* qs[2] = {FAKE, FAKE};
    dustin_batch bt = batch();
    EXPECT(dustin_score_per_layer(0, qs, 800 * 8 * 128, 8 * 128, 128, 8, h_ok, 2, ks, &bt, 0.1f, 1,
                                  static_cast<float*>(FAKE), 1 << 20, 0, 0, FAKE, (size_t)1 << 30, nullptr),
           DUSTIN_ERR_UNSUPPORTED);
    EXPECT(dustin_score_per_layer(2, qs, 800 * 8 * 128, 8 * 128, 128, 8, h_ok, 2, mixed, &bt, 0.1f, 1,
                                  static_cast<float*>(FAKE), 1 << 20, 0, 0, FAKE, (size_t)1 << 30, nullptr),
           DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_score_layers(2, qs, 800 * 8 * 128, 8 * 128, 128, 8, h_ok, 2, ks, &bt, 0.1f, 1, nullptr, 0, 0,
                               static_cast<float*>(FAKE), 0, 0, FAKE, (size_t)1 << 30, nullptr),
           DUSTIN_ERR_LAUNCH);
    // one or two calls in one launch
    dustin_score_call c[3];
    memset(c, 0, sizeof c);
    for (int i = 0; i < 3; ++i) {
      c[i].n_layers = 2;
      c[i].q_layers_host = qs;
      c[i].q_sb = 800 * 8 * 128;
      c[i].q_sj = 8 * 128;
      c[i].q_sh = 128;
      c[i].num_q_heads = 8;
      c[i].heads_host = h_ok;
      c[i].n_heads = 2;
      c[i].k_layers_host = ks;
      c[i].bt = &bt;
      c[i].scale = 0.1f;
      c[i].groups = 1;
      c[i].out = static_cast<float*>(FAKE);
      c[i].workspace = fake((size_t)i << 30);
      c[i].workspace_bytes = (size_t)1 << 30;
    }
    EXPECT(dustin_score_calls(0, c, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_score_calls(3, c, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_score_calls(1, nullptr, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_score_calls(2, c, nullptr), DUSTIN_ERR_LAUNCH);  // valid: reaches the (stubbed) launch
    c[1].workspace = c[0].workspace;
    EXPECT(dustin_score_calls(2, c, nullptr), DUSTIN_ERR_WORKSPACE);
    c[1].workspace = fake((size_t)1 << 30);
    c[1].heads_host = h_dup;
    EXPECT(dustin_score_calls(2, c, nullptr), DUSTIN_ERR_INVALID_ARG);
  }

  // ---- page estimator
  {
    dustin_kv k = kv();
    dustin_batch bt = batch();
    const int sp = 2 * 2 * 128;
    EXPECT(dustin_page_meta(&k, &bt, nullptr, 100, 12, FAKE, 7 * sp, sp, 7, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_page_meta(&k, &bt, nullptr, 100, 16, FAKE, 6 * sp, sp, 6, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_page_meta(&k, &bt, nullptr, 101, 16, FAKE, 7 * sp, sp, 7, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_page_meta(&k, &bt, static_cast<const int32_t*>(fake(2)), 100, 16, FAKE, 7 * sp, sp, 7, nullptr),
           DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_page_meta(nullptr, &bt, nullptr, 10, 16, FAKE, 7 * sp, sp, 7, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_page_meta(&k, &bt, nullptr, 100, 16, FAKE, 7 * sp, sp, 7, nullptr), DUSTIN_ERR_LAUNCH);
    const int h[2] = {0, 3};
    EXPECT(dustin_page_score(FAKE, 800 * 8 * 128, 8 * 128, 128, 8, h, 2, FAKE, 7 * sp, sp, 7, 2, 128, 3, &bt, 0.1f,
                             1, nullptr, 0, 0, static_cast<float*>(FAKE), 0, 0, FAKE, (size_t)1 << 30, nullptr),
           DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_page_score(FAKE, 800 * 8 * 128, 8 * 128, 128, 8, h, 2, FAKE, 7 * sp, sp, 7, 2, 128, 16, &bt, 0.1f,
                             1, nullptr, 0, 0, static_cast<float*>(FAKE), 0, 0, FAKE, 64, nullptr),
           DUSTIN_ERR_WORKSPACE);
  }

  // ---- attention recovery rate, KV append and commit
  {
    dustin_batch bt = batch();
    EXPECT(dustin_arr(nullptr, 100, 0, static_cast<const int32_t*>(FAKE), 40, 40, static_cast<const int32_t*>(FAKE),
                      &bt, 1, 8, static_cast<double*>(FAKE), nullptr),
           DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_arr(static_cast<const float*>(FAKE), 100, 0, static_cast<const int32_t*>(FAKE), 40, 40,
                      static_cast<const int32_t*>(FAKE), &bt, 1, 8, static_cast<double*>(fake(4)), nullptr),
           DUSTIN_ERR_INVALID_ARG);
    dustin_kv k = kv();
    EXPECT(dustin_kv_append(FAKE, 8 * 256, 256, 128, FAKE, 8 * 256, 256, 128, &k, &k, &bt, nullptr), DUSTIN_ERR_LAUNCH);
    EXPECT(dustin_kv_append(fake(2), 8 * 256, 256, 128, FAKE, 8 * 256, 256, 128, &k, &k, &bt, nullptr),
           DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_kv_commit(static_cast<int32_t*>(FAKE), nullptr, nullptr, 2, 4, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_kv_commit(static_cast<int32_t*>(FAKE), static_cast<const int32_t*>(FAKE), nullptr, -1, 4, nullptr),
           DUSTIN_ERR_INVALID_ARG);
  }
  {  // the streaming-read probe
    uint32_t* sums = static_cast<uint32_t*>(FAKE);
    EXPECT(dustin_read_probe(nullptr, 4096, sums, 4, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_read_probe(FAKE, 4096, nullptr, 4, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_read_probe(fake(8), 4096, sums, 4, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_read_probe(FAKE, 4100, sums, 4, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_read_probe(FAKE, 4096, sums, 0, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_read_probe(FAKE, 4096, sums, 65537, nullptr), DUSTIN_ERR_INVALID_ARG);
    EXPECT(dustin_read_probe(FAKE, (size_t)1 << 32, sums, 1, nullptr), DUSTIN_ERR_UNSUPPORTED);
    EXPECT(dustin_read_probe(FAKE, 4096, sums, 4, nullptr), DUSTIN_ERR_LAUNCH);
  }

  printf("%s: %d failed expectations\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
