/*
 * dustin.h -- C ABI of libdustin, the MI355X (gfx950) hot path of Dustin's sparse
 * verification step for long-context speculative decoding.
 *
 * One verification step is
 *   1. dustin_score  (target)           S_T = init_T + sum of scoring-head attention      Eq. 5
 *   2. dustin_score  (draft, per layer) S_D = init_D + sum over draft heads, layers, tokens Eq. 5
 *   3. dustin_topk                      I   = sinks U window U top-m(S_D) U top-rest(S_T)   Eq. 6
 *   4. dustin_sparse_verify_attn        attention of the gamma+1 verification queries over
 *                                       I plus the causal verification window, run for
 *                                       every target layer with the same I (global,
 *                                       layer-invariant selection, method section 4.1)
 * and dense_verify_attn is the full-cache verification attention the paper compares
 * against (Efficiency baselines; Appendix G).  Around the attention, dustin_kv_append
 * writes the verification window's K and V into the caches (per layer, before step 4)
 * and dustin_kv_commit keeps the accepted window tokens after verification.
 * dustin_page_meta and dustin_page_score are the page estimator the paper compares its
 * scoring heads with (page-level key minima and maxima; Quest-16 in the estimation
 * overhead analysis): they produce an importance array that step 3 takes in place of,
 * or on top of, S_T.  dustin_arr measures how much of the window's attention an index set
 * keeps (attention recovery rate), the paper's fidelity measure of a selection.
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are DEVICE pointers unless a name ends in _host.  The caller
 *     owns every buffer; the library never allocates, frees or synchronises.  Work is
 *     enqueued on `stream` (a hipStream_t; NULL = the null stream) and is asynchronous.
 *   - Strides are in elements, int64.  The innermost axis (head_dim or position) must be
 *     contiguous (stride 1).  bf16 means the 16-bit bfloat16 format.
 *   - Base pointers of bf16 tensors and their strides must keep 16-byte alignment of
 *     every row (a multiple of 8 elements); fp32/int32 tensors need 4-byte alignment.
 *   - Arguments are validated on the host before anything is enqueued; a non-OK status
 *     means nothing was enqueued and no output was touched.  Per-sequence values that
 *     live in device arrays (lengths, query counts, budgets, m, selected positions, page
 *     ids) cannot be checked on the host: kernels clamp them into the host-declared
 *     bounds (N_b into [0, max_len], T_b into [0, nq_max], k_b into
 *     [n_sink + n_window, k_max], m_b into [0, k_b - n_sink - n_window], positions into
 *     the cache capacity, page ids into [0, num_pages)), so no device value can make a
 *     kernel read or write outside the buffers the host arguments describe.
 *   - Verification tokens: sequence b has N_b committed positions [0, N_b) and T_b
 *     verification tokens (the last accepted token plus gamma_b drafts) whose K/V rows
 *     are already written at positions [N_b, N_b + T_b).  Query t in [0, T_b) attends
 *     to the selected positions plus N_b .. N_b + t (causal).  The verification tokens
 *     are not counted in the budget k.
 *   - GQA: query head h uses KV head h / (num_q_heads / num_kv_heads).
 *   - Selection groups: groups == 1 gives one index set per sequence (the paper's
 *     global set); groups == num_kv_heads gives one set per (sequence, KV head).
 *   - No exception or C++ object crosses this boundary; every function is reentrant.
 */
#ifndef DUSTIN_H
#define DUSTIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DUSTIN_OK = 0,
  DUSTIN_ERR_INVALID_ARG = 1, /* null pointer, bad size, bad stride or alignment         */
  DUSTIN_ERR_UNSUPPORTED = 2, /* valid but not implemented (head_dim, rows per group...) */
  DUSTIN_ERR_WORKSPACE = 3,   /* workspace missing, misaligned or smaller than required   */
  DUSTIN_ERR_LAUNCH = 4,      /* the HIP runtime refused a launch                          */
  DUSTIN_ERR_SCRATCH_LIMIT = 5 /* more split scratch than dustin_sparse_verify_attn_noalloc's
                                  fixed array holds                                        */
} dustin_status;

/* A bf16 K or V cache of one layer.
 *   contiguous (page_table == NULL): element (b, n, g, c) is at
 *       data[b * stride_b + n * stride_n + g * stride_h + c],  n < capacity
 *   paged: position n of sequence b lives in physical page p = page_table[b * max_pages +
 *       n / page_size] at data[p * stride_page + (n % page_size) * stride_n + g * stride_h + c];
 *       capacity = max_pages * page_size, p < num_pages, num_pages * page_size < 2^31.
 *       K and V of one attention call must share the same page table and page size.
 *   The attention entry points also need the rows of a cache to be reachable with a
 *   32-bit byte offset (rows * stride_n * 2 < 2^32, rows = capacity or num_pages *
 *   page_size) and, when paged, pages packed back to back (stride_page == page_size *
 *   stride_n); otherwise they return DUSTIN_ERR_UNSUPPORTED. */
typedef struct {
  const void* data;
  int32_t num_kv_heads;
  int32_t head_dim;
  int64_t stride_b;
  int64_t stride_n;
  int64_t stride_h;
  int64_t capacity;            /* positions addressable per sequence (contiguous mode) */
  const int32_t* page_table;   /* NULL = contiguous; else device int32 [B, max_pages]  */
  int32_t page_size;           /* paged: a power of two                                */
  int32_t max_pages;
  int32_t num_pages;           /* paged: physical pages in the pool                    */
  int64_t stride_page;
} dustin_kv;

/* Per-sequence sizes.  A NULL device array means "the scalar for every sequence". */
typedef struct {
  int32_t batch;               /* B                                                    */
  int32_t max_len;             /* upper bound of N_b                                   */
  int32_t nq_max;              /* upper bound of T_b (attention) or Gamma_b (score)    */
  int32_t k_max;               /* upper bound of the budget k_b (selection, sparse)    */
  const int32_t* seq_lens;     /* device int32 [B]: N_b (required)                     */
  const int32_t* n_query;      /* device int32 [B] or NULL (= nq_max)                  */
  const int32_t* budget;       /* device int32 [B] or NULL (= k_max)                   */
  const int32_t* m;            /* device int32 [B] or NULL (= m_scalar)                */
  int32_t m_scalar;
} dustin_batch;

/* Human-readable name of a status code (static storage); any other value gives
 * "unknown status".  The code is taken as a plain integer, so that a caller may pass any
 * value it holds. */
const char* dustin_status_string(int32_t status);

/* Library version, (major << 16) | minor. */
int32_t dustin_version(void);

/* ---------------------------------------------------------------------------------
 * dustin_score -- scoring-head importance, Eq. 5 (hybrid_importance) restricted to the
 * semantic retrieval heads (online sparse estimation, method section 4.2; Appendix A).
 *
 *   out[b, go, n] = init[b, go, n]
 *                 + sum_{h in heads, (groups == 1 or h's KV head == go)} sum_{j < nq_b}
 *                   softmax_{n' < N_b}(scale * q[b, j, h] . K[b, n', g(h)])[n]
 *
 * for n < N_b; positions n >= N_b of out are not written.  Used once for the target's
 * last generated token (nq_b = 1, init = the historical score or NULL) and once per draft
 * scoring layer (nq_b = Gamma_b draft tokens; chaining init = out accumulates layers).
 *   q        bf16 [B, nq_max, num_q_heads, head_dim], strides q_sb, q_sj, q_sh
 *   heads_host  host int32 [n_heads], 1 <= n_heads <= 64, distinct, in [0, num_q_heads);
 *               the (head, query) pairs, split by KV head into tiles of 16, fit 64 tiles
 *   k        the layer's K cache; head_dim in {64, 128}
 *   bt       seq_lens, n_query (1 <= nq_max <= 16), max_len
 *   groups   1 or k->num_kv_heads
 *   init     fp32 [B, groups, >= max_len] (strides init_sb, init_sg) or NULL (= 0)
 *   out      fp32 [B, groups, >= max_len] (strides out_sb, out_sg); may alias init
 *   workspace  device scratch of dustin_score_workspace() bytes, 256-byte aligned.  Its
 *              first DUSTIN_SCORE_SYNC_BYTES bytes must be zero before the first call;
 *              every call leaves them zero (the int32 at DUSTIN_SCORE_SYNC_FLAG_OFFSET
 *              aside, see below).  Calls that share a workspace must not overlap.
 * Rounding: fp32 dot products (bf16 products are exact), fp32 exp and sums.
 * Two forms compute the same sums.  When every (head, query) pair fits one 16-column
 * MFMA tile (n_heads * nq_max <= 16, scoring heads over at most 4 KV heads), groups == 1
 * and batch <= 2048, one launch does everything: each workgroup keeps the logits of a
 * chunk of positions in registers and the chunks of a sequence exchange only their
 * softmax statistics, through per-sequence counters at the start of the workspace (a
 * bounded wait; the chunks of a sequence are dispatched together and are few against the
 * GPU's compute units).  Should that wait ever time out, the kernel writes 1 to the
 * int32 at byte DUSTIN_SCORE_SYNC_FLAG_OFFSET of the workspace and its output is
 * unspecified; zero the first DUSTIN_SCORE_SYNC_BYTES bytes again before reusing the
 * workspace.  Otherwise the logits go through the workspace in two launches.
 * --------------------------------------------------------------------------------- */
#define DUSTIN_SCORE_SYNC_BYTES 16896u
#define DUSTIN_SCORE_SYNC_FLAG_OFFSET 16384u
size_t dustin_score_workspace(int32_t batch, int32_t max_len, int32_t nq_max, int32_t n_heads);
dustin_status dustin_score(const void* q, int64_t q_sb, int64_t q_sj, int64_t q_sh,
                           int32_t num_q_heads, const int32_t* heads_host, int32_t n_heads,
                           const dustin_kv* k, const dustin_batch* bt, float scale,
                           int32_t groups, const float* init, int64_t init_sb, int64_t init_sg,
                           float* out, int64_t out_sb, int64_t out_sg, void* workspace,
                           size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_score_layers -- Eq. 5 summed over n_layers scored layers in one call (the draft
 * side: S_D sums the scoring heads of the draft model's scoring layers, Eq. 5 upper):
 *   out = init + sum over layers l of the dustin_score sum of layer l
 * in at most two launches whatever n_layers is.  The layers share every shape and stride:
 *   q_layers_host  host array of n_layers device pointers, each laid out as q above
 *   k_layers_host  host array of n_layers dustin_kv that differ only in `data`
 *   1 <= n_layers <= 32; n_layers * n_heads * nq_max <= 1024; batch * n_layers <= 65535
 *   workspace  dustin_score_workspace(batch, max_len, nq_max, n_heads * n_layers) bytes
 * Every other argument is as for dustin_score.  The sum over layers is accumulated in
 * fp32 together with the heads' and queries' terms and rounded once at the end.  The
 * single-pass form applies as for dustin_score (the pair limit counts one layer's pairs),
 * in one launch whatever n_layers is.
 * --------------------------------------------------------------------------------- */
dustin_status dustin_score_layers(int32_t n_layers, const void* const* q_layers_host, int64_t q_sb,
                                  int64_t q_sj, int64_t q_sh, int32_t num_q_heads,
                                  const int32_t* heads_host, int32_t n_heads,
                                  const dustin_kv* k_layers_host, const dustin_batch* bt, float scale,
                                  int32_t groups, const float* init, int64_t init_sb, int64_t init_sg,
                                  float* out, int64_t out_sb, int64_t out_sg, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_score_calls -- one or two dustin_score_layers calls, such as the target's and the
 * draft's scores of one verification step (both halves of Eq. 5).  Two calls run in one
 * launch when both take the single-pass form with the pair of shapes compiled for it (the
 * first over four KV heads of 128-element rows, the second over two KV heads of 64-element
 * rows, both with the same tiles per wave): the second call's workgroups then start as the
 * first call's leave their compute units.  Otherwise the calls run one after the other.
 * Either way each output has the same bits as the corresponding dustin_score_layers call.
 *   calls    host array of n_calls (1 or 2) descriptors; each holds the arguments of one
 *            dustin_score_layers call (n_layers = 1 is a dustin_score call), with a
 *            workspace of its own (distinct workspaces; each as dustin_score requires)
 *   digit_hist  NULL, or device uint32 [batch * groups][4096], 16-byte aligned, zero before
 *            the call: for every written out[b, go, n] (n < N_b) the call adds one to
 *            digit_hist[(b * groups + go) * 4096 + key >> 20], key the order-preserving
 *            uint32 of the fp32 output (dustin_topk's ranking key).  It is the first-digit
 *            histogram that dustin_topk can take in place of its first pass over the row
 *            (hist_draft / hist_target), and dustin_topk returns it to zero.
 * Neither call may write a buffer that the other reads or writes.  Errors: as
 * dustin_score_layers for either call (nothing is enqueued), DUSTIN_ERR_INVALID_ARG for
 * n_calls outside [1, 2] or a misaligned or shared digit_hist, DUSTIN_ERR_WORKSPACE for a
 * shared workspace.
 * --------------------------------------------------------------------------------- */
typedef struct {
  int32_t n_layers;
  const void* const* q_layers_host;
  int64_t q_sb, q_sj, q_sh;
  int32_t num_q_heads;
  const int32_t* heads_host;
  int32_t n_heads;
  const dustin_kv* k_layers_host;
  const dustin_batch* bt;
  float scale;
  int32_t groups;
  const float* init;
  int64_t init_sb, init_sg;
  float* out;
  int64_t out_sb, out_sg;
  void* workspace;
  size_t workspace_bytes;
  uint32_t* digit_hist;
} dustin_score_call;
dustin_status dustin_score_calls(int32_t n_calls, const dustin_score_call* calls, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_score_per_layer -- Eq. 5 for n_layers layers in two launches, each layer into
 * its own output: the per-layer, per-head relevance of the SpecAttn-style selection the
 * paper compares with (appendix on SpecAttn: every draft layer and head scores tokens for
 * its own target layers, with no aggregation across layers).
 *   out[l, b, go, n] = sum_{h in heads of go} sum_{j < nq_b} softmax_{n' < N_b}(scale * q_l[b, j, h] . K_l[b, n', g(h)])[n]
 * for n < N_b, written at out + l * out_sl + b * out_sb + go * out_sg (fp32, elements).
 * There is no init.  1 <= n_layers <= 32; n_heads * nq_max <= 1024; batch * n_layers <=
 * 65535; groups * n_layers <= 65535; workspace as for dustin_score_layers.  Every other
 * argument is as for dustin_score_layers.  Each layer's output has the same bits as a
 * dustin_score call on that layer alone.
 * --------------------------------------------------------------------------------- */
dustin_status dustin_score_per_layer(int32_t n_layers, const void* const* q_layers_host, int64_t q_sb,
                                     int64_t q_sj, int64_t q_sh, int32_t num_q_heads,
                                     const int32_t* heads_host, int32_t n_heads,
                                     const dustin_kv* k_layers_host, const dustin_batch* bt, float scale,
                                     int32_t groups, float* out, int64_t out_sl, int64_t out_sb,
                                     int64_t out_sg, void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_page_meta -- page statistics of the page estimator.  The paper describes it
 * (related work; estimation overhead analysis; Appendix A's note on shrinking the
 * context dimension) as page-level minima and maxima of the keys that bound a page's
 * relevance in one computation.  For every sequence b, KV head g and page
 * p < ceil(N_b / page_size) that holds a position >= from_b:
 *   meta[b, p, g, 0:d]  = max over n in page p, n < N_b, of K[b, n, g, :]   (per channel)
 *   meta[b, p, g, d:2d] = min over the same positions
 * bf16 values of K, exact (of equal values the earliest position's, which decides only the
 * sign of a zero).  Pages are [p * page_size, (p + 1) * page_size); the last one holds
 * its positions below N_b only.  Other pages are not written.
 *   k          the layer's K cache (contiguous or paged); head_dim in {64, 128}
 *   bt         seq_lens (N_b), max_len; the other fields are not read
 *   from       device int32 [B]: first position whose page is rebuilt (clamped to
 *              [0, N_b]); NULL = 0 (build every page)
 *   max_span   host bound of N_b - from_b (of N_b when from is NULL), 0 <= max_span <=
 *              max_len; pages past from_b + max_span are not rebuilt.  After an append of
 *              T_b tokens, from = the old N_b and max_span = the largest T_b.
 *   page_size  a power of two, 1 ... 4096
 *   meta       bf16 [B, meta_pages, num_kv_heads, 2 * head_dim], strides meta_sb
 *              (sequences) and meta_sp (pages) in elements; meta_sp >= num_kv_heads * 2 *
 *              head_dim; meta_pages >= ceil(max_len / page_size)
 * Errors: DUSTIN_ERR_INVALID_ARG for a bad pointer, size, stride or page size;
 * DUSTIN_ERR_UNSUPPORTED for another head_dim or batch > 65535.
 * --------------------------------------------------------------------------------- */
dustin_status dustin_page_meta(const dustin_kv* k, const dustin_batch* bt, const int32_t* from, int32_t max_span,
                               int32_t page_size, void* meta, int64_t meta_sb, int64_t meta_sp,
                               int32_t meta_pages, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_page_score -- page-estimator importance: Eq. 5's sum of softmaxes, taken over
 * pages with each page's bound on q . k in place of q . k, and given to every position of
 * the page.  With P_b = ceil(N_b / page_size) and u = sum_c max(q_c max_{p,c}, q_c min_{p,c})
 * (the largest q . k over keys inside the page's channel ranges):
 *   out[b, go, n] = init[b, go, n] + sum_{h in heads of go} sum_{j < nq_b}
 *                   softmax_{p < P_b}(scale * u(q[b, j, h], page p of KV head g(h)))[n / page_size]
 * for n < N_b; positions n >= N_b are not written.  "heads of go" is every head when
 * groups == 1, else those whose KV head is go.  With page_size 1 this is dustin_score.
 * Quest's all-heads estimator passes every query head; combined with the scoring heads,
 * heads_host holds those only.
 *   q, heads_host, bt (seq_lens, n_query, nq_max <= 16, max_len), scale, groups, init,
 *   out           as for dustin_score; n_heads * nq_max <= 1024
 *   meta, meta_sb, meta_sp, meta_pages   as written by dustin_page_meta with this
 *                 page_size, num_kv_heads and head_dim (64 or 128)
 *   workspace     dustin_page_score_workspace(batch, max_len, page_size, nq_max, n_heads)
 *                 bytes, 256-byte aligned
 * Rounding: the bound's products are exact in fp32 (bf16 times bf16) and summed in fp32;
 * fp32 exp and sums, as dustin_score.
 * --------------------------------------------------------------------------------- */
size_t dustin_page_score_workspace(int32_t batch, int32_t max_len, int32_t page_size, int32_t nq_max,
                                   int32_t n_heads);
dustin_status dustin_page_score(const void* q, int64_t q_sb, int64_t q_sj, int64_t q_sh, int32_t num_q_heads,
                                const int32_t* heads_host, int32_t n_heads, const void* meta, int64_t meta_sb,
                                int64_t meta_sp, int32_t meta_pages, int32_t num_kv_heads, int32_t head_dim,
                                int32_t page_size, const dustin_batch* bt, float scale, int32_t groups,
                                const float* init, int64_t init_sb, int64_t init_sg, float* out, int64_t out_sb,
                                int64_t out_sg, void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_arr -- windowed attention recovery rate of index sets (the evaluation framework,
 * Eqs. 1-4), averaged over the heads a set serves:
 *   arr[b, go] = (1 / (w_b * heads_per_group)) * sum_{i < count[b, go]} s[b, go, idx[b, go, i]]
 * where s is dustin_score's output over every head the set serves (all query heads when
 * groups == 1, the heads of KV head go otherwise: heads_per_group of them) and the w_b =
 * n_query[b] queries of the verification window, with init = NULL.  Then
 * s / (w_b * heads_per_group) is the window- and head-averaged attention A-bar (Eq. 3) over
 * the committed positions, and, ARR being linear in the weights, arr is the windowed ARR
 * (Eq. 2) averaged over those heads.  The SD oracle (Eq. 4) is dustin_topk on s with
 * n_sink = n_window = 0 and m = 0, followed by this call on its set.
 *   s          fp32 [B, >= groups or 1, >= max_len], strides s_sb, s_sg (0 = one row per b)
 *   idx, count int32 as dustin_topk writes them: distinct positions; count clamped to
 *              [0, k_max]; positions outside [0, N_b) are skipped
 *   bt         seq_lens (N_b), n_query (w_b; NULL = nq_max), k_max
 *   arr        fp64 [B, groups] (device, row-major, 8-byte aligned)
 * The sum is taken in fp64 in a fixed order: repeated calls give identical bits.
 * --------------------------------------------------------------------------------- */
dustin_status dustin_arr(const float* s, int64_t s_sb, int64_t s_sg, const int32_t* idx, int64_t idx_sb,
                         int64_t idx_sg, const int32_t* count, const dustin_batch* bt, int32_t groups,
                         int32_t heads_per_group, double* arr, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_topk -- tiered hybrid selection, Eq. 6 (hybrid_selection), with the protected
 * set of the experimental setup (n_sink attention sinks and an n_window recent window,
 * counted inside the budget; Appendix C).  For every (b, go):
 *   N = N_b, k = k_b, m = m_b, P = [0, n_sink) U [N - n_window, N)
 *   N <= k : I = [0, N)
 *   else   : I_D = the m best of [0,N) \ P by S_D
 *            I_T = the k - m - |P| best of [0,N) \ (P U I_D) by S_T
 *            I   = P U I_D U I_T
 *   "best" orders by value descending, then position ascending; values compare as
 *   numbers with -0 == +0, and NaNs sort beyond +-inf by their sign bit.
 *   idx[b, go, 0 .. count) = I in ascending order, count[b * groups + go] = |I| = min(k, N).
 *   Entries idx[b, go, count ..) are not written.
 *   s_draft / s_target  fp32 [B, G', >= max_len] (strides *_sb, *_sg; *_sg = 0
 *       broadcasts one vector to every group); either may be NULL: no S_D requires
 *       m = 0 (target-only, Dustin-T), no S_T requires m = k - |P| (draft-only, Dustin-D)
 *   bt       seq_lens, budget/k_max, m/m_scalar; 1 <= max_len <= 1 << 19
 *   groups   1 or the KV head count
 *   idx      int32 [B, groups, >= k_max] (strides idx_sb, idx_sg), count int32 [B*groups]
 *   hist_draft / hist_target  NULL, or (groups = 1, with s_draft / s_target given) device
 *       uint32 [B][4096], 16-byte aligned: for each sequence, the count of positions
 *       n < N_b of its S_D / S_T row per top key digit (key >> 20), as dustin_score_calls
 *       writes with digit_hist.  A tier that is its workgroup's first job then takes it, less
 *       the protected positions, instead of a first pass over the row.  Every given histogram
 *       is left at zero.  The histograms must describe the rows passed here (same values,
 *       same N_b): the result is then the same as without them.
 *   workspace  dustin_topk_workspace(batch, groups, max_len) bytes, 256-byte aligned,
 *       required when both s_draft and s_target are given (else NULL, 0 will do): the two
 *       tiers of a row are selected side by side (I_D, and C_T = the k - |P| best free
 *       positions by S_T, of which I_T is the k - m - |P| best outside I_D) and hand off
 *       through it.  It holds a 16 KB counter region (one arrival counter per (b, go);
 *       B * groups <= 4096, beyond which no workspace is needed and the tiers of a row run
 *       one after the other), then two bitmaps of max_len bits per (b, go).  Zero-fill it
 *       once before its first use: every call leaves the counter region at zero again, so
 *       one buffer can then serve calls of any shape.  Calls sharing a workspace must not
 *       overlap.
 * The result is a pure function of the fp32 inputs: bit-exact and deterministic.
 * --------------------------------------------------------------------------------- */
size_t dustin_topk_workspace(int32_t batch, int32_t groups, int32_t max_len);
dustin_status dustin_topk(const float* s_draft, int64_t d_sb, int64_t d_sg,
                          const float* s_target, int64_t t_sb, int64_t t_sg,
                          const dustin_batch* bt, int32_t groups, int32_t n_sink,
                          int32_t n_window, int32_t* idx, int64_t idx_sb, int64_t idx_sg,
                          int32_t* count, uint32_t* hist_draft, uint32_t* hist_target,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_sparse_verify_attn -- verification attention over the selected tokens only
 * (the compressed target KV cache of method section 4.1, never materialised: rows are
 * gathered on the fly).  For b, t < T_b, h:
 *   J = I[b, gi] (gi = g(h) if groups > 1 else 0) followed by N_b .. N_b + t
 *   out[b, t, h] = sum_{n in J} softmax_J(scale * q[b,t,h] . K[b,n,g(h)]) V[b,n,g(h)]
 *   q    bf16 [B, nq_max, num_q_heads, 128] (strides q_sb, q_st, q_sh); head_dim 128;
 *        T_b * num_q_heads / num_kv_heads <= 128 rows per KV head
 *   k, v the layer's K and V caches (same layout kind); capacity >= max_len + nq_max
 *   idx  int32 [B, groups, >= k_max] (strides idx_sb, idx_sg) ascending positions < N_b,
 *        count int32 [B * groups] (as written by dustin_topk)
 *   out  bf16 [B, nq_max, num_q_heads, 128] (strides o_sb, o_st, o_sh); rows t >= T_b
 *        are not written.  Round to nearest even.
 *   workspace  dustin_attn_workspace(..., sparse = 1) bytes, 256-byte aligned (0 bytes,
 *        i.e. NULL, when the batch has enough (b, KV head) pairs to fill the GPU without
 *        splitting the token list).  Its first 256 KB are a counter region (one int32 per
 *        (b, KV head); B * num_kv_heads <= 65536), the partial results of token splits
 *        follow.  Zero-fill the workspace once before its first use: every call leaves the
 *        counter region at zero again, so one buffer can then serve calls of any shape.
 *        Calls sharing a workspace must not overlap.
 * Rounding: bf16 inputs, fp32 MFMA accumulation, fp32 online softmax, probabilities
 * rounded to bf16 before the value product, bf16 output.
 * --------------------------------------------------------------------------------- */
size_t dustin_attn_workspace(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                             int32_t nq_max, int32_t max_tokens, int32_t sparse);
dustin_status dustin_sparse_verify_attn(const void* q, int64_t q_sb, int64_t q_st,
                                        int64_t q_sh, int32_t num_q_heads, const dustin_kv* k,
                                        const dustin_kv* v, const dustin_batch* bt,
                                        const int32_t* idx, int64_t idx_sb, int64_t idx_sg,
                                        const int32_t* count, int32_t groups, float scale,
                                        void* out, int64_t o_sb, int64_t o_st, int64_t o_sh,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_sparse_verify_attn_noalloc -- dustin_sparse_verify_attn for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same arguments without the workspace, the same kernels and
 * the same split schedule, so the output is bit-identical to dustin_sparse_verify_attn's.
 * It calls no hipMalloc or hipFree.
 *
 * Scratch: the split partials and counters live in a fixed device array of the library,
 * DUSTIN_NOALLOC_SCRATCH_BYTES (48 MiB) per GPU, held until the process ends.  A call that
 * needs more than that (dustin_attn_workspace(..., sparse = 1) > the limit) returns
 * DUSTIN_ERR_SCRATCH_LIMIT with nothing enqueued; at the Qwen2.5-72B shape (B = 16, 8 KV
 * heads, 40 rows per KV head) a call needs 6.6 MB.  The first call on a device looks the
 * array up and enqueues one small fill kernel on `stream` that zeroes its counter region:
 * make that first call outside graph capture.  Every call on one GPU shares that GPU's array, which keeps
 * the last call's contents (the counters return to zero after each call): calls that
 * overlap on one GPU, on any streams, race and give wrong outputs.
 * Returns as dustin_sparse_verify_attn, plus DUSTIN_ERR_SCRATCH_LIMIT, or
 * DUSTIN_ERR_LAUNCH when the array cannot be found on the current device.
 * --------------------------------------------------------------------------------- */
#define DUSTIN_NOALLOC_SCRATCH_BYTES (48u << 20)
dustin_status dustin_sparse_verify_attn_noalloc(const void* q, int64_t q_sb, int64_t q_st,
                                                int64_t q_sh, int32_t num_q_heads,
                                                const dustin_kv* k, const dustin_kv* v,
                                                const dustin_batch* bt, const int32_t* idx,
                                                int64_t idx_sb, int64_t idx_sg,
                                                const int32_t* count, int32_t groups,
                                                float scale, void* out, int64_t o_sb,
                                                int64_t o_st, int64_t o_sh, void* stream);

/* ---------------------------------------------------------------------------------
 * dense_verify_attn -- full-cache verification attention (the baseline every speedup
 * in the paper is measured against): as above with J = [0, N_b) followed by
 * N_b .. N_b + t.  max_tokens for the workspace is max_len.
 * --------------------------------------------------------------------------------- */
dustin_status dense_verify_attn(const void* q, int64_t q_sb, int64_t q_st, int64_t q_sh,
                                int32_t num_q_heads, const dustin_kv* k, const dustin_kv* v,
                                const dustin_batch* bt, float scale, void* out, int64_t o_sb,
                                int64_t o_st, int64_t o_sh, void* workspace,
                                size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_kv_append -- the target K and V of the verification window into the caches,
 * before the verification attention reads them (Sec. 3.2, sparse verification workflow:
 * the window tokens are verified against the cache, and accepted ones are appended).
 * For every b < B, t < T_b, h < Hkv:
 *   K[b, N_b + t, h, :] = k_new[b, t, h, :],  V[b, N_b + t, h, :] = v_new[b, t, h, :]
 * through the page table when the caches are paged.  Positions without a page
 * (t beyond max_pages * page_size) or past a contiguous cache's capacity are not written.
 *   k_new, v_new  bf16 [B, nq_max, Hkv, d] (strides *_sb, *_st, *_sh in elements, inner
 *       stride 1, 16-byte aligned rows); read only for t < T_b
 *   k, v          the caches (as for the attention; d a multiple of 8; one page table);
 *                 must address max_len + nq_max positions per sequence
 *   bt            seq_lens (N_b), n_query (T_b, NULL = nq_max), max_len, nq_max
 * Device arrays are read on the stream; nothing is read back on the host.
 * --------------------------------------------------------------------------------- */
dustin_status dustin_kv_append(const void* k_new, int64_t k_sb, int64_t k_st, int64_t k_sh,
                               const void* v_new, int64_t v_sb, int64_t v_st, int64_t v_sh,
                               const dustin_kv* k, const dustin_kv* v, const dustin_batch* bt,
                               void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_kv_commit -- after verification, keep the accepted window tokens and discard the
 * rest (Sec. 3.2): seq_lens[b] += clamp(accepted[b], 0, T_b) for b < batch, with
 * T_b = n_query[b] clamped to [0, nq_max] (n_query NULL: T_b = nq_max).  The rejected
 * window rows stay in the cache beyond the new N_b, where no kernel reads them and the
 * next step's dustin_kv_append overwrites them.
 *   seq_lens  device int32 [batch], updated in place; accepted, n_query device int32 [batch]
 * --------------------------------------------------------------------------------- */
dustin_status dustin_kv_commit(int32_t* seq_lens, const int32_t* accepted, const int32_t* n_query,
                               int32_t batch, int32_t nq_max, void* stream);

/* ---------------------------------------------------------------------------------
 * dustin_read_probe -- a plain streaming read of a device buffer, for measurement only (no
 * part of the method): the practical read rate of the GPU, against which the rates of the
 * bandwidth-bound kernels above are reported.  Workgroup g of `blocks` reads the g-th of
 * `blocks` equal runs of the buffer with 16-byte loads and writes the wrapping sum of the
 * 32-bit words it read to block_sums[g] (so the sums over the workgroups add up to the
 * wrapping sum of every word of the buffer).
 *   data        device buffer, 16-byte aligned; bytes a multiple of 16
 *   block_sums  device uint32 [blocks]; 1 <= blocks <= 65536, bytes / blocks < 2 GiB
 * Returns DUSTIN_ERR_INVALID_ARG on a bad pointer, size or count, DUSTIN_ERR_UNSUPPORTED
 * when a workgroup's run would reach 2 GiB.
 * --------------------------------------------------------------------------------- */
dustin_status dustin_read_probe(const void* data, size_t bytes, uint32_t* block_sums, int32_t blocks,
                                void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DUSTIN_H */
