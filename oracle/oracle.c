/*
 * oracle.c -- plain, slow, CPU reference for the Dustin sparse-verification step
 * (Dustin: Draft-Augmented Sparse Verification for Efficient Long-Context Generation
 * with Speculative Decoding).
 *
 * TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the benchmark's
 * CPU-baseline leg are the only callers.  The HIP library never links, loads or calls
 * this file, and this file shares no source, header, table or helper with it.
 *
 * Conventions
 *   - bf16 tensors arrive as their raw 16-bit patterns (uint16_t); they are widened
 *     here (bits << 16 is the fp32 pattern) and all arithmetic is done in fp64.
 *   - Strides are in elements.  The innermost (head_dim / position) stride is 1.
 *   - Every function returns 0 on success and a negative number for an argument it
 *     refuses; it never aborts.
 *   - OpenMP (when compiled with -fopenmp) only splits independent output rows;
 *     the arithmetic inside a row is sequential, so results do not depend on the
 *     thread count.
 *
 * Readings of the paper that this file fixes (the paper is silent on them):
 *   - GQA map: query head h reads KV head h / (Hq / Hkv).
 *   - Score softmax domain: the committed positions [0, N_b) of sequence b.
 *   - Selection ties: order by value descending, then position ascending, on the
 *     canonical order key of the fp32 value (see oracle_order_key).
 *   - The T_b verification tokens sit at positions [N_b, N_b + T_b) of the cache; query
 *     t attends to the selected set plus positions N_b .. N_b + t (causal), and they are
 *     not counted in the budget k.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_version(void) { return 1; }

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* bf16 -> fp64: a bf16 value is the upper half of an fp32 bit pattern. */
double oracle_bf16_to_double(uint16_t h) {
  uint32_t u = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/*
 * Order key of an fp32 value for the TopK of Eq. 6 (hybrid_selection): a uint32 whose
 * unsigned order is the numeric order of the floats.  -0 is first mapped to +0 so the
 * two zeros tie; negative values map to the complement of their bits, non-negative
 * values get the sign bit set.  NaNs land beyond +-inf by their sign, so every input,
 * NaN included, has a fixed place in the order.
 */
uint32_t oracle_order_key(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

/* -------------------------------------------------------------------------------
 * Eq. 5 (hybrid_importance), restricted to the scoring heads as in the online sparse
 * estimation of the method section and Appendix A:
 *
 *   S[b, go, n] = init[b, go, n] + sum_{h in H(go)} sum_{j < nq_b} softmax_n(scale * q[b,j,h] . K[b,n,g(h)])
 *
 * for n in [0, N_b).  H(go) is every scoring head when groups == 1, else the scoring
 * heads whose KV head g(h) equals go (groups == num_kv_heads).  The sum is formed in
 * fp64 and rounded once to fp32.  Positions n >= N_b are not written.
 *   q    : bf16 [B, nq_max, num_q_heads, head_dim]        strides q_sb, q_sj, q_sh
 *   k    : bf16 [B, >= N_b, num_kv_heads, head_dim]       strides k_sb, k_sn, k_sh
 *   init : fp32 [B, groups, >= N_b] or NULL (= 0)          strides init_sb, init_sg
 *   out  : fp32 [B, groups, >= N_b] (may alias init)      strides out_sb, out_sg
 * ------------------------------------------------------------------------------- */
int oracle_score(const uint16_t* q, int64_t q_sb, int64_t q_sj, int64_t q_sh,
                 const uint16_t* k, int64_t k_sb, int64_t k_sn, int64_t k_sh,
                 int B, const int32_t* seq_lens, const int32_t* n_query,
                 int num_q_heads, int num_kv_heads, int head_dim,
                 const int32_t* heads, int n_heads, int groups, double scale,
                 const float* init, int64_t init_sb, int64_t init_sg,
                 float* out, int64_t out_sb, int64_t out_sg) {
  if (!q || !k || !seq_lens || !n_query || !out || (n_heads > 0 && !heads)) return -1;
  if (B < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 || n_heads < 0) return -1;
  if (num_q_heads % num_kv_heads) return -2;
  if (groups != 1 && groups != num_kv_heads) return -3;
  for (int i = 0; i < n_heads; ++i)
    if (heads[i] < 0 || heads[i] >= num_q_heads) return -4;
  const int group_size = num_q_heads / num_kv_heads;
  int rc = 0;

#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int go = 0; go < groups; ++go) {
      const int N = seq_lens[b];
      const int nq = n_query[b];
      if (N <= 0) continue;
      double* acc = (double*)calloc((size_t)N, sizeof(double));
      double* logit = (double*)malloc((size_t)N * sizeof(double));
      if (!acc || !logit) {
        free(acc);
        free(logit);
#pragma omp atomic write
        rc = -9;
        continue;
      }
      for (int hi = 0; hi < n_heads; ++hi) {
        const int h = heads[hi];
        const int g = h / group_size;
        if (groups != 1 && g != go) continue;
        for (int j = 0; j < nq; ++j) {
          const uint16_t* qv = q + b * q_sb + j * q_sj + h * q_sh;
          double mx = -INFINITY;
          for (int n = 0; n < N; ++n) {
            const uint16_t* kv = k + b * k_sb + (int64_t)n * k_sn + g * k_sh;
            double dot = 0.0;
            for (int c = 0; c < head_dim; ++c)
              dot += oracle_bf16_to_double(qv[c]) * oracle_bf16_to_double(kv[c]);
            logit[n] = scale * dot;
            if (logit[n] > mx) mx = logit[n];
          }
          double z = 0.0;
          for (int n = 0; n < N; ++n) z += exp(logit[n] - mx);
          for (int n = 0; n < N; ++n) acc[n] += exp(logit[n] - mx) / z;
        }
      }
      float* o = out + b * out_sb + go * out_sg;
      const float* in = init ? init + b * init_sb + go * init_sg : NULL;
      for (int n = 0; n < N; ++n) o[n] = (float)((in ? (double)in[n] : 0.0) + acc[n]);
      free(acc);
      free(logit);
    }
  }
  return rc;
}

/* -------------------------------------------------------------------------------
 * Eq. 6 (hybrid_selection) with the protected set of the experimental setup
 * (attention sinks plus a recent window, counted inside the budget k).
 * ------------------------------------------------------------------------------- */
typedef struct {
  uint32_t key;
  int32_t pos;
} oracle_keyed;

/* value descending (key descending), then position ascending */
static int oracle_keyed_cmp(const void* a, const void* b) {
  const oracle_keyed* x = (const oracle_keyed*)a;
  const oracle_keyed* y = (const oracle_keyed*)b;
  if (x->key != y->key) return x->key > y->key ? -1 : 1;
  return (x->pos > y->pos) - (x->pos < y->pos);
}

/* Writes the first `take` positions of cand[0..n) in the (value desc, position asc)
 * order of the scores s into chosen[] (chosen[pos] = 1).  Returns how many it took. */
static int oracle_take_top(const float* s, const int32_t* cand, int n, int take,
                           unsigned char* chosen, oracle_keyed* scratch) {
  if (take <= 0 || n <= 0) return 0;
  for (int i = 0; i < n; ++i) {
    scratch[i].key = oracle_order_key(s[cand[i]]);
    scratch[i].pos = cand[i];
  }
  qsort(scratch, (size_t)n, sizeof(oracle_keyed), oracle_keyed_cmp);
  if (take > n) take = n;
  for (int i = 0; i < take; ++i) chosen[scratch[i].pos] = 1;
  return take;
}

/*
 * For each sequence b and selection group go:
 *   N = seq_lens[b], k = budget[b] (or k_scalar), m = m[b] (or m_scalar)
 *   if N <= k: I = [0, N)
 *   else:
 *     I_prot   = [0, n_sink) U [N - n_window, N)
 *     I_draft  = top-m of S_D over [0,N) \ I_prot
 *     I_target = top-(k - m - |I_prot|) of S_T over [0,N) \ (I_prot U I_draft)
 *     I        = I_prot U I_draft U I_target, ascending
 *   idx[b, go, 0..count) = I, count[b*G + go] = |I|.
 * s_draft == NULL requires m == 0; s_target == NULL requires m == k - |I_prot|.
 * A stride of 0 over groups broadcasts one score vector to every group.
 */
int oracle_select(const float* s_draft, int64_t d_sb, int64_t d_sg,
                  const float* s_target, int64_t t_sb, int64_t t_sg,
                  int B, int G, const int32_t* seq_lens,
                  const int32_t* budget, int k_scalar, const int32_t* m_arr, int m_scalar,
                  int n_sink, int n_window,
                  int32_t* idx, int64_t idx_sb, int64_t idx_sg, int32_t* count) {
  if (!seq_lens || !idx || !count || B < 0 || G <= 0 || n_sink < 0 || n_window < 0) return -1;
  int rc = 0;

#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int go = 0; go < G; ++go) {
      const int N = seq_lens[b];
      const int kb = budget ? budget[b] : k_scalar;
      const int mb = m_arr ? m_arr[b] : m_scalar;
      int32_t* out = idx + b * idx_sb + go * idx_sg;
      if (N <= 0) {
        count[b * G + go] = 0;
        continue;
      }
      if (kb < n_sink + n_window || mb < 0 || mb > kb - n_sink - n_window ||
          (!s_draft && mb != 0) || (!s_target && mb != kb - n_sink - n_window)) {
#pragma omp atomic write
        rc = -2;
        count[b * G + go] = 0;
        continue;
      }
      if (N <= kb) {
        for (int n = 0; n < N; ++n) out[n] = n;
        count[b * G + go] = N;
        continue;
      }
      unsigned char* chosen = (unsigned char*)calloc((size_t)N, 1);
      int32_t* cand = (int32_t*)malloc((size_t)N * sizeof(int32_t));
      oracle_keyed* scratch = (oracle_keyed*)malloc((size_t)N * sizeof(oracle_keyed));
      if (!chosen || !cand || !scratch) {
        free(chosen);
        free(cand);
        free(scratch);
#pragma omp atomic write
        rc = -9;
        count[b * G + go] = 0;
        continue;
      }
      /* protected set: N > k >= n_sink + n_window, so the two parts are disjoint */
      for (int n = 0; n < n_sink; ++n) chosen[n] = 1;
      for (int n = N - n_window; n < N; ++n) chosen[n] = 1;
      const int n_prot = n_sink + n_window;

      /* draft tier over the unprotected positions */
      int nc = 0;
      for (int n = 0; n < N; ++n)
        if (!chosen[n]) cand[nc++] = n;
      if (s_draft) oracle_take_top(s_draft + b * d_sb + go * d_sg, cand, nc, mb, chosen, scratch);

      /* target tier over what is left */
      nc = 0;
      for (int n = 0; n < N; ++n)
        if (!chosen[n]) cand[nc++] = n;
      if (s_target)
        oracle_take_top(s_target + b * t_sb + go * t_sg, cand, nc, kb - mb - n_prot, chosen, scratch);

      int c = 0;
      for (int n = 0; n < N; ++n)
        if (chosen[n]) out[c++] = n;
      count[b * G + go] = c;
      free(chosen);
      free(cand);
      free(scratch);
    }
  }
  return rc;
}

/* -------------------------------------------------------------------------------
 * Verification attention (sparse: attention over the selected set, used for every
 * layer; dense: the full-cache attention the paper compares against).  For each
 * requested output row (b, t, h), with g = h / (Hq / Hkv):
 *
 *   J = I[b, gi] (sparse, gi = g when G == Hkv else 0) or [0, N_b) (dense),
 *       followed by the verification positions N_b + u for u = 0 .. t
 *   l_n = scale * q[b,t,h] . K[b,n,g]            (fp64)
 *   out = sum_{n in J} exp(l_n - max l) V[b,n,g] / sum_{n in J} exp(l_n - max l)
 *
 *   q : bf16 [B, T_max, Hq, d]      k, v : bf16 [B, >= N_b + T_b, Hkv, d]
 *   idx : int32 [B, G, k_max] (NULL = dense), count : int32 [B, G]
 *   out : fp64 [n_rows, d]
 * ------------------------------------------------------------------------------- */
int oracle_attention(const uint16_t* q, int64_t q_sb, int64_t q_st, int64_t q_sh,
                     const uint16_t* k, int64_t k_sb, int64_t k_sn, int64_t k_sh,
                     const uint16_t* v, int64_t v_sb, int64_t v_sn, int64_t v_sh,
                     int num_q_heads, int num_kv_heads, int head_dim,
                     const int32_t* seq_lens,
                     const int32_t* idx, int64_t idx_sb, int64_t idx_sg, const int32_t* count, int G,
                     double scale,
                     int n_rows, const int32_t* row_b, const int32_t* row_t, const int32_t* row_h,
                     double* out) {
  if (!q || !k || !v || !seq_lens || !out || (n_rows > 0 && (!row_b || !row_t || !row_h)))
    return -1;
  if (num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 || num_q_heads % num_kv_heads)
    return -2;
  if (idx && (!count || (G != 1 && G != num_kv_heads))) return -3;
  const int group_size = num_q_heads / num_kv_heads;
  int rc = 0;

#pragma omp parallel for schedule(dynamic)
  for (int r = 0; r < n_rows; ++r) {
    const int b = row_b[r], t = row_t[r], h = row_h[r];
    const int g = h / group_size;
    const int N = seq_lens[b];
    const int gi = (G == 1) ? 0 : g;
    const int n_sel = idx ? count[b * G + gi] : N;
    const int n_tot = n_sel + t + 1;
    int64_t* pos = (int64_t*)malloc((size_t)n_tot * sizeof(int64_t));
    double* logit = (double*)malloc((size_t)n_tot * sizeof(double));
    if (!pos || !logit) {
      free(pos);
      free(logit);
#pragma omp atomic write
      rc = -9;
      continue;
    }
    for (int i = 0; i < n_sel; ++i) pos[i] = idx ? idx[b * idx_sb + gi * idx_sg + i] : i;
    for (int u = 0; u <= t; ++u) pos[n_sel + u] = (int64_t)N + u;

    const uint16_t* qv = q + b * q_sb + t * q_st + h * q_sh;
    double mx = -INFINITY;
    for (int i = 0; i < n_tot; ++i) {
      const uint16_t* kv = k + b * k_sb + pos[i] * k_sn + g * k_sh;
      double dot = 0.0;
      for (int c = 0; c < head_dim; ++c)
        dot += oracle_bf16_to_double(qv[c]) * oracle_bf16_to_double(kv[c]);
      logit[i] = scale * dot;
      if (logit[i] > mx) mx = logit[i];
    }
    double z = 0.0;
    for (int i = 0; i < n_tot; ++i) z += exp(logit[i] - mx);
    double* o = out + (int64_t)r * head_dim;
    for (int c = 0; c < head_dim; ++c) o[c] = 0.0;
    for (int i = 0; i < n_tot; ++i) {
      const double p = exp(logit[i] - mx) / z;
      const uint16_t* vv = v + b * v_sb + pos[i] * v_sn + g * v_sh;
      for (int c = 0; c < head_dim; ++c) o[c] += p * oracle_bf16_to_double(vv[c]);
    }
    free(pos);
    free(logit);
  }
  return rc;
}

/* -------------------------------------------------------------------------------
 * Attention Recovery Rate (Eq. ARR def) and its window average (Eq. ARR window def):
 * ARR of a selected set K over one attention row A is sum_{j in K} A[j]; the windowed
 * form averages it over w consecutive rows.  A : fp64 [w, n_valid] row-major.
 * ------------------------------------------------------------------------------- */
double oracle_arr_window(const double* A, int w, int n_valid, const int32_t* sel, int n_sel) {
  if (!A || w <= 0 || n_valid <= 0 || (n_sel > 0 && !sel)) return NAN;
  double total = 0.0;
  for (int s = 0; s < w; ++s) {
    double arr = 0.0;
    for (int i = 0; i < n_sel; ++i) arr += A[(int64_t)s * n_valid + sel[i]];
    total += arr;
  }
  return total / (double)w;
}

/* -------------------------------------------------------------------------------
 * Appendix A cost model: the share of attention-score heads the sparse estimator
 * materialises relative to materialising every head of both models,
 *   (Hd* Ld* Gamma + Ht* Lt*) / (Hd Ld Gamma + Ht Lt).
 * ------------------------------------------------------------------------------- */
double oracle_overhead_ratio(int hd_sel, int ld_sel, int gamma, int ht_sel, int lt_sel,
                             int hd, int ld, int ht, int lt) {
  const double num = (double)hd_sel * ld_sel * gamma + (double)ht_sel * lt_sel;
  const double den = (double)hd * ld * gamma + (double)ht * lt;
  return den > 0 ? num / den : NAN;
}

/* -------------------------------------------------------------------------------
 * Page estimator: the query-aware page scoring of Quest, which the paper names as the
 * estimator that shrinks the context dimension (related work; the estimation-overhead
 * analysis, where Quest-16 is Quest with 16-position pages; Appendix A's note that it
 * could be combined with the scoring heads).  The paper describes it only as page-level
 * key minima and maxima that bound a page's relevance in one computation; the steps
 * below are that description written out, with these readings:
 *   - pages are the aligned spans [p * page_size, (p + 1) * page_size) of the committed
 *     positions [0, N_b); the last page holds only its positions below N_b;
 *   - a page's relevance to a query is the largest value q . k can take over keys whose
 *     every channel lies between the page's minimum and maximum of that channel:
 *       u = sum_c max(q_c * max_c, q_c * min_c);
 *   - several heads and queries are combined as Eq. 5 combines them: a softmax over the
 *     pages per (head, query), summed; every position of a page carries its page's sum.
 * ------------------------------------------------------------------------------- */

/* meta[b, p, g, 0:d] = channel-wise maximum and meta[b, p, g, d:2d] = minimum of
 * K[b, n, g, :] over the positions n of page p (bf16 patterns of the chosen keys; of
 * equal values, the earliest position's pattern, which decides only the sign of a zero).
 * Pages p < ceil(N_b / page_size) are written, others are not.
 *   k    : bf16 [B, >= N_b, num_kv_heads, head_dim]     strides k_sb, k_sn, k_sh
 *   meta : bf16 [B, >= pages, num_kv_heads, 2 * head_dim] strides m_sb, m_sp, m_sh */
int oracle_page_meta(const uint16_t* k, int64_t k_sb, int64_t k_sn, int64_t k_sh, int B,
                     const int32_t* seq_lens, int num_kv_heads, int head_dim, int page_size,
                     uint16_t* meta, int64_t m_sb, int64_t m_sp, int64_t m_sh) {
  if (!k || !seq_lens || !meta || B < 0 || num_kv_heads <= 0 || head_dim <= 0 || page_size <= 0)
    return -1;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int g = 0; g < num_kv_heads; ++g) {
      const int N = seq_lens[b];
      const int pages = N > 0 ? (N + page_size - 1) / page_size : 0;
      for (int p = 0; p < pages; ++p) {
        const int n0 = p * page_size;
        const int n1 = n0 + page_size < N ? n0 + page_size : N;
        uint16_t* row = meta + b * m_sb + (int64_t)p * m_sp + g * m_sh;
        for (int c = 0; c < head_dim; ++c) {
          uint16_t hi = k[b * k_sb + (int64_t)n0 * k_sn + g * k_sh + c], lo = hi;
          for (int n = n0 + 1; n < n1; ++n) {
            const uint16_t x = k[b * k_sb + (int64_t)n * k_sn + g * k_sh + c];
            if (oracle_bf16_to_double(x) > oracle_bf16_to_double(hi)) hi = x;
            if (oracle_bf16_to_double(x) < oracle_bf16_to_double(lo)) lo = x;
          }
          row[c] = hi;
          row[head_dim + c] = lo;
        }
      }
    }
  }
  return 0;
}

/* out[b, go, n] = init[b, go, n] + sum_{h in H(go)} sum_{j < nq_b}
 *                 softmax_{p < P_b}(scale * sum_c max(q_c * max_{p,c}, q_c * min_{p,c}))[n / page_size]
 * for n < N_b, P_b = ceil(N_b / page_size), with H(go) as in oracle_score.  One fp32
 * rounding at the end; positions n >= N_b are not written.
 *   q    : bf16 [B, nq_max, num_q_heads, head_dim]   strides q_sb, q_sj, q_sh
 *   meta : as written by oracle_page_meta            strides m_sb, m_sp, m_sh */
int oracle_page_score(const uint16_t* q, int64_t q_sb, int64_t q_sj, int64_t q_sh,
                      const uint16_t* meta, int64_t m_sb, int64_t m_sp, int64_t m_sh, int B,
                      const int32_t* seq_lens, const int32_t* n_query, int num_q_heads,
                      int num_kv_heads, int head_dim, int page_size, const int32_t* heads,
                      int n_heads, int groups, double scale, const float* init, int64_t init_sb,
                      int64_t init_sg, float* out, int64_t out_sb, int64_t out_sg) {
  if (!q || !meta || !seq_lens || !n_query || !out || (n_heads > 0 && !heads)) return -1;
  if (B < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 || page_size <= 0) return -1;
  if (num_q_heads % num_kv_heads) return -2;
  if (groups != 1 && groups != num_kv_heads) return -3;
  for (int i = 0; i < n_heads; ++i)
    if (heads[i] < 0 || heads[i] >= num_q_heads) return -4;
  const int group_size = num_q_heads / num_kv_heads;
  int rc = 0;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int go = 0; go < groups; ++go) {
      const int N = seq_lens[b];
      const int nq = n_query[b];
      if (N <= 0) continue;
      const int P = (N + page_size - 1) / page_size;
      double* acc = (double*)calloc((size_t)P, sizeof(double));
      double* u = (double*)malloc((size_t)P * sizeof(double));
      if (!acc || !u) {
        free(acc);
        free(u);
#pragma omp atomic write
        rc = -9;
        continue;
      }
      for (int hi = 0; hi < n_heads; ++hi) {
        const int h = heads[hi];
        const int g = h / group_size;
        if (groups != 1 && g != go) continue;
        for (int j = 0; j < nq; ++j) {
          const uint16_t* qv = q + b * q_sb + j * q_sj + h * q_sh;
          double mx = -INFINITY;
          for (int p = 0; p < P; ++p) {
            const uint16_t* row = meta + b * m_sb + (int64_t)p * m_sp + g * m_sh;
            double bound = 0.0;
            for (int c = 0; c < head_dim; ++c) {
              const double qc = oracle_bf16_to_double(qv[c]);
              const double a = qc * oracle_bf16_to_double(row[c]);
              const double z = qc * oracle_bf16_to_double(row[head_dim + c]);
              bound += a > z ? a : z;
            }
            u[p] = scale * bound;
            if (u[p] > mx) mx = u[p];
          }
          double zsum = 0.0;
          for (int p = 0; p < P; ++p) zsum += exp(u[p] - mx);
          for (int p = 0; p < P; ++p) acc[p] += exp(u[p] - mx) / zsum;
        }
      }
      float* o = out + b * out_sb + go * out_sg;
      const float* in = init ? init + b * init_sb + go * init_sg : NULL;
      for (int n = 0; n < N; ++n) o[n] = (float)((in ? (double)in[n] : 0.0) + acc[n / page_size]);
      free(acc);
      free(u);
    }
  }
  return rc;
}

/* -------------------------------------------------------------------------------
 * Attention recovery rate of the verification window (Eqs. 1-4, the evaluation
 * framework), with these readings: the valid positions of a verification query are the
 * committed positions [0, N_b) (the window's own tokens are attended whatever the policy);
 * the window is the w_b = n_query[b] verification queries; a shared index set is judged
 * by the mean over the heads it serves (every head when groups == 1, else the heads of KV
 * head go).  Per (b, go):
 *   A_{t,h}[n] = softmax_{n < N_b}(scale * q[b, t, h] . K[b, n, g(h)])        (Eq. 1's A)
 *   ARR_t      = sum_{n in I} A_{t,h}[n]                                        (Eq. 1)
 *   arr[b, go] = mean over h of (1 / w_b) sum_{t < w_b} ARR_t                   (Eq. 2)
 *   abar[b, go, n] = mean over h of (1 / w_b) sum_t A_{t,h}[n]                  (Eq. 3's A-bar)
 * so that the SD oracle's set is TopK_k(abar) and its windowed ARR is the sum of abar over
 * that set (Eq. 4).  I is idx[b, go, 0 .. count[b, go]); duplicate positions count once.
 *   arr  : fp64 [B, groups]                      (row-major)
 *   abar : fp64 [B, groups, >= N_b] or NULL       strides abar_sb, abar_sg
 * ------------------------------------------------------------------------------- */
int oracle_arr(const uint16_t* q, int64_t q_sb, int64_t q_sj, int64_t q_sh,
               const uint16_t* k, int64_t k_sb, int64_t k_sn, int64_t k_sh,
               int B, const int32_t* seq_lens, const int32_t* n_query,
               int num_q_heads, int num_kv_heads, int head_dim, int groups, double scale,
               const int32_t* idx, int64_t idx_sb, int64_t idx_sg, const int32_t* count,
               double* arr, double* abar, int64_t abar_sb, int64_t abar_sg) {
  if (!q || !k || !seq_lens || !n_query || !arr || (idx == NULL) != (count == NULL)) return -1;
  if (B < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0) return -1;
  if (num_q_heads % num_kv_heads) return -2;
  if (groups != 1 && groups != num_kv_heads) return -3;
  const int group_size = num_q_heads / num_kv_heads;
  int rc = 0;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int go = 0; go < groups; ++go) {
      const int N = seq_lens[b];
      const int w = n_query[b];
      arr[b * groups + go] = 0.0;
      if (N <= 0 || w <= 0) continue;
      double* a = (double*)malloc((size_t)N * sizeof(double));
      double* acc = (double*)calloc((size_t)N, sizeof(double));
      unsigned char* in_set = (unsigned char*)calloc((size_t)N, 1);
      if (!a || !acc || !in_set) {
        free(a);
        free(acc);
        free(in_set);
#pragma omp atomic write
        rc = -9;
        continue;
      }
      if (idx) {
        const int c = count[b * groups + go];
        for (int i = 0; i < c; ++i) {
          const int n = idx[b * idx_sb + go * idx_sg + i];
          if (n >= 0 && n < N) in_set[n] = 1;
        }
      }
      int nh = 0;
      double arr_sum = 0.0;
      for (int h = 0; h < num_q_heads; ++h) {
        const int g = h / group_size;
        if (groups != 1 && g != go) continue;
        ++nh;
        for (int t = 0; t < w; ++t) {
          const uint16_t* qv = q + b * q_sb + t * q_sj + h * q_sh;
          double mx = -INFINITY;
          for (int n = 0; n < N; ++n) {
            const uint16_t* kv = k + b * k_sb + (int64_t)n * k_sn + g * k_sh;
            double dot = 0.0;
            for (int c = 0; c < head_dim; ++c)
              dot += oracle_bf16_to_double(qv[c]) * oracle_bf16_to_double(kv[c]);
            a[n] = scale * dot;
            if (a[n] > mx) mx = a[n];
          }
          double z = 0.0;
          for (int n = 0; n < N; ++n) z += exp(a[n] - mx);
          double arr_t = 0.0;
          for (int n = 0; n < N; ++n) {
            a[n] = exp(a[n] - mx) / z;
            acc[n] += a[n];
            if (in_set[n]) arr_t += a[n];
          }
          arr_sum += arr_t;
        }
      }
      arr[b * groups + go] = nh ? arr_sum / ((double)w * nh) : 0.0;
      if (abar) {
        double* o = abar + b * abar_sb + go * abar_sg;
        for (int n = 0; n < N; ++n) o[n] = nh ? acc[n] / ((double)w * nh) : 0.0;
      }
      free(a);
      free(acc);
      free(in_set);
    }
  }
  return rc;
}
