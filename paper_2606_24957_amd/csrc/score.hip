// score.hip -- scoring-head importance (Eq. 5 restricted to the semantic retrieval heads),
// and the same sum over the pages of a page-statistics array (the page estimator).
//
// Several layers (the draft model's scoring layers) are scored in the same two launches:
// their logits rows sit side by side and pass 2 sums every layer's pairs into one output.
// Pass 1 (score_logits_kernel): one workgroup per (chunk of rows, column tile, sequence and
//   layer).  A column tile is up to 16 (scoring head, query) pairs of one KV head; each K
//   row of that KV head is read once per tile, with the same 16-byte-per-lane MFMA
//   A-operand loads as the attention kernel, and multiplied by every pair of the tile at
//   once.  The scaled logits (log2 domain) go to the workspace together with the chunk's
//   running (max, sum of exp2) per pair.
//   Page mode: a row is one page's [channel max | channel min] (length 2d) and the query
//   operand is [q+ | q-] (q+ = max(q, 0), q- = min(q, 0)), so that the MFMA dot product is
//   sum_c max(q_c max_c, q_c min_c), the largest q . k over keys inside the page's box.
// Pass 2 (score_finish_kernel): per (chunk, output group, sequence): merge the chunk
//   statistics of every pair into its softmax normaliser, then
//   out[n] = init[n] + sum_pairs exp2(logit - M) / Z, pairs in (layer, head, query) order.
//   With per-layer outputs each layer's pairs go to that layer's own output row instead.
//   Page mode (score_finish_pages_kernel): the same sum per page, written to every
//   position of the page.
#include "kernels.hpp"

namespace dustin {

// rows of sequence b scored: positions, or pages covering them
__device__ __forceinline__ int score_rows(const ScoreArgs& a, int b) {
  return (a.dims.len(b) + (1 << a.page_shift) - 1) >> a.page_shift;
}

// the non-negative (neg = false) or non-positive (neg = true) part of 8 bf16 values
__device__ __forceinline__ u32x4 sign_part(u32x4 x, bool neg) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t m = ((x[i] >> 15) & 0x00010001u) * 0xFFFFu;  // 0xFFFF where the sign is set
    r[i] = x[i] & (neg ? m : ~m);
  }
  return r;
}

template <int D, bool kPaged, bool kSign, int NT>
__global__ __launch_bounds__(kScoreWaves * kWave) void score_logits_kernel(ScoreArgs a) {
  constexpr int KS = D / 32;
  // 16-row tiles per iteration (loads issued together); fewer when the query operands of
  // several column tiles take the registers
  constexpr int U = NT == 1 ? 4 : 2;
  // KV heads vary fastest: workgroups that run together read the same positions of every
  // used KV head (neighbouring pieces of the same cache rows)
  const int grp = blockIdx.x, chunk = blockIdx.y;
  const int layer = blockIdx.z / a.batch, b = blockIdx.z - layer * a.batch;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int lr = lane & 15, lg = lane >> 4;
  const int u0 = a.tile_first[grp];
  const int nt = NT == 1 ? 1 : a.tile_count[grp];  // column tiles of this group, one KV head
  const int g = a.used_kv[u0];
  const int N = score_rows(a, b);
  const int nq = a.dims.nq(b);
  const int p_begin = chunk * a.chunk;
  const int p_end = min(N, p_begin + a.chunk);
  const int64_t rb = (int64_t)layer * a.batch + b;  // (layer, sequence) row block

  // column lr of tile t: (scoring head slot, query)
  bf16x8 qb[NT][KS];
  int pair_slot[NT], pair_q[NT];
  bool pair_ok[NT];
  float* lrow[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int u = u0 + (t < nt ? t : 0);
    const int npairs = t < nt ? a.pairs_per_kv[u] : 0;
    pair_slot[t] = lr < npairs ? a.pair_head[u * 16 + lr] : 0;
    pair_q[t] = lr < npairs ? a.pair_query[u * 16 + lr] : 0;
    pair_ok[t] = lr < npairs && pair_q[t] < nq;
    lrow[t] = a.logits + ((rb * a.n_heads + pair_slot[t]) * a.nq_max + pair_q[t]) * a.ld;
    if (pair_ok[t]) {
      const uint16_t* qp = a.q_layers[layer] + (int64_t)b * a.q_sb + (int64_t)pair_q[t] * a.q_sj +
                           (int64_t)a.heads[pair_slot[t]] * a.q_sh + 8 * lg;
      if constexpr (kSign) {  // [q+ | q-] from a query of length D / 2
#pragma unroll
        for (int ks = 0; ks < KS / 2; ++ks) {
          const u32x4 x = load16(qp + 32 * ks);
          qb[t][ks] = as_bf16x8(sign_part(x, false));
          qb[t][ks + KS / 2] = as_bf16x8(sign_part(x, true));
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qb[t][ks] = as_bf16x8(load16(qp + 32 * ks));
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qb[t][ks] = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
    }
  }
  KvView kv = a.k;
  kv.data = a.k_layers[layer];

  float m_run[NT], s_run[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    m_run[t] = -INFINITY;
    s_run[t] = 0.f;
  }
  for (int p0 = p_begin + wave * 16 * U; p0 < p_end; p0 += kScoreWaves * 16 * U) {
    u32x4 kr[U][KS];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int p = min(p0 + 16 * u + lr, max(N - 1, 0));
      const uint16_t* kp = kv.row<kPaged>(b, p, g) + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kr[u][ks] = load16(kp + 32 * ks);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int pb = p0 + 16 * u + 4 * lg;  // this lane's 4 rows, column lr
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t >= nt) break;  // uniform over the workgroup
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) c = mfma16x16x32(as_bf16x8(kr[u][ks]), qb[t][ks], c);
        float x[4];
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[e] = (pb + e < p_end) ? c[e] * a.scale_log2 : -INFINITY;
          mx = fmaxf(mx, x[e]);
        }
        const float m_new = fmaxf(m_run[t], mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        float add = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) add += fast_exp2(x[e] - m_use);
        s_run[t] = s_run[t] * fast_exp2(m_run[t] - m_use) + add;
        m_run[t] = m_new;
        if (pair_ok[t]) {
          if (pb + 3 < p_end) {
            *reinterpret_cast<f32x4*>(lrow[t] + pb) = f32x4{x[0], x[1], x[2], x[3]};
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (pb + e < p_end) lrow[t][pb + e] = x[e];
          }
        }
      }
    }
  }

  // reduce (max, sum) over lane groups, then over waves (fixed order)
  __shared__ float sm[NT][kScoreWaves][16][2];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float mo = __shfl_xor(m_run[t], off), so = __shfl_xor(s_run[t], off);
      const float mn = fmaxf(m_run[t], mo);
      const float mu = mn == -INFINITY ? 0.f : mn;
      s_run[t] = s_run[t] * fast_exp2(m_run[t] - mu) + so * fast_exp2(mo - mu);
      m_run[t] = mn;
    }
    if (lg == 0) {
      sm[t][wave][lr][0] = m_run[t];
      sm[t][wave][lr][1] = s_run[t];
    }
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (threadIdx.x < 16 && t < nt && pair_ok[t]) {
      float M = -INFINITY;
      for (int w = 0; w < kScoreWaves; ++w) M = fmaxf(M, sm[t][w][lr][0]);
      const float mu = M == -INFINITY ? 0.f : M;
      float S = 0.f;
      for (int w = 0; w < kScoreWaves; ++w) S += sm[t][w][lr][1] * fast_exp2(sm[t][w][lr][0] - mu);
      float* st = a.stats + (((rb * a.n_heads + pair_slot[t]) * a.nq_max + pair_q[t]) * a.n_chunks + chunk) * 2;
      st[0] = M;
      st[1] = S;
    }
  }
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

constexpr int kFinishThreads = 256;
constexpr int kFinishBatch = 8;  // logits rows loaded together per thread

// The (layer, head slot, query) rows that output group go of sequence b sums, in that
// order (every layer, or layer lo alone when each layer has its own output), with each
// row's softmax max M (log2 domain) and 1 / Z merged from the pass-1 chunk statistics.
// Returns the number of rows.
// Rows up to which a wave merges each row's chunk statistics (one round trip); past it one
// thread per row does (the same count for every caller, so a row's merge never depends on
// the workgroup size of the kernel that calls this).
constexpr int kFinishFewRows = 16;

template <int kThreads>
__device__ int finish_setup(const ScoreArgs& a, int b, int go, int lo, int nq, int n_rows, int* sm_row,
                            float* sm_M, float* sm_iz, int* sm_slots, int* sm_ns) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  if (tid == 0) {
    int ns = 0;
    for (int slot = 0; slot < a.n_heads; ++slot)
      if (a.groups == 1 || a.heads[slot] / a.group_size == go) sm_slots[ns++] = slot;
    *sm_ns = ns;
  }
  __syncthreads();
  const int ns = *sm_ns, per_layer = ns * nq;
  const int l0 = a.per_layer ? lo : 0, np = (a.per_layer ? 1 : a.n_layers) * per_layer;
  for (int i = tid; i < np; i += kThreads) {
    const int l = l0 + i / per_layer, r = i % per_layer, s = r / nq, j = r - s * nq;
    sm_row[i] = ((l * a.batch + b) * a.n_heads + sm_slots[s]) * a.nq_max + j;
  }
  __syncthreads();
  const int nch = (n_rows + a.chunk - 1) / a.chunk;
  if (np <= kFinishFewRows) {
    // few rows: the waves take the rows in turn, one chunk per lane (one round trip)
    for (int i = wave; i < np; i += kThreads / kWave) {
      const float* st = a.stats + (int64_t)sm_row[i] * a.n_chunks * 2;
      float M = -INFINITY;
      for (int c = lane; c < nch; c += kWave) M = fmaxf(M, st[2 * c]);
      M = wave_max(M);
      const float mu = M == -INFINITY ? 0.f : M;
      float Z = 0.f;
      for (int c = lane; c < nch; c += kWave) Z += st[2 * c + 1] * fast_exp2(st[2 * c] - mu);
      Z = wave_sum(Z);
      if (lane == 0) {
        sm_M[i] = mu;
        sm_iz[i] = Z > 0.f ? 1.f / Z : 0.f;
      }
    }
  } else {
    // many rows: one row per thread, its chunks' (max, sum) loaded kFinishBatch at a time
    // and merged in chunk order
    for (int i = tid; i < np; i += kThreads) {
      const float2* st = reinterpret_cast<const float2*>(a.stats + (int64_t)sm_row[i] * a.n_chunks * 2);
      float M = -INFINITY, Z = 0.f;
      for (int c0 = 0; c0 < nch; c0 += kFinishBatch) {
        float2 v[kFinishBatch];
#pragma unroll
        for (int u = 0; u < kFinishBatch; ++u) v[u] = c0 + u < nch ? st[c0 + u] : make_float2(-INFINITY, 0.f);
#pragma unroll
        for (int u = 0; u < kFinishBatch; ++u) {
          const float mn = fmaxf(M, v[u].x);
          const float mu = mn == -INFINITY ? 0.f : mn;
          Z = Z * fast_exp2(M - mu) + v[u].y * fast_exp2(v[u].x - mu);
          M = mn;
        }
      }
      sm_M[i] = M == -INFINITY ? 0.f : M;
      sm_iz[i] = Z > 0.f ? 1.f / Z : 0.f;
    }
  }
  __syncthreads();
  return np;
}

__global__ __launch_bounds__(kFinishThreads) void score_finish_kernel(ScoreArgs a) {
  const int chunk = blockIdx.x, go = blockIdx.y % a.groups, lo = blockIdx.y / a.groups, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int N = a.dims.len(b);
  const int nq = a.dims.nq(b);
  const int p_begin = chunk * kScoreFinishChunk;
  if (p_begin >= N) return;

  __shared__ int sm_row[kScoreMaxPairs];
  __shared__ float sm_M[kScoreMaxPairs], sm_iz[kScoreMaxPairs];
  __shared__ int sm_slots[kScoreMaxHeads];
  __shared__ int sm_ns;
  const int np = finish_setup<kFinishThreads>(a, b, go, lo, nq, N, sm_row, sm_M, sm_iz, sm_slots, &sm_ns);

  // four consecutive positions per thread (the logits rows are 64-element aligned, so
  // the vector load stays inside a row even past N)
  const int n0 = p_begin + 4 * tid;
  if (!a.hist && n0 >= N) return;  // (with a histogram every thread reaches its barriers)
  const bool live = n0 < N;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int i0 = 0; live && i0 < np; i0 += kFinishBatch) {
    f32x4 x[kFinishBatch];
#pragma unroll
    for (int u = 0; u < kFinishBatch; ++u) {
      const int i = i0 + u < np ? i0 + u : i0;
      x[u] = *reinterpret_cast<const f32x4*>(a.logits + (int64_t)sm_row[i] * a.ld + n0);
    }
#pragma unroll
    for (int u = 0; u < kFinishBatch; ++u) {
      if (i0 + u < np) {
        const float M = sm_M[i0 + u], iz = sm_iz[i0 + u];
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] += fast_exp2(x[u][e] - M) * iz;
      }
    }
  }
  const float* init_row = a.init ? a.init + (int64_t)b * a.init_sb + (int64_t)go * a.init_sg : nullptr;
  float* out_row = a.out + (int64_t)b * a.out_sb + (int64_t)go * a.out_sg + (int64_t)lo * a.out_sl;
  f32x4 val = {0.f, 0.f, 0.f, 0.f};
  if (live) {
    if (n0 + 3 < N && aligned16(out_row + n0) && (!init_row || aligned16(init_row + n0))) {
      const f32x4 in = init_row ? *reinterpret_cast<const f32x4*>(init_row + n0) : f32x4{0.f, 0.f, 0.f, 0.f};
      val = in + acc;
      *reinterpret_cast<f32x4*>(out_row + n0) = val;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        val[e] = (init_row && n0 + e < N ? init_row[n0 + e] : 0.f) + acc[e];
        if (n0 + e < N) out_row[n0 + e] = val[e];
      }
    }
  }
  // the chunk's outputs counted by top key digit, then the non-zero bins added into the
  // output row's histogram (summed outputs only: the host passes none with per-layer ones)
  if (a.hist) {
    __shared__ uint32_t h[kDigitBins];
    for (int i = tid; i < kDigitBins; i += kFinishThreads) h[i] = 0u;
    __syncthreads();
    if (live) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n0 + e < N) atomicAdd(&h[order_key(val[e]) >> 20], 1u);
    }
    __syncthreads();
    uint32_t* const gh = a.hist + ((int64_t)b * a.groups + go) * kDigitBins;
    for (int i = tid; i < kDigitBins; i += kFinishThreads) {
      const uint32_t v = h[i];
      if (v) __hip_atomic_fetch_add(gh + i, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Page mode: kScoreFinishPages pages per workgroup; wave w sums the rows i = w mod 4 of
// lane's page, the four partial sums are added in wave order, and every position of the
// page below N_b receives init + the page's sum.
// 16 waves per workgroup: each wave's share of a page's rows (320 with every head of a
// Qwen2.5-72B-shaped layer) is loaded in two batches instead of five, and a CU keeps about
// twice as many loads in flight.
constexpr int kFinishPagesThreads = 1024;

__global__ __launch_bounds__(kFinishPagesThreads) void score_finish_pages_kernel(ScoreArgs a) {
  const int chunk = blockIdx.x, go = blockIdx.y % a.groups, lo = blockIdx.y / a.groups, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int N = a.dims.len(b);
  const int P = score_rows(a, b);
  const int nq = a.dims.nq(b);
  const int p0 = chunk * kScoreFinishPages;
  if (p0 >= P) return;

  __shared__ int sm_row[kScoreMaxPairs];
  __shared__ float sm_M[kScoreMaxPairs], sm_iz[kScoreMaxPairs];
  __shared__ int sm_slots[kScoreMaxHeads];
  __shared__ int sm_ns;
  __shared__ float sm_acc[kFinishPagesThreads / kWave][kScoreFinishPages];
  const int np = finish_setup<kFinishPagesThreads>(a, b, go, lo, nq, P, sm_row, sm_M, sm_iz, sm_slots, &sm_ns);

  static_assert(kScoreFinishPages == kWave, "one page per lane");
  const int p = p0 + lane;
  const bool live = p < P;
  float acc = 0.f;
  constexpr int kWaves = kFinishPagesThreads / kWave;
  constexpr int kBatch = 2 * kFinishBatch;  // rows loaded together per lane
  for (int i0 = wave; i0 < np; i0 += kWaves * kBatch) {
    float x[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = i0 + u * kWaves < np ? i0 + u * kWaves : i0;
      x[u] = live ? a.logits[(int64_t)sm_row[i] * a.ld + p] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = i0 + u * kWaves;
      if (i < np) acc += fast_exp2(x[u] - sm_M[i]) * sm_iz[i];
    }
  }
  sm_acc[wave][lane] = acc;
  __syncthreads();

  const float* init_row = a.init ? a.init + (int64_t)b * a.init_sb + (int64_t)go * a.init_sg : nullptr;
  float* out_row = a.out + (int64_t)b * a.out_sb + (int64_t)go * a.out_sg + (int64_t)lo * a.out_sl;
  const int n_end = min(N, (p0 + kScoreFinishPages) << a.page_shift);
  for (int n = (p0 << a.page_shift) + tid; n < n_end; n += kFinishPagesThreads) {
    const int pp = (n >> a.page_shift) - p0;
    float v = sm_acc[0][pp];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) v += sm_acc[w][pp];
    out_row[n] = (init_row ? init_row[n] : 0.f) + v;
  }
}

template <int NT>
hipError_t launch_logits(const ScoreArgs& a, dim3 grid, int row_dim, bool paged, bool pages, hipStream_t stream) {
  const dim3 block(kScoreWaves * kWave);
  if (pages) {
    if (paged) return hipErrorInvalidValue;  // page statistics are a contiguous array
    if (row_dim == 256) hipLaunchKernelGGL((score_logits_kernel<256, false, true, NT>), grid, block, 0, stream, a);
    else if (row_dim == 128) hipLaunchKernelGGL((score_logits_kernel<128, false, true, NT>), grid, block, 0, stream, a);
    else return hipErrorInvalidValue;
  } else if (row_dim == 128) {
    if (paged) hipLaunchKernelGGL((score_logits_kernel<128, true, false, NT>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((score_logits_kernel<128, false, false, NT>), grid, block, 0, stream, a);
  } else if (row_dim == 64) {
    if (paged) hipLaunchKernelGGL((score_logits_kernel<64, true, false, NT>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((score_logits_kernel<64, false, false, NT>), grid, block, 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_score(const ScoreArgs& a, int B, int n_groups, int max_group, int row_dim, hipStream_t stream) {
  const dim3 grid1(n_groups, a.n_chunks, B * a.n_layers);
  const bool paged = a.k.page_table != nullptr;
  const bool pages = a.page_mode != 0;
  hipError_t e = max_group > 1 ? launch_logits<kScoreGroupTiles>(a, grid1, row_dim, paged, pages, stream)
                               : launch_logits<1>(a, grid1, row_dim, paged, pages, stream);
  if (e != hipSuccess) return e;
  const int outs = a.per_layer ? a.n_layers : 1;  // outputs per (group, sequence)
  if (pages) {
    const int max_pages = (a.dims.max_len + (1 << a.page_shift) - 1) >> a.page_shift;
    dim3 grid2((max_pages + kScoreFinishPages - 1) / kScoreFinishPages, a.groups * outs, B);
    hipLaunchKernelGGL(score_finish_pages_kernel, grid2, dim3(kFinishPagesThreads), 0, stream, a);
  } else {
    dim3 grid2((a.dims.max_len + kScoreFinishChunk - 1) / kScoreFinishChunk, a.groups * outs, B);
    hipLaunchKernelGGL(score_finish_kernel, grid2, dim3(kFinishThreads), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace dustin
