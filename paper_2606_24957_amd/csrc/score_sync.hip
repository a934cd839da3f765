// score_sync.hip -- Eq. 5 in one pass, for calls whose (head, query) pairs fit one MFMA
// column tile.
//
// The two-pass form (score.hip) writes every pair's logits to the workspace and reads them
// back, because the softmax of Eq. 5 needs each pair's max and sum over all N_b positions
// before any position's share is known.  When the pairs fit one 16-column MFMA tile (at
// most 16 pairs over at most 4 KV heads: the target's scoring heads for its last token, or
// the draft's scoring heads for its draft tokens), a workgroup's logits fit its registers
// instead and only the softmax statistics travel:
//   * one workgroup of 16 waves per (sequence b, chunk of C = 256 TW positions); wave w
//     takes TW tiles of 16 consecutive positions.  A tile's K rows of every used KV head
//     are multiplied by the 16 query columns on MFMA 16x16x32 (one accumulator per KV head;
//     a column keeps the one of its own head).  Lane (row r, group q) keeps the scaled
//     logits (log2 domain) of positions 4q .. 4q + 3 of the tile for column r.
//   * Per layer the workgroup reduces its (max, sum of exp2) per column, publishes them
//     with write-through stores, counts itself in on the sequence's counter and waits until
//     all G_b chunks of the sequence have.  It then merges the G_b statistics in chunk
//     order and adds sum_columns exp2(x - M) / Z to its positions' running sums, which live
//     in registers across the layers.
//   * The chunks of a sequence have consecutive block ids, so each XCD dispatches them after
//     every chunk of the earlier sequences: a waiting chunk only waits for chunks that hold a
//     CU or get one as earlier sequences finish (the host keeps G_b far below the CUs of the
//     chip).  The wait is bounded anyway: on a timeout the workgroup sets a flag in the
//     workspace and goes on.
//   * The next layer's first K rows and its queries are in flight across the wait.
//   * The last chunk of a sequence to leave returns the sequence's counters to zero.
#include <type_traits>

#include "kernels.hpp"

namespace dustin {

namespace {

constexpr int kSyncThreads = kSyncWaves * kWave;
constexpr int kSpinLimit = 1 << 16;  // polls of a counter (each a memory round trip)

// (m, s) <- the union of two (max, sum of exp2(x - max)) summaries
__device__ __forceinline__ void merge_ms(float& m, float& s, float mo, float so) {
  const float mn = fmaxf(m, mo);
  const float mu = mn == -INFINITY ? 0.f : mn;
  s = s * fast_exp2(m - mu) + so * fast_exp2(mo - mu);
  m = mn;
}

__device__ __forceinline__ float2 load_pair_sc1(const float2* p) {
  const uint64_t u = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)u), __uint_as_float((uint32_t)(u >> 32)));
}
__device__ __forceinline__ void store_pair_sc1(float2* p, float m, float s) {
  const uint64_t u = (uint64_t)__float_as_uint(m) | ((uint64_t)__float_as_uint(s) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

// LDS of a single-pass workgroup: the chunk's logits column by column, a pitch of C + 4
// staggering the columns over the banks (only the pairs' columns are written), and the
// paged rows' physical pages.
constexpr int kSyncMaxTW = 8;
constexpr int kSyncXPitch = kSyncWaves * kSyncMaxTW * 16 + 4;
struct SyncLds {
  float x[16 * kSyncXPitch];
  int page[kSyncWaves * kSyncMaxTW * 16];
  float2 st[kSyncWaves][16];
  float2 mz[16];
  uint32_t hist[kDigitBins];  // the chunk's outputs by top key digit (with a histogram)
};

// One call's share of the grid: block blk of the call's blocks.
template <int D, int NU, int TW, bool kPaged>
__device__ __forceinline__ void score_sync_call(const SyncCall& a, int blk, SyncLds& lds) {
  const SeqDims& dims = a.dims;
  constexpr int KS = D / 32;                 // MFMA k-steps of one KV head's row
  constexpr int HPS = 4 / KS;                // KV heads per load stage (64 bytes per lane)
  constexpr int SPT = (NU + HPS - 1) / HPS;  // load stages per tile
  constexpr int NST = TW * SPT;              // load stages per layer
  constexpr int C = kSyncWaves * TW * 16;    // positions per workgroup
  static_assert(TW % 2 == 0, "a layer's stages alternate between two buffers and end on the second");
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int lr = lane & 15, lg = lane >> 4;
  // (sequence, chunk) of this workgroup: a sequence's chunks are consecutive block ids, or,
  // when every sequence's chunks fit one XCD, consecutive among the ids of one XCD
  // (workgroups go to the XCDs round-robin by id): the chunks then share its L2 and pace
  int b, c;
  if (a.local) {
    const int x = blk & 7, k = blk >> 3;
    b = k / a.chunks * 8 + x;
    c = k % a.chunks;
  } else {
    b = blk / a.chunks;
    c = blk - b * a.chunks;
  }
  if (b >= a.batch) return;
  const int N = dims.len(b);
  const int G = (N + C - 1) / C;  // chunks of this sequence
  if (c >= G) return;
  const int nq = dims.nq(b);
  const int L = a.n_layers;
  if (a.hist)  // cleared now; the layers' barriers order this before the counting at the end
    for (int i = threadIdx.x; i < kDigitBins; i += kSyncThreads) lds.hist[i] = 0u;

  // column lr: (scoring head slot, query) on used KV head cu; columns past the pairs, and
  // queries past nq_b, count for nothing
  const int col = lr < a.np ? lr : 0;
  const bool col_ok = lr < a.np && (int)a.col_query[col] < nq;
  const int cu = a.col_u[col];
  const int64_t q_off = (int64_t)b * a.q_sb + (int64_t)a.col_query[col] * a.q_sj +
                        (int64_t)a.col_head[col] * a.q_sh + 8 * lg;
  const int p0 = c * C + wave * (TW * 16);  // this wave's first position

  // K rows through a buffer resource per layer (32-bit byte offsets, checked on the host):
  // this lane's row of tile t (clamped to the last position) and the stage's KV heads
  // (paged: the physical page of every row the wave reads, looked up once, kept in LDS so
  // that a stage's loads wait for no global load)
  int* const sm_page = lds.page;
  if constexpr (kPaged) {
    if (lg == 0) {
#pragma unroll
      for (int t = 0; t < TW; ++t) {
        const int p = min(p0 + 16 * t + lr, N - 1);
        sm_page[(wave * TW + t) * 16 + lr] =
            clampi(a.k.page_table[(int64_t)b * a.k.max_pages + (p >> a.k.page_shift)], 0, a.k.num_pages - 1);
      }
    }
    __syncthreads();
  }
  const uint32_t sn = (uint32_t)a.k.stride_n * 2u, sh = (uint32_t)a.k.stride_h * 2u;
  auto row_off = [&](int t) -> uint32_t {
    const int p = min(p0 + 16 * t + lr, N - 1);
    if constexpr (kPaged)
      return (uint32_t)sm_page[(wave * TW + t) * 16 + lr] * ((uint32_t)a.k.stride_page * 2u) +
             (uint32_t)(p & ((1 << a.k.page_shift) - 1)) * sn;
    else
      return (uint32_t)p * sn;
  };
  auto rsrc = [&](int l) {
    const uint16_t* base = a.k_layers[l] + (kPaged ? 0 : (int64_t)b * a.k.stride_b);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, a.extent, 0x00020000);
  };
  // stage s of tile t: KV heads s HPS .. s HPS + HPS - 1, in the MFMA A layout (row lr,
  // elements 32 kk + 8 lg .. + 7)
  auto issue = [&](__amdgpu_buffer_rsrc_t rs, int t, int s, u32x4 (&dst)[4]) {
    const uint32_t off = row_off(t) + 16u * lg;
#pragma unroll
    for (int h = 0; h < HPS; ++h) {
      const int u = s * HPS + h;
      if (u < NU) {
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
          dst[h * KS + kk] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, (int)((uint32_t)a.kv[u] * sh + 64u * kk), 0));
      }
    }
  };
  // B operand of layer l: column lr's query, elements 32 kk + 8 lg .. + 7 (zero when the
  // column counts for nothing; the load itself is unconditional)
  auto load_q = [&](int l, bf16x8 (&dst)[KS]) {
    const uint16_t* qp = a.q_layers[l] + q_off;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const u32x4 v = load16(qp + 32 * kk);
      dst[kk] = as_bf16x8(col_ok ? v : u32x4{0u, 0u, 0u, 0u});
    }
  };
  // With 64-element rows the next layer's queries are loaded with its first rows, before
  // the wait; with 128-element rows their registers are needed for the tiles, and they are
  // loaded after it.
  constexpr bool kQNext = D == 64;

  constexpr int kXPitch = kSyncXPitch;
  float* const sm_x = lds.x;
  auto& sm_st = lds.st;
  auto& sm_mz = lds.mz;
  int* const cnt = a.sync + b;
  int* const done = a.sync + kScoreSyncMaxBatch + b;
  int* const flag = a.sync + 2 * kScoreSyncMaxBatch;
  const int np = a.np;

  // A ring of NB load stages: stage qi's buffer is reloaded with stage qi + NB - 1 (of this
  // layer, or of the next one) as soon as qi is consumed, so NB - 1 stages are in flight
  // while one is computed, across the layer's end and the wait as well.  NB is a multiple
  // of the stages of a tile, so a group of NB stages holds whole tiles.
  constexpr int NB = SPT == 3 ? 3 : (NST < 4 ? NST : 4);
  static_assert(NST % NB == 0 && NB % SPT == 0, "groups of whole tiles");
  u32x4 buf[NB][4];
  bf16x8 bq[KS], bq_next[kQNext ? KS : 1];
  f32x4 acc_pos = {0.f, 0.f, 0.f, 0.f};  // threads below C / 4: positions 4 tid .. 4 tid + 3
  load_q(0, bq);
  auto rs = rsrc(0);
#pragma unroll
  for (int qi = 0; qi < NB - 1; ++qi) issue(rs, qi / SPT, qi % SPT, buf[qi]);
  for (int l = 0; l < L; ++l) {
    if constexpr (kQNext) {
      load_q(l + 1 < L ? l + 1 : l, bq_next);
    } else {
      if (l > 0) load_q(l, bq);
    }
    // the next layer's rows
    const auto rs_next = rsrc(l + 1 < L ? l + 1 : l);
    float m = -INFINITY, ssum = 0.f;  // running (max, sum of exp2) of column lr
    // ---- logits of the wave's TW tiles, NB stages at a time
#pragma unroll 1
    for (int g0 = 0; g0 < NST; g0 += NB) {
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int r = 0; r < NB; ++r) {
        const int qi = g0 + r, qn = qi + NB - 1, s = r % SPT;
        // the stage NB - 1 ahead: of this layer, else of the next one; past the last layer,
        // this layer's last stage again (its rows are in flight or in L2, so these loads,
        // which keep the number of loads behind every stage the same, cost no HBM traffic)
        const bool next = qn >= NST, past = next && l + 1 >= L;
        const int qs = past ? NST - 1 : (next ? qn - NST : qn);
        issue(next && !past ? rs_next : rs, qs / SPT, past ? (NST - 1) % SPT : (NB - 1 + r) % SPT,
              buf[(r + NB - 1) % NB]);
#pragma unroll
        for (int h = 0; h < HPS; ++h) {
          const int u = s * HPS + h;
          if (u < NU) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) acc = mfma16x16x32(as_bf16x8(buf[r][h * KS + kk]), bq[kk], acc);
            v = (NU == 1 || cu == u) ? acc : v;  // a column keeps its own KV head's products
          }
        }
        if (s == SPT - 1) {  // the tile is complete
          const int t = qi / SPT;
          const int pt = p0 + 16 * t + 4 * lg;  // this lane's first position of the tile
          f32x4 xv;
#pragma unroll
          for (int e = 0; e < 4; ++e) xv[e] = pt + e < N ? v[e] * a.scale_log2 : -INFINITY;
          if (lr < np) *reinterpret_cast<f32x4*>(sm_x + lr * kXPitch + (pt - c * C)) = xv;
          const float mt = fmaxf(fmaxf(xv[0], xv[1]), fmaxf(xv[2], xv[3]));
          const float mn = fmaxf(m, mt), mu = mn == -INFINITY ? 0.f : mn;
          ssum = ssum * fast_exp2(m - mu) + (fast_exp2(xv[0] - mu) + fast_exp2(xv[1] - mu)) +
                 (fast_exp2(xv[2] - mu) + fast_exp2(xv[3] - mu));
          m = mn;
          v = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
    rs = rs_next;

    // ---- (max, sum of exp2) of each column over the workgroup's positions
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float mo = __shfl_xor(m, off), so = __shfl_xor(ssum, off);
      merge_ms(m, ssum, mo, so);
    }
    if (lg == 0) sm_st[wave][lr] = make_float2(m, ssum);
    __syncthreads();
    // Wave 0 alone publishes, waits and merges; the other waves' next loads stay in flight
    // (a wait for this wave's write-through stores is a wait for all its loads as well).
    if (wave == 0) {
      float2* const stats_l = reinterpret_cast<float2*>(a.stats) + ((int64_t)l * a.batch + b) * a.chunks * 16;
      if (lane < 16) {  // the workgroup's summary, merged over the waves in order
        float M = -INFINITY, S = 0.f;
#pragma unroll
        for (int w = 0; w < kSyncWaves; ++w) merge_ms(M, S, sm_st[w][lr].x, sm_st[w][lr].y);
        if (G == 1) sm_mz[lr] = make_float2(M == -INFINITY ? 0.f : M, S > 0.f ? 1.f / S : 0.f);
        else store_pair_sc1(stats_l + c * 16 + lr, M, S);
      }
      if (G > 1) {
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the write-through stores have completed
        asm volatile("" ::: "memory");
        if (lane == 0) {
          __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          const int target = (l + 1) * G;
          for (int spins = 0; __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target;) {
            __builtin_amdgcn_s_sleep(1);
            if (++spins > kSpinLimit) {
              __hip_atomic_store(flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              break;
            }
          }
        }
        asm volatile("" ::: "memory");  // the summaries are read only after the count is complete
        // every chunk has published: lane group lg merges chunks lg, lg + 4, ... in order,
        // then the four groups are merged
        float M = -INFINITY, S = 0.f;
        for (int cc = lg; cc < G; cc += 4) {
          const float2 v = load_pair_sc1(stats_l + cc * 16 + lr);
          merge_ms(M, S, v.x, v.y);
        }
#pragma unroll
        for (int off = 16; off <= 32; off <<= 1) {
          const float mo = __shfl_xor(M, off), so = __shfl_xor(S, off);
          merge_ms(M, S, mo, so);
        }
        if (lane < 16) sm_mz[lr] = make_float2(M == -INFINITY ? 0.f : M, S > 0.f ? 1.f / S : 0.f);
      }
    }
    __syncthreads();

    // ---- this layer's share of four positions per thread: exp2(x - M) / Z summed over
    // the columns in column order
    if ((int)threadIdx.x < C / 4) {
      f32x4 y = {0.f, 0.f, 0.f, 0.f};
      for (int j = 0; j < np; ++j) {
        if ((int)a.col_query[j] >= nq) continue;  // uniform
        const f32x4 xv = *reinterpret_cast<const f32x4*>(sm_x + j * kXPitch + 4 * threadIdx.x);
        const float2 mz = sm_mz[j];
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] += fast_exp2(xv[e] - mz.x) * mz.y;
      }
      acc_pos += y;
    }
    __syncthreads();  // the logits have been read before the next layer writes its own
    if constexpr (kQNext)
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) bq[kk] = bq_next[kk];
  }

  // the last chunk of the sequence to leave returns its counters to zero
  if (G > 1 && threadIdx.x == 0) {
    if (__hip_atomic_fetch_add(done, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == G - 1) {
      __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  // out = init + the sums, for positions below N_b
  const int n0 = c * C + 4 * threadIdx.x;
  f32x4 val = {0.f, 0.f, 0.f, 0.f};
  if ((int)threadIdx.x < C / 4) {
    const float* init_row = a.init ? a.init + (int64_t)b * a.init_sb : nullptr;
    float* out_row = a.out + (int64_t)b * a.out_sb;
    const bool vec = n0 + 3 < N && ((uintptr_t)(out_row + n0) & 15) == 0 &&
                     (!init_row || ((uintptr_t)(init_row + n0) & 15) == 0);
    if (vec) {
      const f32x4 in = init_row ? *reinterpret_cast<const f32x4*>(init_row + n0) : f32x4{0.f, 0.f, 0.f, 0.f};
      val = in + acc_pos;
      *reinterpret_cast<f32x4*>(out_row + n0) = val;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        val[e] = (init_row && n0 + e < N ? init_row[n0 + e] : 0.f) + acc_pos[e];
        if (n0 + e < N) out_row[n0 + e] = val[e];
      }
    }
  }
  // the chunk's outputs counted by top key digit, then the non-zero bins added into the
  // sequence's histogram
  if (a.hist) {
    uint32_t* const h = lds.hist;
    if ((int)threadIdx.x < C / 4) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n0 + e < N) atomicAdd(&h[order_key(val[e]) >> 20], 1u);
    }
    __syncthreads();
    uint32_t* const gh = a.hist + (int64_t)b * kDigitBins;
    for (int i = threadIdx.x; i < kDigitBins; i += kSyncThreads) {
      const uint32_t v = h[i];
      if (v) __hip_atomic_fetch_add(gh + i, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Shapes of the single-pass form: row length, used KV heads, tiles per wave, paged.
template <int D_, int NU_, int TW_, bool P_>
struct SyncShape {
  static constexpr int D = D_, NU = NU_, TW = TW_;
  static constexpr bool kPaged = P_;
};
struct NoShape {};

// One launch runs one call, or two (the first call's blocks, a multiple of 8, then the
// second's: workgroups of the second start as the first's leave their CUs).
template <class S0, class S1>
__global__ __launch_bounds__(kSyncThreads) void score_sync_kernel(SyncArgs a) {
  __shared__ __attribute__((aligned(16))) SyncLds lds;
  if constexpr (std::is_same<S1, NoShape>::value) {
    score_sync_call<S0::D, S0::NU, S0::TW, S0::kPaged>(a.call[0], blockIdx.x, lds);
  } else {
    if ((int)blockIdx.x < a.blocks0)
      score_sync_call<S0::D, S0::NU, S0::TW, S0::kPaged>(a.call[0], blockIdx.x, lds);
    else
      score_sync_call<S1::D, S1::NU, S1::TW, S1::kPaged>(a.call[1], blockIdx.x - a.blocks0, lds);
  }
}

// blocks of one call: a multiple of 8 (sequences of an XCD, or all sequences, times chunks)
static int sync_blocks(const SyncCall& c) {
  const int seqs = c.local ? (c.batch + 7) / 8 * 8 : c.batch;
  return (seqs * c.chunks + 7) / 8 * 8;
}

template <class S0, class S1>
static hipError_t launch_sync(SyncArgs a, hipStream_t stream) {
  a.blocks0 = sync_blocks(a.call[0]);
  const int blocks = a.blocks0 + (std::is_same<S1, NoShape>::value ? 0 : sync_blocks(a.call[1]));
  hipLaunchKernelGGL((score_sync_kernel<S0, S1>), dim3(blocks), dim3(kSyncThreads), 0, stream, a);
  return hipGetLastError();
}

template <int D, int NU, bool kPaged>
static hipError_t launch_sync_tw(const SyncArgs& a, int tw, hipStream_t stream) {
  if (tw == 8) return launch_sync<SyncShape<D, NU, 8, kPaged>, NoShape>(a, stream);
  if (tw == 2) return launch_sync<SyncShape<D, NU, 2, kPaged>, NoShape>(a, stream);
  return hipErrorInvalidValue;
}

template <int D, bool kPaged>
static hipError_t launch_sync_nu(const SyncArgs& a, int nu, int tw, hipStream_t stream) {
  switch (nu) {
    case 1: return launch_sync_tw<D, 1, kPaged>(a, tw, stream);
    case 2: return launch_sync_tw<D, 2, kPaged>(a, tw, stream);
    case 3: return launch_sync_tw<D, 3, kPaged>(a, tw, stream);
    case 4: return launch_sync_tw<D, 4, kPaged>(a, tw, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_score_sync(const SyncArgs& a, hipStream_t stream) {
  const SyncCall& c = a.call[0];
  const bool paged = c.k.page_table != nullptr;
  if (c.head_dim == 128)
    return paged ? launch_sync_nu<128, true>(a, c.nu, c.tw, stream) : launch_sync_nu<128, false>(a, c.nu, c.tw, stream);
  if (c.head_dim == 64)
    return paged ? launch_sync_nu<64, true>(a, c.nu, c.tw, stream) : launch_sync_nu<64, false>(a, c.nu, c.tw, stream);
  return hipErrorInvalidValue;
}

// Two calls in one launch: the pairs of shapes compiled for it (a target call with four
// KV heads of 128-element rows, then a draft call with two KV heads of 64-element rows, as
// one verification step scores them); false when the two calls have another pair.
bool score_sync_pair_supported(const SyncCall& c0, const SyncCall& c1) {
  return c0.head_dim == 128 && c0.nu == 4 && c1.head_dim == 64 && c1.nu == 2 && c0.tw == c1.tw &&
         (c0.tw == 8 || c0.tw == 2) && (c0.k.page_table != nullptr) == (c1.k.page_table != nullptr);
}

hipError_t launch_score_sync_pair(const SyncArgs& a, hipStream_t stream) {
  const bool paged = a.call[0].k.page_table != nullptr;
  if (a.call[0].tw == 8)
    return paged ? launch_sync<SyncShape<128, 4, 8, true>, SyncShape<64, 2, 8, true>>(a, stream)
                 : launch_sync<SyncShape<128, 4, 8, false>, SyncShape<64, 2, 8, false>>(a, stream);
  return paged ? launch_sync<SyncShape<128, 4, 2, true>, SyncShape<64, 2, 2, true>>(a, stream)
               : launch_sync<SyncShape<128, 4, 2, false>, SyncShape<64, 2, 2, false>>(a, stream);
}

}  // namespace dustin
