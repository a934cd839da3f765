// topk.hip -- tiered hybrid selection (Eq. 6), bit-exact and deterministic.
//
// One workgroup of 1024 threads per (sequence, selection group).  The chosen set lives
// in an LDS bitmap of the row (thread t owns whole 32-position words, so no atomics are
// needed to mark).  Each tier is a radix select on the order key of the fp32 scores
// (digits of 11, 11 and 10 bits, MSB first, histograms in LDS) over the positions whose
// bit is still clear; it yields the threshold key tau and how many positions equal to
// tau still fit.  Marking takes every candidate above tau and the first of those equal
// to tau in position order (a block-wide scan over the words).  A final scan of the word
// popcounts writes the set in ascending order.
#include "kernels.hpp"

namespace dustin {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / kWave;

__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive scan of one value per thread over the block; returns the block total too.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* sm_wave, uint32_t& total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  uint32_t inc = x;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t y = __shfl_up(inc, off);
    if (lane >= off) inc += y;
  }
  if (lane == kWave - 1) sm_wave[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    uint32_t w = lane < kTopkWaves ? sm_wave[lane] : 0u;
#pragma unroll
    for (int off = 1; off < kTopkWaves; off <<= 1) {
      const uint32_t y = __shfl_up(w, off);
      if (lane >= off) w += y;
    }
    if (lane < kTopkWaves) sm_wave[lane] = w;  // inclusive wave totals
  }
  __syncthreads();
  const uint32_t before = wave ? sm_wave[wave - 1] : 0u;
  total = sm_wave[kTopkWaves - 1];
  __syncthreads();
  return before + inc - x;
}

// Select `need` more positions among the clear bits of `bm` (words [0, nwords)) by
// (key(s) descending, position ascending) and set their bits.
__device__ void select_tier(const float* __restrict__ s, int N, uint32_t need, uint32_t* bm,
                            int nwords, uint32_t* hist, uint32_t* sm_wave, uint32_t* sm_misc) {
  if (need == 0) return;
  const int tid = threadIdx.x;
  uint32_t prefix = 0, pmask = 0, remaining = need;
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = shifts[pass];
    const uint32_t dmask = (1u << widths[pass]) - 1u;
    const int nbins = 1 << widths[pass];
    for (int i = tid; i < nbins; i += kTopkThreads) hist[i] = 0u;
    __syncthreads();
    for (int w = tid; w < nwords; w += kTopkThreads) {
      const uint32_t free_bits = ~bm[w];
      if (!free_bits) continue;
      const int n0 = w * 32;
      for (int i = 0; i < 32; ++i) {
        const int n = n0 + i;
        if (n >= N) break;
        if (!((free_bits >> i) & 1u)) continue;
        const uint32_t key = order_key(s[n]);
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> sh) & dmask], 1u);
      }
    }
    __syncthreads();
    // suffix sums over bins: thread t scans its bins from the top (bins per thread = nbins/1024)
    const int per = nbins / kTopkThreads;  // 2 or 1
    const int lo = (kTopkThreads - 1 - tid) * per;  // thread 0 takes the highest bins
    uint32_t mine = 0;
    for (int i = 0; i < per; ++i) mine += hist[lo + i];
    uint32_t tot;
    const uint32_t above = block_exclusive_scan(mine, sm_wave, tot);  // count in higher bins
    // the digit where the cumulative count from the top reaches `remaining`
    if (above < remaining && above + mine >= remaining) {
      uint32_t run = above;
      for (int i = per - 1; i >= 0; --i) {
        const uint32_t c = hist[lo + i];
        if (run + c >= remaining) {
          sm_misc[0] = (uint32_t)(lo + i);
          sm_misc[1] = remaining - run;
          break;
        }
        run += c;
      }
    }
    __syncthreads();
    prefix |= sm_misc[0] << sh;
    pmask |= dmask << sh;
    remaining = sm_misc[1];
    __syncthreads();
  }
  const uint32_t tau = prefix;
  // mark: keys above tau, and the first `remaining` keys equal to tau in position order
  uint32_t carry = 0;
  for (int base = 0; base < nwords; base += kTopkThreads) {
    const int w = base + tid;
    uint32_t eq_bits = 0, gt_bits = 0;
    if (w < nwords) {
      const uint32_t free_bits = ~bm[w];
      const int n0 = w * 32;
      for (int i = 0; i < 32; ++i) {
        const int n = n0 + i;
        if (n >= N) break;
        if (!((free_bits >> i) & 1u)) continue;
        const uint32_t key = order_key(s[n]);
        if (key > tau) gt_bits |= 1u << i;
        else if (key == tau) eq_bits |= 1u << i;
      }
    }
    uint32_t tot;
    const uint32_t rank0 = carry + block_exclusive_scan(__popc(eq_bits), sm_wave, tot);
    if (w < nwords) {
      uint32_t take = gt_bits;
      uint32_t r = rank0;
      uint32_t eb = eq_bits;
      while (eb && r < remaining) {
        const uint32_t bit = eb & (~eb + 1u);
        take |= bit;
        eb ^= bit;
        ++r;
      }
      bm[w] |= take;
    }
    carry += tot;
  }
  __syncthreads();
}

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(TopkArgs a) {
  extern __shared__ uint32_t bm[];  // [nwords]
  __shared__ uint32_t hist[2048];
  __shared__ uint32_t sm_wave[kTopkWaves];
  __shared__ uint32_t sm_misc[2];
  const int go = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x;
  const int N = a.dims.len(b);
  const int P = a.n_sink + a.n_window;
  const int k = clampi(a.dims.budget ? a.dims.budget[b] : a.dims.k_max, P, a.dims.k_max);
  int m = clampi(a.dims.m ? a.dims.m[b] : a.dims.m_scalar, 0, k - P);
  if (!a.s_draft) m = 0;
  if (!a.s_target) m = k - P;
  int32_t* out = a.idx + (int64_t)b * a.idx_sb + (int64_t)go * a.idx_sg;
  if (N <= k) {
    for (int n = tid; n < N; n += kTopkThreads) out[n] = n;
    if (tid == 0) a.count[b * a.groups + go] = N;
    return;
  }
  const int nwords = (N + 31) / 32;
  for (int w = tid; w < nwords; w += kTopkThreads) {
    uint32_t bits = 0;
    const int n0 = w * 32;
    for (int i = 0; i < 32; ++i) {
      const int n = n0 + i;
      if (n < N && (n < a.n_sink || n >= N - a.n_window)) bits |= 1u << i;
    }
    // positions >= N are marked taken so they are never candidates
    if (n0 + 32 > N) bits |= ~0u << (N - n0);
    bm[w] = bits;
  }
  __syncthreads();
  if (a.s_draft)
    select_tier(a.s_draft + (int64_t)b * a.d_sb + (int64_t)go * a.d_sg, N, (uint32_t)m, bm, nwords,
                hist, sm_wave, sm_misc);
  if (a.s_target)
    select_tier(a.s_target + (int64_t)b * a.t_sb + (int64_t)go * a.t_sg, N, (uint32_t)(k - m - P), bm,
                nwords, hist, sm_wave, sm_misc);
  // ascending write-out of the set bits (positions >= N were set only as padding)
  uint32_t carry = 0;
  for (int base = 0; base < nwords; base += kTopkThreads) {
    const int w = base + tid;
    uint32_t bits = 0;
    if (w < nwords) {
      bits = bm[w];
      const int n0 = w * 32;
      if (n0 + 32 > N) bits &= (N - n0 >= 32) ? ~0u : ((1u << (N - n0)) - 1u);
    }
    uint32_t tot;
    uint32_t o = carry + block_exclusive_scan(__popc(bits), sm_wave, tot);
    while (bits) {
      const int i = __ffs(bits) - 1;
      bits &= bits - 1u;
      if (o < (uint32_t)k) out[o] = w * 32 + i;  // never past the budget
      ++o;
    }
    carry += tot;
  }
  if (tid == 0) a.count[b * a.groups + go] = (int32_t)min(carry, (uint32_t)k);
}

hipError_t launch_topk(const TopkArgs& a, int B, hipStream_t stream) {
  const int nwords = (a.dims.max_len + 31) / 32;
  dim3 grid(a.groups, B);
  hipLaunchKernelGGL(topk_kernel, grid, dim3(kTopkThreads), (size_t)nwords * sizeof(uint32_t),
                     stream, a);
  return hipGetLastError();
}

}  // namespace dustin
