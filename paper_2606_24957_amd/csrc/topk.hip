// topk.hip -- tiered hybrid selection (Eq. 6), bit-exact and deterministic.
//
// One workgroup of 1024 threads (16 waves) per (sequence, selection group).  The row's
// order-preserving keys are staged in LDS, a segment at a time (one segment holds a whole
// row of up to ~32K positions, so such a row is read from HBM once per tier); the chosen
// set is an LDS bitmap.  Inside a segment wave w owns a contiguous run of positions and
// walks it 64 at a time, so a ballot covers two whole bitmap words that only this wave
// writes.
//
// Each tier selects `need` more positions among the clear bits by (key desc, position
// asc), key = the order-preserving uint32 of the fp32 score:
//   1. 12-bit histogram of the key's top digit over the free positions, then the digit
//      whose cumulative count from the top reaches `need`;
//   2. the same for bits 19..10 and then 9..0 among the free keys matching the prefix so
//      far, which yields the threshold key tau and how many keys equal to tau still fit;
//   3. in position order, every free key above tau and the first `remaining` equal to it
//      are marked.
// A final ordered pass over the bitmap writes the set in ascending position order.
//
// Steps 1-3 as written take five full scans of the row per tier; they remain as the
// general path (select_tier).  The tier normally runs select_tier_fast instead: the first
// digit over the whole row, then one pass that marks every key above the boundary digit
// and collects the keys of that digit as candidates; the lower digits and the tie order
// are then resolved among the candidates alone.
#include "kernels.hpp"

namespace dustin {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / kWave;
constexpr int kBins1 = kDigitBins;                      // first digit: key bits 31..20
constexpr int kBins = 1024;                             // later digits: 19..10, 9..0
constexpr int kTopkLds = 160 * 1024;                    // LDS of one gfx950 workgroup
constexpr int kLoadBatch = 16;                          // global loads in flight per thread
constexpr int kScanBatch = 8;                           // LDS key reads in flight per lane
constexpr int kSegQuantum = kTopkThreads * kLoadBatch;  // segments are multiples of this

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return (1ull << lane) - 1ull; }

// hist[bin] += 1 for every active lane.  (Aggregating lanes of one bin with ballots
// first measured slower on score rows than the LDS atomics it saves.)
__device__ __forceinline__ void hist_add(uint32_t* hist, uint32_t bin, bool active) {
  if (active) atomicAdd(&hist[bin], 1u);
}

struct TopkSmem {
  uint32_t hist[kBins1];
  uint32_t wave_cnt[kTopkWaves];
  uint32_t digit_cnt[kTopkWaves];  // find_digit's own per-wave sums (see there)
  uint32_t misc[4];
};

// Exclusive prefix over 16 per-wave counts (after a barrier) and their total.
__device__ __forceinline__ uint32_t wave_offset(const uint32_t* cnt, int wave, uint32_t* total) {
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kTopkWaves; ++w) {
    const uint32_t c = cnt[w];
    off += w < wave ? c : 0u;
    tot += c;
  }
  *total = tot;
  return off;
}

// Per-wave counts -> (this wave's exclusive offset, block total); two barriers.
__device__ __forceinline__ uint32_t block_offsets(TopkSmem& s, uint32_t wave_count, uint32_t* total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  if (lane == 0) s.wave_cnt[wave] = wave_count;
  __syncthreads();
  const uint32_t off = wave_offset(s.wave_cnt, wave, total);
  __syncthreads();
  return off;
}

// The digit where the count of keys from the top of hist[0..kN) reaches `remaining`;
// writes (digit, remaining within that digit) to s.misc[0..1].  Each thread reads its own
// bins once, keeps them in registers and returns them to zero, so that hist[0..kN) is zero
// again when this returns (the next histogram over at most kN bins needs no clearing).
// Its scan goes through digit_cnt, not wave_cnt, which other waves may still be reading
// when a wave enters here.
template <int kN>
__device__ void find_digit(TopkSmem& s, uint32_t remaining) {
  constexpr int per = kN / kTopkThreads;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int lo = (kTopkThreads - 1 - tid) * per;  // thread 0 owns the highest bins
  uint32_t v[per];
  uint32_t mine = 0;
#pragma unroll
  for (int i = 0; i < per; ++i) {
    v[i] = s.hist[lo + i];
    mine += v[i];
  }
#pragma unroll
  for (int i = 0; i < per; ++i) s.hist[lo + i] = 0u;
  uint32_t inc = mine;  // inclusive scan in tid order = from the top bin down
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t y = __shfl_up(inc, off);
    if (lane >= off) inc += y;
  }
  if (lane == kWave - 1) s.digit_cnt[wave] = inc;
  __syncthreads();
  uint32_t tot;
  const uint32_t above = wave_offset(s.digit_cnt, wave, &tot) + inc - mine;  // keys in higher bins
  if (above < remaining && above + mine >= remaining) {
    uint32_t run = above;
    bool found = false;
#pragma unroll
    for (int i = per - 1; i >= 0; --i) {
      if (!found && run + v[i] >= remaining) {
        s.misc[0] = (uint32_t)(lo + i);
        s.misc[1] = remaining - run;
        found = true;
      }
      run += v[i];
    }
  }
  __syncthreads();
}

// One row's keys staged in LDS, `seg` positions at a time.
struct KeyStage {
  const float* row;
  uint32_t* keys;      // [seg] in LDS
  const uint32_t* bm;  // chosen bitmap, [ceil(N / 32)] words in LDS
  int N, seg, nseg, loaded;

  // positions [s seg, s seg + seg) -> keys: thread t takes j = t + 1024 r, sixteen loads
  // in flight at a time (seg is a multiple of kSegQuantum; positions past the row read
  // its last element and store 0)
  __device__ void load(int s) {
    if (loaded == s) return;
    __syncthreads();  // the previous segment's readers are done
    const int base = s * seg, R = seg / kTopkThreads;
    for (int r0 = 0; r0 < R; r0 += kLoadBatch) {
      float v[kLoadBatch];
#pragma unroll
      for (int u = 0; u < kLoadBatch; ++u) {
        const int n = base + (int)threadIdx.x + (r0 + u) * kTopkThreads;
        v[u] = row[n < N ? n : N - 1];
      }
#pragma unroll
      for (int u = 0; u < kLoadBatch; ++u) {
        const int j = (int)threadIdx.x + (r0 + u) * kTopkThreads;
        keys[j] = base + j < N ? order_key(v[u]) : 0u;
      }
    }
    __syncthreads();
    loaded = s;
  }

  // Wave w's run inside the segment is [w per, (w + 1) per), per a multiple of 64.
  __device__ int per_wave() const { return seg / kTopkWaves; }

  // Is the segment-relative position j free (inside the row and not yet chosen)?
  __device__ bool free_at(int s, int j) const {
    const int n = s * seg + j;
    return n < N && !((bm[n >> 5] >> (n & 31)) & 1u);
  }

  // Keys and free flags of kScanBatch consecutive 64-position steps of this wave's run,
  // steps i0 .. i0 + kScanBatch - 1 (steps past the run read step 0 and come out taken).
  __device__ __forceinline__ void fetch(int s, int w0, int i0, int steps, uint32_t* key,
                                        bool* fr) const {
    const int lane = threadIdx.x & (kWave - 1);
    uint32_t word[kScanBatch];
#pragma unroll
    for (int u = 0; u < kScanBatch; ++u) {
      const int i = i0 + u < steps ? i0 + u : 0;
      const int j = w0 + i * kWave + lane;
      const int n = min(s * seg + j, N - 1);
      key[u] = keys[j];
      word[u] = bm[n >> 5];
    }
#pragma unroll
    for (int u = 0; u < kScanBatch; ++u) {
      const int n = s * seg + w0 + (i0 + u) * kWave + lane;
      fr[u] = i0 + u < steps && n < N && !((word[u] >> (n & 31)) & 1u);
    }
  }
};

// ORs the ballot of the 64 positions starting at n (a multiple of 64) into the bitmap, with
// LDS atomic ORs whose result is not used: one instruction each and no wait, where a read,
// OR and write would wait for the read (the word is the calling wave's alone either way).
__device__ __forceinline__ void mark64(uint32_t* bm, int n, int N, uint64_t m) {
  const int lane = threadIdx.x & (kWave - 1);
  if (lane == 0 && n < N && (uint32_t)m)
    __hip_atomic_fetch_or(&bm[n >> 5], (uint32_t)m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  if (lane == 32 && n + 32 < N && (uint32_t)(m >> 32))
    __hip_atomic_fetch_or(&bm[(n >> 5) + 1], (uint32_t)(m >> 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ void select_tier(TopkSmem& s, KeyStage& ks, uint32_t need, uint32_t* bm) {
  if (need == 0) return;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int per = ks.per_wave(), w0 = wave * per, steps = per / kWave;

  // ---- 1. the three digits: 31..20 over every free key, then 19..10 and 9..0 among
  // the free keys that match the digits found so far
  uint32_t prefix = 0, pmask = 0, remaining = need;
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = pass == 0 ? 20 : (pass == 1 ? 10 : 0);
    const uint32_t dmask = pass == 0 ? 4095u : 1023u;
    const int nbins = pass == 0 ? kBins1 : kBins;
    for (int i = tid; i < nbins; i += kTopkThreads) s.hist[i] = 0u;
    __syncthreads();
    for (int sg = 0; sg < ks.nseg; ++sg) {
      ks.load(sg);
      for (int i0 = 0; i0 < steps; i0 += kScanBatch) {
        uint32_t key[kScanBatch];
        bool fr[kScanBatch];
        ks.fetch(sg, w0, i0, steps, key, fr);
#pragma unroll
        for (int u = 0; u < kScanBatch; ++u)
          hist_add(s.hist, (key[u] >> sh) & dmask, fr[u] && (key[u] & pmask) == prefix);
      }
    }
    __syncthreads();
    if (pass == 0)
      find_digit<kBins1>(s, remaining);
    else
      find_digit<kBins>(s, remaining);
    prefix |= s.misc[0] << sh;
    pmask |= dmask << sh;
    remaining = s.misc[1];
  }
  const uint32_t tau = prefix;

  // ---- 2. ordered marking: every free key above tau, then the first `remaining` free
  // keys equal to tau in position order
  uint32_t rank_base = 0;
  for (int sg = 0; sg < ks.nseg; ++sg) {
    ks.load(sg);
    uint32_t c = 0;
    for (int i0 = 0; i0 < steps; i0 += kScanBatch) {
      uint32_t key[kScanBatch];
      bool fr[kScanBatch];
      ks.fetch(sg, w0, i0, steps, key, fr);
#pragma unroll
      for (int u = 0; u < kScanBatch; ++u) c += __popcll(__ballot(fr[u] && key[u] == tau));
    }
    uint32_t seg_total;
    uint32_t rank = rank_base + block_offsets(s, c, &seg_total);
    for (int i0 = 0; i0 < steps; i0 += kScanBatch) {
      uint32_t key[kScanBatch];
      bool fr[kScanBatch];
      ks.fetch(sg, w0, i0, steps, key, fr);
      uint64_t take[kScanBatch];
#pragma unroll
      for (int u = 0; u < kScanBatch; ++u) {
        const bool eq = fr[u] && key[u] == tau;
        const uint64_t eqm = __ballot(eq);
        const uint32_t r = rank + __popcll(eqm & lanemask_lt(lane));
        rank += __popcll(eqm);
        take[u] = __ballot((fr[u] && key[u] > tau) || (eq && r < remaining));
      }
      // bitmap words change only after every read of this batch
#pragma unroll
      for (int u = 0; u < kScanBatch; ++u)
        if (i0 + u < steps) mark64(bm, sg * ks.seg + w0 + (i0 + u) * kWave, ks.N, take[u]);
    }
    rank_base += seg_total;
  }
  __syncthreads();
}

// Fast tier: two streamed passes over the row (from global memory; a row is L2-resident
// after the first) instead of five over LDS-staged keys.
//   A. 12-bit histogram of the top digit over the free keys -> boundary digit d1 and how
//      many keys r1 still fit inside it;
//   B. every free key above d1 is marked; the free keys of bin d1 are appended, unordered,
//      to a candidate list of (key, position);
// then the two lower digits run over the candidates only, the candidates above the exact
// threshold tau are marked, and the ties at tau are taken in position order by ranking them
// among themselves.  If the candidate list or the tie set is too large (heavily tied
// rows), the rest of the tier runs through select_tier, which only ever sees what is still
// free, so the chosen set is the same either way.
constexpr int kMaxRankedTies = 1024;
constexpr int kFastBatch = 8;  // 64-position groups of a wave loaded together

__device__ __forceinline__ void select_tier_fast(TopkSmem& s, KeyStage& ks, uint32_t need, uint32_t* bm, uint32_t* cand,
                                 int cap, uint32_t* hist = nullptr, int n_sink = 0, int n_window = 0) {
  if (need == 0) {
    if (hist)
      for (int i = threadIdx.x; i < kBins1; i += kTopkThreads) hist[i] = 0u;
    return;
  }
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int N = ks.N;
  const int ngroups = (N + kWave - 1) / kWave;  // 64-position groups
  // wave w takes the run of groups [w gpw, (w + 1) gpw), kFastBatch at a time; a run of up
  // to kFastBatch groups is loaded once for both passes
  const int gpw = (ngroups + kTopkWaves - 1) / kTopkWaves;
  const int g_first = wave * gpw;
  const bool resident = gpw <= kFastBatch;
  // the row through a buffer resource: loads past its N values read 0.0, at positions the
  // bitmap (padded with taken bits to a whole number of groups) marks taken
  // (the row pointer comes through a small local array: made explicitly uniform, so that
  // the resource lives in scalar registers)
  // (readfirstlane returns a signed int: each half is taken back through uint32_t, so that
  // the low half is not sign-extended into the high one)
  const uint64_t rp = reinterpret_cast<uint64_t>(ks.row);
  const uint32_t rp_hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(rp >> 32));
  const uint32_t rp_lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)rp);
  const uint64_t rpu = ((uint64_t)rp_hi << 32) | (uint64_t)rp_lo;
  const auto rs = __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(rpu), 0,
                                                    __builtin_amdgcn_readfirstlane(N * 4), 0x00020000);
  const int lane_pos = g_first * kWave + lane;  // this lane's position in the run's first group
  const uint32_t* const bm_lane = bm + 2 * g_first + (lane >> 5);  // its bitmap word there
  const int bit = lane & 31;
  uint32_t kb[kFastBatch];
  auto load_batch = [&](int i0) {
    float v[kFastBatch];
    const int off = (lane_pos + i0 * kWave) * 4;
#pragma unroll
    for (int u = 0; u < kFastBatch; ++u)
      v[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off + u * kWave * 4, 0, 0));
#pragma unroll
    for (int u = 0; u < kFastBatch; ++u) kb[u] = order_key(v[u]);
  };
  // free flags of the batch at i0: inside this wave's run and the row, and not yet chosen
  auto free_flags = [&](int i0, bool* fr) {
    uint32_t word[kFastBatch];
#pragma unroll
    for (int u = 0; u < kFastBatch; ++u) word[u] = bm_lane[2 * (i0 + u)];
#pragma unroll
    for (int u = 0; u < kFastBatch; ++u)
      fr[u] = i0 + u < gpw && g_first + i0 + u < ngroups && !((word[u] >> bit) & 1u);
  };
  if (resident) load_batch(0);

  // ---- A (or the row's histogram counted when the scores were written, less the protected
  // positions, which are taken when the tier starts: the same counts over the free keys;
  // the histogram is then returned to zero for the next call)
  if (hist) {
    for (int i = tid; i < kBins1; i += kTopkThreads) s.hist[i] = hist[i];
    __syncthreads();
    const int s0 = min(n_sink, N), w0 = max(s0, N - n_window), np = s0 + (N - w0);
    for (int i = tid; i < np; i += kTopkThreads) {
      const int n = i < s0 ? i : w0 + (i - s0);
      atomicSub(&s.hist[order_key(ks.row[n]) >> 20], 1u);
    }
    for (int i = tid; i < kBins1; i += kTopkThreads) hist[i] = 0u;
  } else {
    for (int i = tid; i < kBins1; i += kTopkThreads) s.hist[i] = 0u;
    __syncthreads();
    for (int i0 = 0; i0 < gpw; i0 += kFastBatch) {
      if (!resident) load_batch(i0);
      bool fr[kFastBatch];
      free_flags(i0, fr);
#pragma unroll
      for (int u = 0; u < kFastBatch; ++u) hist_add(s.hist, kb[u] >> 20, fr[u]);
    }
  }
  __syncthreads();
  find_digit<kBins1>(s, need);
  const uint32_t d1 = s.misc[0], r1 = s.misc[1];

  // ---- B (each wave appends to its own slice of the candidate list; a wave whose slice
  // would overflow stops appending, and the tier then takes the general path below)
  const int wcap = cap / kTopkWaves;
  uint32_t* const wlist = cand + 2 * wave * wcap;
  uint32_t wcount = 0;  // wave-uniform
  for (int i0 = 0; i0 < gpw; i0 += kFastBatch) {
    if (!resident) load_batch(i0);
    bool fr[kFastBatch];
    free_flags(i0, fr);
    uint64_t take[kFastBatch];
#pragma unroll
    for (int u = 0; u < kFastBatch; ++u) {
      const uint32_t dig = kb[u] >> 20;
      take[u] = __ballot(fr[u] && dig > d1);
      const bool inbin = fr[u] && dig == d1;
      const uint64_t cm = __ballot(inbin);
      if (cm) {
        const uint32_t c = (uint32_t)__popcll(cm);
        if (wcount + c <= (uint32_t)wcap && inbin) {
          const uint32_t at = wcount + __builtin_amdgcn_mbcnt_hi((uint32_t)(cm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)cm, 0u));
          *reinterpret_cast<u32x2*>(wlist + 2 * at) = u32x2{kb[u], (uint32_t)(lane_pos + (i0 + u) * kWave)};
        }
        wcount += c;
      }
    }
    // the bitmap words of the batch's groups are this wave's alone: lanes 0 and 32 write the
    // low and the high word of each group, after every read of the batch
#pragma unroll
    for (int u = 0; u < kFastBatch; ++u) {
      if (take[u] && (lane & 31) == 0) {
        uint32_t* const w = const_cast<uint32_t*>(bm_lane) + 2 * (i0 + u);
        *w |= lane == 0 ? (uint32_t)take[u] : (uint32_t)(take[u] >> 32);
      }
    }
  }
  if (lane == 0) s.wave_cnt[wave] = wcount;
  if (tid == 0) s.misc[3] = 0u;  // the tie count below
  __syncthreads();
  bool overflow = false;
#pragma unroll
  for (int w = 0; w < kTopkWaves; ++w) overflow |= s.wave_cnt[w] > (uint32_t)wcap;
  if (overflow) {
    ks.loaded = -1;
    select_tier(s, ks, r1, bm);
    return;
  }
  // from here on every wave works through its own candidates

  // ---- the lower digits among the candidates
  uint32_t prefix = d1 << 20, pmask = 4095u << 20, remaining = r1;
  for (int pass = 0; pass < 2; ++pass) {
    const int sh = pass == 0 ? 10 : 0;
    // hist is zero here: the previous find_digit left it so
    for (uint32_t c = lane; c < wcount; c += kWave) {
      const uint32_t key = wlist[2 * c];
      if ((key & pmask) == prefix) atomicAdd(&s.hist[(key >> sh) & 1023u], 1u);
    }
    __syncthreads();
    find_digit<kBins>(s, remaining);
    prefix |= s.misc[0] << sh;
    pmask |= 1023u << sh;
    remaining = s.misc[1];
  }
  const uint32_t tau = prefix;

  // ---- candidates above tau are taken; the ties at tau are collected
  uint32_t* const ties = s.hist;  // positions of the candidates equal to tau
  for (uint32_t c = lane; c < wcount; c += kWave) {
    const uint32_t key = wlist[2 * c], n = wlist[2 * c + 1];
    if (key > tau) {
      atomicOr(&bm[n >> 5], 1u << (n & 31));
    } else if (key == tau) {
      const uint32_t at = atomicAdd(&s.misc[3], 1u);
      if (at < (uint32_t)kMaxRankedTies) ties[at] = n;
    }
  }
  __syncthreads();
  const uint32_t nt = s.misc[3];
  if (nt > (uint32_t)kMaxRankedTies) {  // many equal keys: the ordered full-row path
    ks.loaded = -1;
    select_tier(s, ks, remaining, bm);
    return;
  }
  // tie t is taken iff fewer than `remaining` ties precede it in position
  for (uint32_t t = tid; t < nt; t += kTopkThreads) {
    const uint32_t n = ties[t];
    uint32_t rank = 0;
    for (uint32_t o = 0; o < nt; ++o) rank += ties[o] < n;
    if (rank < remaining) atomicOr(&bm[n >> 5], 1u << (n & 31));
  }
  __syncthreads();
}

// The same, as a call of its own (the rare fallback of the tier hand-off below).
__device__ __noinline__ void select_tier_fast_outlined(TopkSmem& s, KeyStage& ks, uint32_t need, uint32_t* bm,
                                                       uint32_t* cand, int cap) {
  select_tier_fast(s, ks, need, bm, cand, cap);
}

// Key-segment length for rows of up to max_len positions: the LDS left beside the
// static state and the bitmap, a multiple of kSegQuantum, at most the row rounded up.
// Bitmap words kept for rows of up to max_len positions: two per 64-position group, plus the
// groups past the row that the waves' runs (16 runs of whole groups, up to 15 groups past
// the row) and a last batch (up to 7 groups past a run) may read, all initialised as taken.
__host__ __device__ inline int topk_bitmap_words(int max_len) { return 2 * ((max_len + 63) / 64 + 24); }

static int topk_segment(int max_len) {
  const int nwords = topk_bitmap_words(max_len);
  const int avail = (kTopkLds - (int)sizeof(TopkSmem)) / 4 - nwords;
  const int cap = avail / kSegQuantum * kSegQuantum;
  const int row = (max_len + kSegQuantum - 1) / kSegQuantum * kSegQuantum;
  return row < cap ? row : cap;
}

// Calls emit(i, n) for the set bits n of words(w), w < nwords, positions below N, in
// ascending order of n, i = 0, 1, ...; returns how many there were.  Wave w owns the
// words [w W, (w + 1) W), one word per lane per iteration (two passes: counts, then
// positions).
template <class Words, class Emit>
__device__ uint32_t ordered_bits(TopkSmem& s, int nwords, int N, Words words, Emit emit) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int wper = (nwords + kTopkWaves - 1) / kTopkWaves;
  const int w0 = min(nwords, wave * wper), w1 = min(nwords, w0 + wper);
  auto word_bits = [&](int w) -> uint32_t {
    uint32_t bits = w < w1 ? words(w) : 0u;
    if (w == nwords - 1 && (N & 31)) bits &= (1u << (N & 31)) - 1u;
    return bits;
  };
  uint32_t c = 0;
  for (int base = w0; base < w1; base += kWave) {
    uint32_t pc = __popc(word_bits(base + lane));
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) pc += __shfl_xor(pc, off);
    c += pc;  // every lane holds this iteration's wave total
  }
  uint32_t total;
  uint32_t o = block_offsets(s, c, &total);
  for (int base = w0; base < w1; base += kWave) {
    const int w = base + lane;
    uint32_t bits = word_bits(w);
    const uint32_t pc = __popc(bits);
    uint32_t inc = pc;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const uint32_t y = __shfl_up(inc, off);
      if (lane >= off) inc += y;
    }
    uint32_t pos = o + inc - pc;
    o += __shfl(inc, kWave - 1);
    while (bits) {
      const int i = __ffs(bits) - 1;
      bits &= bits - 1u;
      emit(pos, w * 32 + i);
      ++pos;
    }
  }
  return total;
}

// The `need` best of a list of c (key, position) pairs in LDS, the positions ascending
// (key[i] = list[2 i], position = list[2 i + 1]), by (key desc, position asc): the three
// digits of the threshold key tau as in select_tier, over the listed keys, then every key
// above tau and the first `remaining` keys equal to it in list order are marked in bm.
__device__ void select_list(TopkSmem& s, const uint32_t* list, int c, uint32_t need, uint32_t* bm) {
  if (need == 0) return;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  for (int i = tid; i < kBins1; i += kTopkThreads) s.hist[i] = 0u;
  __syncthreads();
  uint32_t prefix = 0, pmask = 0, remaining = need;
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = pass == 0 ? 20 : (pass == 1 ? 10 : 0);
    const uint32_t dmask = pass == 0 ? 4095u : 1023u;
    for (int i = tid; i < c; i += kTopkThreads) {
      const uint32_t key = list[2 * i];
      if ((key & pmask) == prefix) atomicAdd(&s.hist[(key >> sh) & dmask], 1u);
    }
    __syncthreads();
    if (pass == 0)
      find_digit<kBins1>(s, remaining);
    else
      find_digit<kBins>(s, remaining);
    prefix |= s.misc[0] << sh;
    pmask |= dmask << sh;
    remaining = s.misc[1];
  }
  const uint32_t tau = prefix;
  // the list in chunks of the block, in order: ties at tau ranked by list position
  uint32_t rank = 0;
  for (int i0 = 0; i0 < c; i0 += kTopkThreads) {
    const int i = i0 + tid;
    const uint32_t key = i < c ? list[2 * i] : 0u, n = i < c ? list[2 * i + 1] : 0u;
    const bool eq = i < c && key == tau;
    const uint64_t em = __ballot(eq);
    uint32_t chunk_total;
    const uint32_t before = rank + block_offsets(s, __popcll(em), &chunk_total) + __popcll(em & lanemask_lt(lane));
    if (i < c && (key > tau || (eq && before < remaining))) atomicOr(&bm[n >> 5], 1u << (n & 31));
    rank += chunk_total;
  }
  __syncthreads();
}

// Agent-scope (cross-XCD) write-through stores and loads of the tier hand-off, through a
// buffer resource over the row's two bitmaps.
constexpr int kSC1 = 16;

// One workgroup per (selection group, tier, sequence).  The two tiers of Eq. 6 are
// independent up to a final filter: with C_T the k - |P| best free positions by S_T,
// I_T is the k - m - |P| best of C_T \ I_D (|I_D| = m, so C_T holds at least k - m - |P|
// positions outside I_D, and every position that beats one of those in S_T order is in
// C_T).  So, when both tiers are present, workgroup 0 of the row selects I_D and
// workgroup 1 selects C_T at the same time; each publishes its chosen set as a bitmap and
// counts itself in, and the one that arrives second lists C_T \ I_D in position order,
// selects its k - m - |P| best by S_T among the list alone, and writes I.  A row with one
// tier (m = 0, or m = k - |P|, or one score array absent) is selected by workgroup 0 alone.
__global__ __launch_bounds__(kTopkThreads) void topk_kernel(TopkArgs a, int seg) {
  extern __shared__ __align__(16) uint32_t dyn[];  // [seg] staged keys | [nwords] chosen bitmap
  __shared__ TopkSmem s;
  const int go = blockIdx.x % a.groups, tier = blockIdx.x / a.groups, b = blockIdx.y;
  const int tid = threadIdx.x;
  const int N = a.dims.len(b);
  const int P = a.n_sink + a.n_window;
  const int k = clampi(a.dims.budget ? a.dims.budget[b] : a.dims.k_max, P, a.dims.k_max);
  int m = clampi(a.dims.m ? a.dims.m[b] : a.dims.m_scalar, 0, k - P);
  if (!a.s_draft) m = 0;
  if (!a.s_target) m = k - P;
  int32_t* out = a.idx + (int64_t)b * a.idx_sb + (int64_t)go * a.idx_sg;
  // the rows' histograms, when given (one selection group): each is read by the tier that
  // uses it first, or else cleared here, so that every call leaves them at zero
  uint32_t* const hd = a.hist_d ? a.hist_d + (int64_t)b * kBins1 : nullptr;
  uint32_t* const ht = a.hist_t ? a.hist_t + (int64_t)b * kBins1 : nullptr;
  auto clear = [&](uint32_t* h) {
    if (h)
      for (int i = tid; i < kBins1; i += kTopkThreads) h[i] = 0u;
  };
  if (N <= k) {
    if (tier == 0) {
      for (int n = tid; n < N; n += kTopkThreads) out[n] = n;
      if (tid == 0) a.count[b * a.groups + go] = N;
      clear(hd);
      clear(ht);
    }
    return;
  }
  const bool has_d = a.s_draft && m > 0;
  const bool has_t = a.s_target && k - m - P > 0;
  const bool both = has_d && has_t && a.counters;  // kernel-uniform but for m
  if (tier == 1 && !both) return;
  const bool run_d = both ? tier == 0 : has_d;
  const bool run_t = both ? tier == 1 : has_t;
  // a histogram serves a tier that is its workgroup's first job (the target tier after the
  // draft tier in one workgroup has I_D taken as well, which the histogram does not know)
  if (tier == 0) {
    if (!run_d) clear(hd);
    if (!both && !(run_t && !run_d)) clear(ht);
  }

  uint32_t* bm = dyn + seg;
  // protected positions (and the padding past N) start out taken
  const int nwords = (N + 31) / 32;
  // (bit i of word w is position 32 w + i; taken: below n_sink, or at or above N - n_window,
  // which includes every position at or above N)
  auto below = [](int x, int n0) -> uint32_t {  // bits i with n0 + i < x
    const int c = x - n0;
    return c <= 0 ? 0u : (c >= 32 ? ~0u : (1u << c) - 1u);
  };
  for (int w = tid; w < topk_bitmap_words(N); w += kTopkThreads)
    bm[w] = below(a.n_sink, w * 32) | ~below(N - a.n_window, w * 32);
  // a row shorter than the segment uses a shorter one (still a multiple of kSegQuantum)
  const int rseg = min(seg, (N + kSegQuantum - 1) / kSegQuantum * kSegQuantum);
  KeyStage ks{nullptr, dyn, bm, N, rseg, (N + rseg - 1) / rseg, -1};
  __syncthreads();
  // the candidate list of the fast tier uses the key-staging area: (key, position) pairs
  const int cap = rseg / 2;
  const float* row_t = a.s_target ? a.s_target + (int64_t)b * a.t_sb + (int64_t)go * a.t_sg : nullptr;
  // the tiers this workgroup selects, in order (one call site, so that the tier code is
  // inlined once): D, then T -- with both tiers side by side T takes C_T, the k - |P|
  // best, alone it takes I_T itself
  const float* rows[2];
  uint32_t needs[2];
  int jobs = 0;
  if (run_d) {
    rows[jobs] = a.s_draft + (int64_t)b * a.d_sb + (int64_t)go * a.d_sg;
    needs[jobs++] = (uint32_t)m;
  }
  if (run_t) {
    rows[jobs] = row_t;
    needs[jobs++] = (uint32_t)(both ? k - P : k - m - P);
  }
  for (int j = 0; j < jobs; ++j) {
    ks.row = j == 0 ? rows[0] : rows[1];
    ks.loaded = -1;
    select_tier_fast(s, ks, j == 0 ? needs[0] : needs[1], bm, dyn, cap, j == 0 ? (run_d ? hd : ht) : nullptr,
                     a.n_sink, a.n_window);
  }

  if (both) {
    // publish this tier's bitmap, count in; the second to arrive merges
    const int r = b * a.groups + go;
    uint32_t* const maps = a.bitmaps + (int64_t)r * 2 * a.words;
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(maps, 0, 2 * a.words * 4, 0x00020000);
    for (int w = tid; w < nwords; w += kTopkThreads)
      __builtin_amdgcn_raw_buffer_store_b32(bm[w], rs, (tier * a.words + w) * 4, 0, kSC1);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's stores have completed
    __syncthreads();                     // ... and every other thread's
    if (tid == 0)
      s.misc[2] = __hip_atomic_fetch_add(a.counters + r, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 1u;
    __syncthreads();
    if (!s.misc[2]) return;
    if (tid == 0) __hip_atomic_store(a.counters + r, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // the other tier's bitmap; then bm := P u I_D and the candidates C_T \ I_D listed in
    // position order (in the key-staging area, (key, position) pairs; keys filled below)
    const int other = 1 - tier;
    for (int w = tid; w < nwords; w += kTopkThreads) {
      const uint32_t mine = bm[w];
      const uint32_t theirs = __builtin_amdgcn_raw_buffer_load_b32(rs, (other * a.words + w) * 4, 0, kSC1);
      const uint32_t bd = tier == 0 ? mine : theirs, bt = tier == 0 ? theirs : mine;
      bm[w] = bd;
      dyn[seg - nwords + w] = bt & ~bd;  // C_T \ I_D, at the end of the key-staging area
    }
    __syncthreads();
    const uint32_t* cand_words = dyn + seg - nwords;
    const uint32_t c = ordered_bits(s, nwords, N, [&](int w) { return cand_words[w]; }, [](uint32_t, int) {});
    const uint32_t need = (uint32_t)(k - m - P);
    if (2 * c + nwords > (uint32_t)seg) {
      // too many to list beside the words: the target tier again over the whole row, with
      // P u I_D taken (the sequential form of Eq. 6)
      ks.row = row_t;
      ks.loaded = -1;
      select_tier_fast_outlined(s, ks, need, bm, dyn, cap);
    } else {
      ordered_bits(s, nwords, N, [&](int w) { return cand_words[w]; },
                   [&](uint32_t i, int n) { dyn[2 * i + 1] = (uint32_t)n; });
      __syncthreads();
      for (uint32_t i = tid; i < c; i += kTopkThreads) dyn[2 * i] = order_key(row_t[dyn[2 * i + 1]]);
      __syncthreads();
      select_list(s, dyn, (int)c, need, bm);
    }
  }

  // ascending write-out of P u I_D u I_T
  const uint32_t total = ordered_bits(s, nwords, N, [&](int w) { return bm[w]; }, [&](uint32_t pos, int n) {
    if (pos < (uint32_t)k) out[pos] = n;  // never past the budget
  });
  if (tid == 0) a.count[b * a.groups + go] = (int32_t)min(total, (uint32_t)k);
}

hipError_t launch_topk(const TopkArgs& a, int B, hipStream_t stream) {
  const int seg = topk_segment(a.dims.max_len);
  if (seg < kSegQuantum) return hipErrorInvalidValue;
  const size_t dyn = (size_t)(seg + topk_bitmap_words(a.dims.max_len)) * sizeof(uint32_t);
  // the dynamic-LDS limit is raised once per device (not per launch, so that launches can
  // be recorded in a graph after the first one)
  static bool lds_raised[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64 || !lds_raised[dev]) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(topk_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                            kTopkLds - (int)sizeof(TopkSmem));
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64) lds_raised[dev] = true;
  }
  // two workgroups per (group, sequence) when the tiers hand off (the second of a row
  // returns at once when its row has one tier)
  dim3 grid(a.groups * (a.counters ? 2 : 1), B);
  hipLaunchKernelGGL(topk_kernel, grid, dim3(kTopkThreads), dyn, stream, a, seg);
  return hipGetLastError();
}

}  // namespace dustin
