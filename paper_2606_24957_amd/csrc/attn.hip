// attn.hip -- verification attention for gfx950: sparse (gathered selected positions)
// and dense (every committed position), both followed by the causal verification window.
//
// Work decomposition
//   unit  (split, sequence b, KV head g).  All T_b * (Hq / Hkv) query rows of the KV head
//         (its GQA group for every verification token) share each K/V row, so a selected
//         row is fetched from HBM once per layer.
//   slice the NH = 128 / DH workgroups of a unit each produce DH of the 128 output columns.
//         They all need the full K row (for the scores) but only their V columns.  Their
//         block ids are congruent mod 8, so the dispatcher puts them on the same XCD and
//         the K rows the first one fetches are served to the others from that XCD's L2.
//         This fills the chip without splitting the token list, so no partial results
//         travel through memory; token splits are only used when units are scarce, and
//         their partials are merged by a second, tiny kernel.
//   wave  walks 32-token steps of the unit (waves interleave steps), with the next step's
//         K/V loads in flight while the current one is computed:
//           S^T[32 tok x rows] = K[32 x 128] Q^T    MFMA 16x16x32, K rows loaded straight
//                                                   into A-operand registers (16 B/lane)
//           online softmax over tokens (fp32, exp2 domain); the running max is only moved
//           when a row's max grows by more than 2^8, a wave-uniform event, so the
//           accumulator is rarely rescaled
//           V^T via the LDS transpose load          V rows go to a wave-private LDS tile
//                                                   and come back with 4 tokens of one
//                                                   d column per lane, the PV layout
//           O^T[DH x rows] += V^T P^T               MFMA 16x16x32; a ones tile gives the
//                                                   row sums of the same bf16 weights
//   merge the W waves' (max, sum, acc) through LDS in a fixed order (deterministic).
//
// Gathered positions (sparse) and page translations (paged) are resolved once per unit
// into an LDS table of physical rows, so the inner loop does no dependent global loads.
#include "kernels.hpp"

namespace dustin {

constexpr int kD = 128;
#ifndef DUSTIN_ATTN_WAVES
#define DUSTIN_ATTN_WAVES 4
#endif
#ifndef DUSTIN_ATTN_DEPTH
#define DUSTIN_ATTN_DEPTH 1
#endif
constexpr int kAttnWavesPerGroup = DUSTIN_ATTN_WAVES;  // one wave per SIMD
constexpr int kDepth = DUSTIN_ATTN_DEPTH;              // steps in flight ahead of the compute
constexpr int kStageSteps = 192;         // 32-token steps whose rows are staged per chunk
constexpr float kRescaleLog2 = 8.f;      // lazy rescale threshold (factor 256)

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// gfx950 LDS transpose load: within each 16-lane group, lane i receives element i % 4 of
// the 8 bytes addressed by group lane 4 e + i / 4, for e = 0..3.
__device__ __forceinline__ v4i16 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)(reinterpret_cast<uintptr_t>(p)));
}

__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

template <int NKS>
struct StepRegs {
  u32x4 k[2][4];    // K rows of the step's two 16-token tiles (all 128 columns)
  u32x4 v[2][NKS];  // V rows, this slice's columns only
};

template <int RT, int W, int DH, bool kStage, bool kPaged>
__global__ __launch_bounds__(W * kWave) void verify_attn_kernel(AttnArgs a) {
  constexpr int NH = kD / DH;      // d slices per unit
  constexpr int NDT = DH / 16;     // output 16-column tiles per wave
  constexpr int NVK = DH / 32;     // 32-column V chunks per row
  constexpr int kVPitch = DH + 8;  // LDS row pitch (bf16) of a wave's V tile
  constexpr int kQPitch = kD + 8;  // LDS row pitch (bf16) of the staged queries
  constexpr int kPitch = DH + 4;   // LDS row pitch (fp32) of the merged accumulator
  // One LDS arena: staged rows | V tiles | queries during the token loop, the merged
  // accumulator afterwards.
  constexpr int kStageBytes = kStage ? kStageSteps * 32 * 4 : 0;
  constexpr int kVBytes = W * 32 * kVPitch * 2;
  constexpr int kQBytes = RT * 16 * kQPitch * 2;
  constexpr int kLoopBytes = kStageBytes + kVBytes + kQBytes;
  constexpr int kMergeBytes = RT * 16 * kPitch * 4;
  __shared__ __attribute__((aligned(16))) char smem[kLoopBytes > kMergeBytes ? kLoopBytes : kMergeBytes];
  uint32_t* const sm_phys = reinterpret_cast<uint32_t*>(smem);
  uint16_t* const sm_q = reinterpret_cast<uint16_t*>(smem + kStageBytes + kVBytes);
  float* const sm_acc = reinterpret_cast<float*>(smem);

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // wave-uniform
  const int lr = lane & 15, lg = lane >> 4;
  uint16_t* const vtile = reinterpret_cast<uint16_t*>(smem + kStageBytes) + wave * 32 * kVPitch;

  const int id = blockIdx.x, xcd = id & 7, slot = id >> 3;
  const int half = slot % NH;
  const int unit = (slot / NH) * 8 + xcd;
  if (unit >= a.splits * a.pairs) return;
  const int pair = unit % a.pairs, split = unit / a.pairs;
  const int b = pair / a.num_kv_heads, g = pair - b * a.num_kv_heads;
  const int dbase = half * DH;

  const int N = a.dims.len(b);
  const int T = a.dims.nq(b);
  if (T == 0) return;
  const int gi = a.groups == 1 ? 0 : g;
  int wstart = N;
  const int32_t* idx_row = nullptr;
  if (a.idx) {
    wstart = clampi(a.count[b * a.groups + gi], 0, a.dims.k_max);
    idx_row = a.idx + (int64_t)b * a.idx_sb + (int64_t)gi * a.idx_sg;
  }
  const int total = wstart + T;        // virtual tokens: selected (or all) then window
  const int rows = T * a.group_size;   // <= RT * 16 (checked on the host via nq_max)
  const int nsteps = (total + 31) >> 5;
  const int per_split = (nsteps + a.splits - 1) / a.splits;
  const int s_begin = split * per_split;
  const int s_end = min(nsteps, s_begin + per_split);

  // Rows are addressed as uniform base + 32-bit byte offset phys * stride_n (the host
  // checks that every offset fits): phys is the position (contiguous) or
  // page * page_size + slot (paged, pages laid out back to back).
  const char* kbase = reinterpret_cast<const char*>(
      a.k.data + (kPaged ? 0 : (int64_t)b * a.k.stride_b) + (int64_t)g * a.k.stride_h);
  const char* vbase = reinterpret_cast<const char*>(
      a.v.data + (kPaged ? 0 : (int64_t)b * a.v.stride_b) + (int64_t)g * a.v.stride_h + dbase);
  const uint32_t kstride = (uint32_t)a.k.stride_n * 2u, vstride = (uint32_t)a.v.stride_n * 2u;

  // physical row of virtual token v (clamped into the cache; past-the-end -> row 0)
  auto phys_of = [&](int v) -> uint32_t {
    int64_t pos;
    if (v < wstart) pos = idx_row ? (int64_t)idx_row[v] : (int64_t)v;
    else if (v < total) pos = (int64_t)N + (v - wstart);
    else pos = 0;
    pos = pos < 0 ? 0 : (pos >= a.k.capacity ? a.k.capacity - 1 : pos);
    if constexpr (kPaged) {
      const int page = clampi(a.k.page_table[(int64_t)b * a.k.max_pages + (pos >> a.k.page_shift)], 0,
                              a.k.num_pages - 1);
      return ((uint32_t)page << a.k.page_shift) | (uint32_t)(pos & ((1 << a.k.page_shift) - 1));
    } else {
      return (uint32_t)pos;
    }
  };

  // Q^T as B operands: lane holds Q[row rt*16+lr][32 ks + 8 lg + e] (row r = t G + hh).
  // They are staged in LDS and read per step (16-byte reads), which keeps the VGPRs for
  // the in-flight K/V rows.
  constexpr bool kQLds = true;
  bf16x8 qreg[kQLds ? 1 : RT][4];
  int limit[RT];  // token v is visible to this lane's row iff v <= limit
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = rt * 16 + lr;
    limit[rt] = wstart + (r < rows ? r / a.group_size : T - 1);
  }
  auto q_row_ptr = [&](int r) {
    const int t = r / a.group_size, hh = r - t * a.group_size;
    return a.q + (int64_t)b * a.q_sb + (int64_t)t * a.q_st + (int64_t)(g * a.group_size + hh) * a.q_sh;
  };
  if constexpr (kQLds) {
    for (int u = threadIdx.x; u < RT * 16 * (kD / 8); u += W * kWave) {
      const int r = u / (kD / 8), c0 = (u % (kD / 8)) * 8;
      const u32x4 x = r < rows ? load16(q_row_ptr(r) + c0) : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(sm_q + r * kQPitch + c0) = x;
    }
  } else {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = rt * 16 + lr;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        qreg[rt][ks] = r < rows ? as_bf16x8(load16(q_row_ptr(r) + 8 * lg + 32 * ks))
                                : as_bf16x8(u32x4{0u, 0u, 0u, 0u});
    }
  }
  auto q_operand = [&](int rt, int ks) -> bf16x8 {
    if constexpr (kQLds)
      return as_bf16x8(*reinterpret_cast<const u32x4*>(sm_q + (rt * 16 + lr) * kQPitch + 8 * lg + 32 * ks));
    else
      return qreg[rt][ks];
  };

  // A operand of ones: one MFMA per row tile sums the bf16 probabilities of a step, so the
  // softmax denominator is formed from exactly the values the PV product uses.
  const bf16x8 ones = as_bf16x8(u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});

  float m_ref[RT];
  f32x4 acc[RT][NDT], accl[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    m_ref[rt] = -INFINITY;
    accl[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) acc[rt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  int chunk_v0 = 0;  // first virtual token staged in sm_phys

  // K rows of both tiles first, then V rows: the score MFMAs wait for K only.
  auto issue = [&](int st, StepRegs<NVK>& R) {
    uint32_t phys[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int v = (st << 5) + 16 * i + lr;
      if constexpr (kStage) phys[i] = sm_phys[v - chunk_v0];
      else phys[i] = v < total ? (uint32_t)v : 0u;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint16_t* kp = reinterpret_cast<const uint16_t*>(kbase + phys[i] * kstride) + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) R.k[i][ks] = load16(kp + 32 * ks);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint16_t* vp = reinterpret_cast<const uint16_t*>(vbase + phys[i] * vstride) + 8 * lg;
#pragma unroll
      for (int kv = 0; kv < NVK; ++kv) R.v[i][kv] = load16(vp + 32 * kv);
    }
  };

  // One 32-token step: V rows to this wave's LDS tile; (1) the score tiles of every 16-row
  // tile; (2) the softmax of each (one wave-uniform decision to move the reference maxima);
  // (3) per 16-column tile of V, its transposed operand read back with the LDS transpose
  // load and applied to every row tile.  Scores stay in raw units until one FMA forms
  // (s * scale * log2 e - m) inside exp2; the reference max m is in scaled units.
  auto compute = [&](int st, const StepRegs<NVK>& R) {
    const int v0 = st << 5;
    const bool edge = v0 + 31 >= wstart;  // wave-uniform: masking only near the window
    // (1) S^T tiles: lane holds tokens v0 + 16 i + 4 lg + e for query row rt*16 + lr
    f32x4 sc[RT][2];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) c = mfma16x16x32(as_bf16x8(R.k[i][ks]), q_operand(rt, ks), c);
        sc[rt][i] = c;
      }
    // V rows of the step into this wave's LDS tile (read back transposed in (3))
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int kv = 0; kv < NVK; ++kv)
        *reinterpret_cast<u32x4*>(vtile + (16 * i + lr) * kVPitch + 32 * kv + 8 * lg) = R.v[i][kv];
    // (2) masked row maxima, lazy rescale, probabilities
    float mx[RT];
    bool grow = false;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      if (edge) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (v0 + 16 * i + 4 * lg + e > limit[rt]) sc[rt][i][e] = -INFINITY;
      }
      const float m = fmaxf(fmaxf(fmaxf(sc[rt][0][0], sc[rt][0][1]), fmaxf(sc[rt][0][2], sc[rt][0][3])),
                            fmaxf(fmaxf(sc[rt][1][0], sc[rt][1][1]), fmaxf(sc[rt][1][2], sc[rt][1][3])));
      mx[rt] = max_over_lane_groups(m) * a.scale_log2;
      grow |= mx[rt] > m_ref[rt] + kRescaleLog2;
    }
    if (__any(grow)) {  // wave-uniform, rare after the first step
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const float mn = fmaxf(m_ref[rt], mx[rt]);
        const float alpha = m_ref[rt] == -INFINITY ? 0.f : fast_exp2(m_ref[rt] - mn);
        m_ref[rt] = mn;
        accl[rt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[rt][dt] *= alpha;
      }
    }
    bf16x8 pT[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const float nmu = m_ref[rt] == -INFINITY ? 0.f : -m_ref[rt];
      float p[2][4];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) p[i][e] = fast_exp2(fmaf(sc[rt][i][e], a.scale_log2, nmu));
      // B operand of the PV product: k slot 8 lg + e <-> token 4 lg + e (e < 4, tile 0)
      // and token 16 + 4 lg + e - 4 (e >= 4, tile 1)
      pT[rt] = as_bf16x8(u32x4{cvt_pk_bf16(p[0][0], p[0][1]), cvt_pk_bf16(p[0][2], p[0][3]),
                               cvt_pk_bf16(p[1][0], p[1][1]), cvt_pk_bf16(p[1][2], p[1][3])});
      accl[rt] = mfma16x16x32(ones, pT[rt], accl[rt]);
    }
    // (3) V^T A operand of column tile dt via the LDS transpose load: in each 16-lane
    // group, lane j points at row 4 lg + j / 4 (+16 for tile 1), columns 16 dt + 4 (j % 4);
    // lane lr then receives V[token 4 lg + e (+16)][16 dt + lr], e = 0..3.
    const uint16_t* trow = vtile + (4 * lg + (lr >> 2)) * kVPitch + 4 * (lr & 3);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const v4i16 lo = lds_read_tr16(trow + 16 * dt);
      const v4i16 hi = lds_read_tr16(trow + 16 * kVPitch + 16 * dt);
      const bf16x8 vt = as_bf16x8(u32x4{__builtin_bit_cast(u32x2, lo)[0], __builtin_bit_cast(u32x2, lo)[1],
                                        __builtin_bit_cast(u32x2, hi)[0], __builtin_bit_cast(u32x2, hi)[1]});
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt][dt] = mfma16x16x32(vt, pT[rt], acc[rt][dt]);
    }
  };

  // Ring of kDepth + 1 register buffers: step i + kDepth is issued before step i is
  // computed.  Issues past this wave's last step repeat that step (an L2 hit), so every
  // compute is preceded by exactly kDepth younger steps and waits for its own loads only.
  StepRegs<NVK> R[kDepth + 1];
  for (int cs = s_begin; cs < s_end; cs += kStageSteps) {
    const int ce = min(s_end, cs + kStageSteps);
    if constexpr (kStage) {
      __syncthreads();  // the previous chunk's rows are no longer read
      chunk_v0 = cs << 5;
      for (int v = chunk_v0 + threadIdx.x; v < (ce << 5); v += W * kWave) sm_phys[v - chunk_v0] = phys_of(v);
    }
    __syncthreads();  // staged rows (and staged queries) are visible
    const int first = cs + wave;
    const int nw = first < ce ? (ce - first + W - 1) / W : 0;  // this wave's steps: first + i W
    if (nw == 0) continue;
    auto step = [&](int i) { return first + min(i, nw - 1) * W; };
#pragma unroll
    for (int j = 0; j < kDepth; ++j) issue(step(j), R[j]);
    int i = 0;
    bool more = true;
    while (more) {
#pragma unroll
      for (int j = 0; j <= kDepth; ++j) {
        issue(step(i + kDepth), R[(j + kDepth) % (kDepth + 1)]);
        // keep the prefetch ahead of every wait of this step's compute
        __builtin_amdgcn_sched_barrier(0);
        compute(step(i), R[j]);
        if (++i == nw) {
          more = false;
          break;
        }
      }
    }
  }

  // ---- merge the W waves (fixed order: deterministic) ----
  __shared__ float sm_m[W][RT * 16];
  __shared__ float sm_l[W][RT * 16];
  __shared__ float sm_ML[2][RT * 16];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    if (lg == 0) {
      sm_m[wave][rt * 16 + lr] = m_ref[rt];
      sm_l[wave][rt * 16 + lr] = accl[rt][0];
    }
  }
  __syncthreads();
  float fac[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = rt * 16 + lr;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < W; ++w) M = fmaxf(M, sm_m[w][r]);
    const float Mu = M == -INFINITY ? 0.f : M;
    fac[rt] = m_ref[rt] == -INFINITY ? 0.f : fast_exp2(m_ref[rt] - Mu);
    if (wave == 0 && lg == 0) {
      float L = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w)
        L += sm_m[w][r] == -INFINITY ? 0.f : sm_l[w][r] * fast_exp2(sm_m[w][r] - Mu);
      sm_ML[0][r] = M;
      sm_ML[1][r] = L;
    }
  }
#pragma unroll 1
  for (int w = 0; w < W; ++w) {
    if (wave == w) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          float* dst = sm_acc + (rt * 16 + lr) * kPitch + 16 * dt + 4 * lg;
          const f32x4 val = acc[rt][dt] * fac[rt];
          if (w == 0) *reinterpret_cast<f32x4*>(dst) = val;
          else *reinterpret_cast<f32x4*>(dst) = *reinterpret_cast<f32x4*>(dst) + val;
        }
    }
    __syncthreads();
  }

  const int nthreads = W * kWave;
  if (a.splits == 1) {
    for (int u = threadIdx.x; u < rows * (DH / 8); u += nthreads) {
      const int r = u / (DH / 8), c0 = (u % (DH / 8)) * 8;
      const int t = r / a.group_size, hh = r - t * a.group_size;
      const float L = sm_ML[1][r];
      const float inv = L > 0.f ? 1.f / L : 0.f;
      const float* src = sm_acc + r * kPitch + c0;
      u32x4 o;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) o[e2] = cvt_pk_bf16(src[2 * e2] * inv, src[2 * e2 + 1] * inv);
      uint16_t* op = a.out + (int64_t)b * a.o_sb + (int64_t)t * a.o_st +
                     (int64_t)(g * a.group_size + hh) * a.o_sh + dbase + c0;
      *reinterpret_cast<u32x4*>(op) = o;
    }
    return;
  }
  // several token splits: publish this split's partial; verify_attn_combine merges them
  const int64_t prow = ((int64_t)pair * a.splits + split) * a.rows_pad;
  for (int u = threadIdx.x; u < rows * (DH / 4); u += nthreads) {
    const int r = u / (DH / 4), c0 = (u % (DH / 4)) * 4;
    *reinterpret_cast<f32x4*>(a.part_acc + (prow + r) * kD + dbase + c0) =
        *reinterpret_cast<const f32x4*>(sm_acc + r * kPitch + c0);
  }
  if (half == 0)
    for (int r = threadIdx.x; r < rows; r += nthreads) {
      a.part_ml[(prow + r) * 2] = sm_ML[0][r];
      a.part_ml[(prow + r) * 2 + 1] = sm_ML[1][r];
    }
}

// Merges the token splits of every (b, g): one workgroup per unit, fixed split order.
__global__ __launch_bounds__(256) void verify_attn_combine(AttnArgs a) {
  const int pair = blockIdx.x;
  const int b = pair / a.num_kv_heads, g = pair - b * a.num_kv_heads;
  const int T = a.dims.nq(b);
  const int rows = T * a.group_size;
  const int64_t base = (int64_t)pair * a.splits * a.rows_pad;
  extern __shared__ float fac[];  // [splits][rows_pad]
  for (int r = threadIdx.x; r < rows; r += blockDim.x) {
    float M = -INFINITY;
    for (int sp = 0; sp < a.splits; ++sp) M = fmaxf(M, a.part_ml[(base + (int64_t)sp * a.rows_pad + r) * 2]);
    const float Mu = M == -INFINITY ? 0.f : M;
    float L = 0.f;
    for (int sp = 0; sp < a.splits; ++sp) {
      const float* ml = a.part_ml + (base + (int64_t)sp * a.rows_pad + r) * 2;
      const float f = ml[0] == -INFINITY ? 0.f : exp2f(ml[0] - Mu);
      fac[sp * a.rows_pad + r] = f;
      L += ml[1] * f;
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    for (int sp = 0; sp < a.splits; ++sp) fac[sp * a.rows_pad + r] *= inv;
  }
  __syncthreads();
  for (int u = threadIdx.x; u < rows * (kD / 8); u += blockDim.x) {
    const int r = u / (kD / 8), c0 = (u % (kD / 8)) * 8;
    float o8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < a.splits; ++sp) {
      const float f = fac[sp * a.rows_pad + r];
      const float* src = a.part_acc + (base + (int64_t)sp * a.rows_pad + r) * kD + c0;
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(src);
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(src + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o8[e] += f * x0[e];
        o8[4 + e] += f * x1[e];
      }
    }
    const int t = r / a.group_size, hh = r - t * a.group_size;
    u32x4 o;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) o[e2] = cvt_pk_bf16(o8[2 * e2], o8[2 * e2 + 1]);
    uint16_t* op = a.out + (int64_t)b * a.o_sb + (int64_t)t * a.o_st +
                   (int64_t)(g * a.group_size + hh) * a.o_sh + c0;
    *reinterpret_cast<u32x4*>(op) = o;
  }
}

// ------------------------------------------------------------------------- host side

template <int RT, int W, int DH, bool kStage, bool kPaged>
static hipError_t launch_rt(const AttnArgs& a, hipStream_t stream) {
  constexpr int NH = kD / DH;
  const int units = a.splits * a.pairs;
  const int blocks = ((units + 7) / 8) * 8 * NH;
  hipLaunchKernelGGL((verify_attn_kernel<RT, W, DH, kStage, kPaged>), dim3(blocks), dim3(W * kWave), 0,
                     stream, a);
  return hipGetLastError();
}

template <int DH, bool kStage, bool kPaged>
static hipError_t launch_kind(const AttnArgs& a, int rt, hipStream_t stream) {
  constexpr int W = kAttnWavesPerGroup;
  switch (rt) {
    case 1: return launch_rt<1, W, DH, kStage, kPaged>(a, stream);
    case 2: return launch_rt<2, W, DH, kStage, kPaged>(a, stream);
    case 3: return launch_rt<3, W, DH, kStage, kPaged>(a, stream);
    case 4: return launch_rt<4, W, DH, kStage, kPaged>(a, stream);
    case 5: return launch_rt<5, W, DH, kStage, kPaged>(a, stream);
    case 6: return launch_rt<6, W, DH, kStage, kPaged>(a, stream);
    case 7:
    case 8: return launch_rt<8, W, DH, kStage, kPaged>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_verify_attn(const AttnArgs& a, int rt, int slices, bool sparse, bool paged,
                              hipStream_t stream) {
  const bool stage = sparse || paged;
  hipError_t e;
  if (slices == 2) {
    if (paged) e = launch_kind<64, true, true>(a, rt, stream);
    else if (stage) e = launch_kind<64, true, false>(a, rt, stream);
    else e = launch_kind<64, false, false>(a, rt, stream);
  } else {
    if (paged) e = launch_kind<128, true, true>(a, rt, stream);
    else if (stage) e = launch_kind<128, true, false>(a, rt, stream);
    else e = launch_kind<128, false, false>(a, rt, stream);
  }
  if (e != hipSuccess || a.splits == 1) return e;
  hipLaunchKernelGGL(verify_attn_combine, dim3(a.pairs), dim3(256),
                     (size_t)a.splits * a.rows_pad * sizeof(float), stream, a);
  return hipGetLastError();
}

}  // namespace dustin
