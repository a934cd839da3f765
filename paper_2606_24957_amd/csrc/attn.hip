// attn.hip -- verification attention for gfx950: sparse (gathered selected positions)
// and dense (every committed position), both followed by the causal verification window.
//
// Work decomposition
//   grid  (split, kv head g, sequence b); a workgroup of W waves owns one split of the
//         token list of (b, g).  All T_b * (Hq / Hkv) query rows of the KV head (the GQA
//         group of every verification token) share each K/V row that is read, so every
//         selected row is read from HBM exactly once per layer.
//   wave  walks the split in 32-token steps (waves interleave steps).  Per step:
//           S^T[32 tok x rows] = K[32 x 128] Q^T     MFMA 16x16x32, K rows loaded straight
//                                                    into A-operand registers (16 B/lane)
//           online softmax over tokens, fp32, exp2 domain
//           V^T via an identity MFMA                 puts 4 tokens of one d column in a
//                                                    lane, the layout the PV MFMA wants,
//                                                    with no LDS round trip
//           O^T[128 x rows] += V^T P^T               MFMA 16x16x32
//   merge the W waves' (max, sum, acc) through LDS in a fixed order (deterministic), then
//         either write bf16 output (one split) or write a partial and let the last split
//         to finish combine all partials (counter per (b, g), reset by that split).
#include "kernels.hpp"

namespace dustin {



constexpr int kD = 128;
constexpr int kAccStride = kD + 4;  // LDS row pitch (floats) of the merged accumulator

template <int RT, int W, bool kSparse, bool kPaged>
__global__ __launch_bounds__(W * kWave) void verify_attn_kernel(AttnArgs a) {
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int lr = lane & 15, lg = lane >> 4;

  const int N = a.dims.len(b);
  const int T = a.dims.nq(b);
  if (T == 0) return;  // the same for every split of (b, g): no counter is touched
  const int gi = a.groups == 1 ? 0 : g;
  int wstart;
  const int32_t* idx_row = nullptr;
  if constexpr (kSparse) {
    wstart = clampi(a.count[b * a.groups + gi], 0, a.dims.k_max);
    idx_row = a.idx + (int64_t)b * a.idx_sb + (int64_t)gi * a.idx_sg;
  } else {
    wstart = N;
  }
  const int total = wstart + T;          // virtual tokens: selected (or all) then window
  const int rows = T * a.group_size;     // <= RT * 16 (checked on the host via nq_max)
  const int nsteps = (total + 31) >> 5;
  const int per_split = (nsteps + a.splits - 1) / a.splits;
  const int s_begin = split * per_split;
  const int s_end = min(nsteps, s_begin + per_split);

  // Q^T as B operands: lane holds Q[row rt*16+lr][32 ks + 8 lg + e]
  bf16x8 qb[RT][4];
  int limit[RT];  // token v is visible to this lane's row iff v <= limit
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = rt * 16 + lr;
    const int t = r < rows ? r / a.group_size : T - 1;
    limit[rt] = wstart + t;
    if (r < rows) {
      const int hh = r - t * a.group_size;
      const uint16_t* qp = a.q + (int64_t)b * a.q_sb + (int64_t)t * a.q_st +
                           (int64_t)(g * a.group_size + hh) * a.q_sh + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) qb[rt][ks] = as_bf16x8(load16(qp + 32 * ks));
    } else {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) qb[rt][ks] = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
    }
  }

  // Identity B operands: column j of block hh picks k = 16 hh + j.
  bf16x8 ident[2];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    u32x4 u;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const int k0 = 8 * lg + 2 * e2;
      const uint32_t lo = (k0 == 16 * hh + lr) ? 0x3f80u : 0u;
      const uint32_t hi = (k0 + 1 == 16 * hh + lr) ? 0x3f80u : 0u;
      u[e2] = lo | (hi << 16);
    }
    ident[hh] = as_bf16x8(u);
  }

  float m_run[RT], l_run[RT];
  f32x4 acc[RT][8];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    m_run[rt] = -INFINITY;
    l_run[rt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[rt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int st = s_begin + wave; st < s_end; st += W) {
    const int v0 = st << 5;
    u32x4 kr[2][4], vr[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int vt = v0 + 16 * i + lr;
      int64_t pos;
      if (vt < wstart) pos = kSparse ? (int64_t)idx_row[vt] : (int64_t)vt;
      else if (vt < total) pos = (int64_t)N + (vt - wstart);
      else pos = 0;  // past the end: loaded, then masked
      const uint16_t* kp = a.k.row<kPaged>(b, pos, g) + 8 * lg;
      const uint16_t* vp = a.v.row<kPaged>(b, pos, g) + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        kr[i][ks] = load16(kp + 32 * ks);
        vr[i][ks] = load16(vp + 32 * ks);
      }
    }

    // S^T tiles: lane holds tokens v0 + 16 i + 4 lg + e for query row rt*16 + lr
    f32x4 s[2][RT];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) c = mfma16x16x32(as_bf16x8(kr[i][ks]), qb[rt][ks], c);
        s[i][rt] = c;
      }

    bf16x8 pT[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int vt = v0 + 16 * i + 4 * lg + e;
          const float x = vt <= limit[rt] ? s[i][rt][e] * a.scale_log2 : -INFINITY;
          s[i][rt][e] = x;
          mx = fmaxf(mx, x);
        }
      mx = max_over_lane_groups(mx);
      const float m_new = fmaxf(m_run[rt], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = exp2f(m_run[rt] - m_use);
      m_run[rt] = m_new;
      uint32_t pb[2][4];
      float lsum = 0.f;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pb[i][e] = bf16_rne_bits(exp2f(s[i][rt][e] - m_use));
          lsum += bf16_bits_to_float(pb[i][e]);
        }
      l_run[rt] = l_run[rt] * alpha + lsum;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) acc[rt][dt] *= alpha;
      // B operand of the PV product: k slot 8 lg + e <-> token 4 lg + e (e < 4, tile 0)
      // and token 16 + 4 lg + e - 4 (e >= 4, tile 1)
      pT[rt] = as_bf16x8(u32x4{pb[0][0] | (pb[0][1] << 16), pb[0][2] | (pb[0][3] << 16),
                               pb[1][0] | (pb[1][1] << 16), pb[1][2] | (pb[1][3] << 16)});
    }

    // V^T A operands: lane holds V[token(k slot 8 lg + e)][16 dt + lr]
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        const f32x4 d0 = mfma16x16x32(as_bf16x8(vr[0][ks]), ident[hh], z);
        const f32x4 d1 = mfma16x16x32(as_bf16x8(vr[1][ks]), ident[hh], z);
        const bf16x8 vtile = as_bf16x8(u32x4{pack_exact_bf16(d0[0], d0[1]), pack_exact_bf16(d0[2], d0[3]),
                                             pack_exact_bf16(d1[0], d1[1]), pack_exact_bf16(d1[2], d1[3])});
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          acc[rt][2 * ks + hh] = mfma16x16x32(vtile, pT[rt], acc[rt][2 * ks + hh]);
      }
  }

  // ---- merge the W waves of this split (fixed order: deterministic) ----
  __shared__ float sm_m[W][RT * 16];
  __shared__ float sm_l[W][RT * 16];
  __shared__ float sm_acc[RT * 16 * kAccStride];
  __shared__ float sm_ML[2][RT * 16];
  __shared__ int sm_last;

#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    l_run[rt] = sum_over_lane_groups(l_run[rt]);
    if (lg == 0) {
      sm_m[wave][rt * 16 + lr] = m_run[rt];
      sm_l[wave][rt * 16 + lr] = l_run[rt];
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
    const float M_use = M == -INFINITY ? 0.f : M;
    fac[rt] = exp2f(m_run[rt] - M_use);
    if (wave == 0 && lg == 0) {
      float L = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w) L += sm_l[w][r] * exp2f(sm_m[w][r] - M_use);
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
        for (int dt = 0; dt < 8; ++dt) {
          float* dst = sm_acc + (rt * 16 + lr) * kAccStride + 16 * dt + 4 * lg;
          const f32x4 val = acc[rt][dt] * fac[rt];
          if (w == 0) {
            *reinterpret_cast<f32x4*>(dst) = val;
          } else {
            *reinterpret_cast<f32x4*>(dst) = *reinterpret_cast<f32x4*>(dst) + val;
          }
        }
    }
    __syncthreads();
  }

  const int nthreads = W * kWave;
  if (a.splits == 1) {
    // normalise and store bf16: each thread writes 8 consecutive d (16 bytes)
    for (int u = threadIdx.x; u < rows * (kD / 8); u += nthreads) {
      const int r = u / (kD / 8), d0 = (u % (kD / 8)) * 8;
      const int t = r / a.group_size, hh = r - t * a.group_size;
      const float L = sm_ML[1][r];
      const float inv = L > 0.f ? 1.f / L : 0.f;
      const float* src = sm_acc + r * kAccStride + d0;
      u32x4 o;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2)
        o[e2] = bf16_rne_bits(src[2 * e2] * inv) | (bf16_rne_bits(src[2 * e2 + 1] * inv) << 16);
      uint16_t* op = a.out + (int64_t)b * a.o_sb + (int64_t)t * a.o_st +
                     (int64_t)(g * a.group_size + hh) * a.o_sh + d0;
      *reinterpret_cast<u32x4*>(op) = o;
    }
    return;
  }

  // ---- several splits: publish this split's partial ----
  const int64_t pair = (int64_t)b * a.num_kv_heads + g;
  float* pacc = a.part_acc + ((pair * a.splits + split) * a.rows_pad) * kD;
  float* pml = a.part_ml + ((pair * a.splits + split) * a.rows_pad) * 2;
  for (int u = threadIdx.x; u < rows * (kD / 4); u += nthreads) {
    const int r = u / (kD / 4), d0 = (u % (kD / 4)) * 4;
    *reinterpret_cast<f32x4*>(pacc + r * kD + d0) =
        *reinterpret_cast<const f32x4*>(sm_acc + r * kAccStride + d0);
  }
  for (int r = threadIdx.x; r < rows; r += nthreads) {
    pml[2 * r] = sm_ML[0][r];
    pml[2 * r + 1] = sm_ML[1][r];
  }
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t prev = atomicAdd(a.counters + pair, 1u);
    sm_last = prev == (uint32_t)(a.splits - 1);
  }
  __syncthreads();
  if (!sm_last) return;
  __threadfence();

  // ---- last split of (b, g): combine every partial (fixed split order) ----
  const float* base_acc = a.part_acc + (pair * a.splits) * a.rows_pad * kD;
  const float* base_ml = a.part_ml + (pair * a.splits) * a.rows_pad * 2;
  float* fac_s = sm_acc;  // [splits][rows], reuses the merge buffer
  for (int r = threadIdx.x; r < rows; r += nthreads) {
    float M = -INFINITY;
    for (int sp = 0; sp < a.splits; ++sp) M = fmaxf(M, base_ml[(sp * a.rows_pad + r) * 2]);
    const float M_use = M == -INFINITY ? 0.f : M;
    float L = 0.f;
    for (int sp = 0; sp < a.splits; ++sp) {
      const float f = exp2f(base_ml[(sp * a.rows_pad + r) * 2] - M_use);
      fac_s[sp * rows + r] = f;
      L += base_ml[(sp * a.rows_pad + r) * 2 + 1] * f;
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    for (int sp = 0; sp < a.splits; ++sp) fac_s[sp * rows + r] *= inv;
  }
  __syncthreads();
  for (int u = threadIdx.x; u < rows * (kD / 8); u += nthreads) {
    const int r = u / (kD / 8), d0 = (u % (kD / 8)) * 8;
    float o8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < a.splits; ++sp) {
      const float f = fac_s[sp * rows + r];
      const float* src = base_acc + ((int64_t)sp * a.rows_pad + r) * kD + d0;
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
    for (int e2 = 0; e2 < 4; ++e2) o[e2] = bf16_rne_bits(o8[2 * e2]) | (bf16_rne_bits(o8[2 * e2 + 1]) << 16);
    uint16_t* op = a.out + (int64_t)b * a.o_sb + (int64_t)t * a.o_st +
                   (int64_t)(g * a.group_size + hh) * a.o_sh + d0;
    *reinterpret_cast<u32x4*>(op) = o;
  }
  if (threadIdx.x == 0) a.counters[pair] = 0u;  // ready for the next call on this workspace
}

// ------------------------------------------------------------------------- host side

template <int RT, int W, bool kSparse, bool kPaged>
static hipError_t launch_rt(const AttnArgs& a, int B, hipStream_t stream) {
  dim3 grid(a.splits, a.num_kv_heads, B);
  hipLaunchKernelGGL((verify_attn_kernel<RT, W, kSparse, kPaged>), grid, dim3(W * kWave), 0,
                     stream, a);
  return hipGetLastError();
}

template <bool kSparse, bool kPaged>
static hipError_t launch_kind(const AttnArgs& a, int rt, int B, hipStream_t stream) {
  constexpr int W = 4;
  switch (rt) {
    case 1: return launch_rt<1, W, kSparse, kPaged>(a, B, stream);
    case 2: return launch_rt<2, W, kSparse, kPaged>(a, B, stream);
    case 3: return launch_rt<3, W, kSparse, kPaged>(a, B, stream);
    case 4: return launch_rt<4, W, kSparse, kPaged>(a, B, stream);
    case 5: return launch_rt<5, W, kSparse, kPaged>(a, B, stream);
    case 6: return launch_rt<6, W, kSparse, kPaged>(a, B, stream);
    case 7:
    case 8: return launch_rt<8, W, kSparse, kPaged>(a, B, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_verify_attn(const AttnArgs& a, int rt, int B, bool sparse, bool paged,
                              hipStream_t stream) {
  if (sparse) return paged ? launch_kind<true, true>(a, rt, B, stream) : launch_kind<true, false>(a, rt, B, stream);
  return paged ? launch_kind<false, true>(a, rt, B, stream) : launch_kind<false, false>(a, rt, B, stream);
}

}  // namespace dustin
