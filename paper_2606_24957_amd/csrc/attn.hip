// attn.hip -- verification attention for gfx950: sparse (gathered selected positions)
// and dense (every committed position), both followed by the causal verification window.
//
// Work decomposition
//   unit   (sequence b, KV head g, token split).  All T_b * (Hq / Hkv) query rows of the
//          KV head (its GQA group for every verification token) share each K/V row, so a
//          row is fetched from HBM exactly once per layer, and a workgroup produces all
//          128 output columns of its rows.  The token list is cut into as many splits as
//          it takes to put one workgroup on every CU; the splits of a unit get block ids
//          congruent mod 8 (one XCD) and the last one to finish merges them (below).
//   wave   walks 32-token steps of its workgroup's range (the four waves interleave
//          steps).  A step's K and V rows go straight from HBM into a wave-private LDS
//          tile with a gfx950 direct-to-LDS load (buffer_load_dwordx4 ... lds, or
//          global_load_lds_dwordx4; see load_lds16): every load instruction moves four
//          whole 256-byte rows, and no VGPR holds data in flight.
//          The chunks of a row are XOR-swizzled so that the MFMA operand reads below are
//          free of bank conflicts.  Per step:
//            wait for the step's rows, read K (MFMA A layout) and V^T (LDS transpose
//            load) into registers, start the next step's loads, then
//            S^T[32 tok x rows] = K[32 x 128] Q^T     MFMA 16x16x32 bf16
//            online softmax over tokens (fp32, exp2 domain); the running max only moves
//            when a row's max grows by more than 2^8, a wave-uniform event, so the
//            accumulator is rarely rescaled
//            O^T[128 x rows] += V^T P^T               MFMA 16x16x32; a ones tile gives
//                                                     the row sums of the same bf16 P
//          so each wave keeps exactly one step (16 KB) in flight while it computes.
//   merge  the waves' (max, sum, acc) combine through LDS in a fixed order.  With one
//          split the workgroup writes the normalised output.  Otherwise it publishes its
//          partial with write-through (agent-scope) stores, waits for them to complete,
//          and counts itself in with an atomic add on the unit's counter; the workgroup
//          that arrives last reads the other partials back with agent-scope loads,
//          merges all of them in split order (deterministic whichever arrives last),
//          writes the output and returns the counter to zero.  No workgroup waits for
//          another and no cache is flushed.
//
// Gathered positions (sparse) and page translations (paged) are resolved into an LDS table
// of physical rows before the token loop, so the loop does no dependent global loads.
#include <type_traits>

#include "kernels.hpp"

namespace dustin {

constexpr int kD = 128;
constexpr int kW = 4;                  // waves per workgroup: one per SIMD
constexpr int kStep = 32;              // tokens per wave step
constexpr int kTile = kStep * kD * 2;  // bytes of one step's K (or V) rows: 8 KB
constexpr int kStageBatch = 8;         // staged positions per thread per chunk
constexpr int kStageSteps = kW * kWave * kStageBatch / 32;  // steps staged per chunk (64)
constexpr float kRescaleLog2 = 8.f;    // lazy rescale threshold (factor 256)


typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

// gfx950 LDS transpose load: within each 16-lane group, lane i receives element i % 4 of
// the 8 bytes addressed by group lane 4 e + i / 4, for e = 0..3.
__device__ __forceinline__ v4i16 lds_read_tr16(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(const_cast<char*>(p)));
}

// gfx950 direct-to-LDS loads: lane l's 16 bytes land at lds + 16 l.
// The buffer form (byte offset off into a resource; past its extent reads zeros) is not a
// FLAT instruction, so while such loads are in flight the compiler keeps counting loads in
// order and waits for an earlier ordinary load with a partial vmcnt; with global_load_lds
// in flight it waits with vmcnt(0).  Kernels that issue their first step speculatively use
// the buffer form throughout; the others keep the global form, which measured faster for
// them (and about 1% faster per launch in a plain full-chip gather, while the buffer form is
// faster for one CU alone).
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t rs, uint32_t off, char* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(lds), 16, (int)off, 0, 0, 0);
}
__device__ __forceinline__ void load_lds16(const char* base, uint32_t off, char* lds) {
  __builtin_amdgcn_global_load_lds(base + off, (lds_void*)(lds), 16, 0, 0);
}
// Resource over [base, base + bytes) (gfx9 raw buffer: stride 0, 32-bit data format)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t byte_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Workgroup barrier for hand-offs of ds_write data only.  It waits for the wave's LDS
// instructions but, unlike __syncthreads (whose fence also covers direct-to-LDS loads),
// not for its outstanding global loads: the wave's own loads of its next step keep flowing
// across it.  The empty asm statements keep the compiler from moving memory accesses
// across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt with only one counter constrained (gfx9 encoding; the others at their maxima)
__device__ __forceinline__ void wait_vmem_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)
__device__ __forceinline__ void wait_vmem_8() { __builtin_amdgcn_s_waitcnt(0x0F78); }    // vmcnt(8)
__device__ __forceinline__ void wait_lds_all() { __builtin_amdgcn_s_waitcnt(0xC07F); }   // lgkmcnt(0)

// Inclusive prefix sum over the 64 lanes of a wave: a Hillis-Steele scan inside each row of
// 16 lanes (DPP row shifts; lanes without a source add 0), then lane 15 of rows 0 and 2 is
// added to rows 1 and 3 (row_bcast:15) and lane 31 to rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ int wave_inclusive_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

// floor(a / b) for 0 <= a < 2^22 and 1 <= b < 2^22: the fp32 reciprocal estimate is within
// one of the quotient there, and one correction each way makes it exact.  The products
// checked, q b and (q + 1) b with q at most one above the quotient, stay below 2^23, so
// 24-bit multiplies are exact.  (A plain 32-bit multiply-add is lowered to a 64-bit
// multiply-add whose unused high addend can land in a register with a load still pending,
// and the wait for that load then stalls this arithmetic behind every earlier load.)
__device__ __forceinline__ int small_div(int a, int b) {
  int q = (int)((float)a * __builtin_amdgcn_rcpf((float)b));
  q -= (int)__umul24((unsigned)q, (unsigned)b) > a ? 1 : 0;
  q += (int)__umul24((unsigned)(q + 1), (unsigned)b) <= a ? 1 : 0;
  return q;
}

// Placement of a step's rows in a wave's 8 KB tile.  Load instruction i (0..7) fills LDS
// rows 4 i .. 4 i + 3 with tokens i, 8 + i, 16 + i, 24 + i (lanes 16 q .. 16 q + 15 move
// token 8 q + i), so token j of the step sits in LDS row 4 (j & 7) + (j >> 3).  Within a
// row, the 16-byte chunk c of K is stored at chunk c ^ (j & 15) and chunk c of V at
// c ^ 2 (j & 7): the 16 rows read by one MFMA operand load (K) and the four rows x eight
// half-chunks of one transpose load (V) then fall into distinct LDS banks.
__device__ __forceinline__ int tile_row(int j) { return 4 * (j & 7) + (j >> 3); }
__device__ __forceinline__ int k_chunk(int j, int c) { return c ^ (j & 15); }
__device__ __forceinline__ int v_chunk(int j, int c) { return c ^ ((j & 7) << 1); }

template <int RT, bool kSparse, bool kPaged, bool kQReg>
__global__ __launch_bounds__(kW * kWave) void verify_attn_kernel(AttnArgs a) {
  constexpr bool kStage = kSparse || kPaged;  // rows resolved through an LDS table
  constexpr int NDT = kD / 16;     // output 16-column tiles
  constexpr int kQPitch = kD + 8;  // LDS row pitch (bf16) of staged queries
  constexpr int kPitch = kD + 4;   // LDS row pitch (fp32) of the merged accumulator
  // Beyond four row tiles a wave over a contiguous cache waits for a step's K rows and its
  // V rows separately (the token loop below); the V tiles then form an LDS object of their
  // own, so that the compiler can tell the two tiles' direct-to-LDS loads apart.  (In the
  // paged kernels the compiler still waits for every load before the score tile's query
  // reads, which made the split form slower there.)
  constexpr bool kSplitKV = RT > 4 && !kPaged;
  constexpr int kTilesBytes = kW * (kSplitKV ? 1 : 2) * kTile;   // K (and V) tiles of every wave
  // The table of staged rows is an LDS object of its own up to three row tiles and beyond
  // four (then the compiler can tell that accessing it does not touch a tile whose rows are
  // in flight); at four it shares the tile area's object to leave LDS for the wave
  // accumulators.
  constexpr bool kOwnStage = kStage && (RT <= 3 || kSplitKV);
  constexpr int kStageBytes = kStage && !kOwnStage ? kStageSteps * kStep * 4 : 0;
  constexpr int kLoopBytes = kTilesBytes + kStageBytes;
  constexpr int kBufFloats = RT * 16 * kPitch;                  // one wave's accumulator
  constexpr int kNB = RT <= 4 ? kW : (RT <= (kSplitKV ? 5 : 6) ? 2 : 1);  // wave accumulators LDS holds
  constexpr int kFinalBytes = kNB * kBufFloats * 4;
  __shared__ __attribute__((aligned(1024))) char smem[kLoopBytes > kFinalBytes ? kLoopBytes : kFinalBytes];
  __shared__ __attribute__((aligned(16))) uint32_t sm_phys_own[kOwnStage ? kStageSteps * kStep : 4];
  uint32_t* const sm_phys = kOwnStage ? sm_phys_own : reinterpret_cast<uint32_t*>(smem + kTilesBytes);
  // The queries are loaded once per workgroup (each thread a few 16-byte chunks) and
  // staged in LDS; with up to three row tiles every wave then copies them to registers
  // after the staging barrier, else they are read from LDS at every step.  They live in an
  // LDS object of their own: the compiler can then see that the direct-to-LDS row loads in
  // flight never write them, and reads them without waiting for those loads.
  __shared__ __attribute__((aligned(16))) uint16_t sm_q[RT * 16 * kQPitch];
  // The verification window's tokens as a step of their own (up to three row tiles): one
  // wave of the pair's last split loads them in the prologue, beside its first step, into
  // this tile (K then V, the same layout as the wave tiles), and computes them while that
  // step is in flight.  The selected tokens then fill whole 32-token steps, so a pair of
  // 2048 selected tokens takes 64 steps, 8 per wave over two splits, and no wave spends a
  // ninth load round trip on a step of a few window tokens.
  __shared__ __attribute__((aligned(1024))) char sm_win[2 * kTile];
  __shared__ uint32_t sm_wphys[kStep];  // paged: physical rows of the window's tokens

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // wave-uniform
  const int lr = lane & 15, lg = lane >> 4;
  __shared__ __attribute__((aligned(1024))) char sm_vtiles[kSplitKV ? kW * kTile : 16];
  char* const ktile = smem + wave * (kSplitKV ? 1 : 2) * kTile;
  char* const vtile = kSplitKV ? sm_vtiles + wave * kTile : ktile + kTile;
  // Every kernel argument the prologue reads is held in SGPRs from here on: the arguments
  // then arrive as one batch with one wait, instead of in dependent batches between the
  // first global loads.
  asm volatile("" ::"s"(a.q), "s"(a.q_sb), "s"(a.q_st), "s"(a.q_sh), "s"(a.idx), "s"(a.idx_sb),
               "s"(a.idx_sg), "s"(a.count), "s"(a.dims.seq_lens), "s"(a.dims.n_query),
               "s"(a.dims.max_len), "s"(a.dims.nq_max), "s"(a.dims.k_max), "s"(a.groups),
               "s"(a.num_kv_heads), "s"(a.group_size), "s"(a.pairs), "s"(a.splits),
               "s"(a.split_steps), "s"(a.min_split_steps));
  asm volatile("" ::"s"(a.k.data), "s"(a.k.stride_b), "s"(a.k.stride_n), "s"(a.k.stride_h),
               "s"(a.k.capacity), "s"(a.v.data), "s"(a.v.stride_b), "s"(a.v.stride_n), "s"(a.v.stride_h),
               "s"(a.out), "s"(a.counters), "s"(a.part_acc), "s"(a.part_ml), "s"(a.rows_pad),
               "s"(a.scale_log2));

  // ---- which (pair, split) this workgroup runs.  The grid holds U = pairs * splits unit
  // slots; XCD x (blockIdx % 8) runs units ceil(x A / 8) .. ceil((x + 1) A / 8) - 1 of the A
  // units there are, a contiguous run, so that the splits of a pair and the KV heads of a
  // sequence share an XCD (its L2 and its address translations).
  const int xcd = blockIdx.x & 7, xslot = blockIdx.x >> 3;
  const int U = a.pairs * a.splits;
  auto unit_of = [&](int A, int& unit) {
    unit = (xcd * A + 7) / 8 + xslot;
    return unit < ((xcd + 1) * A + 7) / 8;
  };
  // With one split per pair, unit = pair.  With several, every wave sizes the splits from
  // the actual per-pair token counts below.  Meanwhile the prologue loads of the uniform guess
  // (every pair `splits` splits of split_steps steps, exact when the lengths are equal) are
  // already in flight; they are issued again only if the guess was wrong.
  const bool balance = a.splits > 1;  // kernel-uniform
  int unit = 0;
  const bool guess_ok = unit_of(U, unit);
  int pair = guess_ok ? unit / a.splits : 0;
  int split = unit - pair * a.splits;
  int s_begin = split * a.split_steps;
  int split_steps = a.split_steps, nsplit = 1, slot0 = 0;

  // ---- prologue: one round trip.  The per-sequence sizes, the queries and the selected
  // positions of the first chunk are loaded together; the latter two speculatively (every
  // query slot, positions below k_max), which stays in bounds whatever the sizes are.
  int b = 0, g = 0, gi = 0;
  const int32_t* idx_row = nullptr;
  bool idx_vec = false;  // the index row is 16-byte aligned (wave-uniform)
  int n_raw = 0, t_raw = 0, c_raw = 0;
  const int rows_mem = a.dims.nq_max * a.group_size;  // query rows present in memory
  auto q_row_ptr = [&](int r) {
    const int t = small_div(r, a.group_size), hh = r - t * a.group_size;
    return a.q + (int64_t)b * a.q_sb + (int64_t)t * a.q_st + (int64_t)(g * a.group_size + hh) * a.q_sh;
  };
  // Q^T as B operands: lane holds Q[row rt*16+lr][32 ks + 8 lg + e] (row r = t G + hh),
  // in registers for up to 3 row tiles, else read from the LDS staging at every step.
  bf16x8 qreg[kQReg ? RT : 1][4];
  constexpr int kQChunks = RT * 16 * (kD / 8), kQPer = (kQChunks + kW * kWave - 1) / (kW * kWave);
  u32x4 qx[kQPer];
  // Entries v .. v + 7 of the index row (v a multiple of 8; entries from k_max on read the
  // last one): two 16-byte loads where the row is aligned and the eight are inside it.
  auto load_idx8 = [&](int v, int32_t (&dst)[8]) {
    if (idx_vec && v + 8 <= a.dims.k_max) {
      const u32x4 x0 = *reinterpret_cast<const u32x4*>(idx_row + v);
      const u32x4 x1 = *reinterpret_cast<const u32x4*>(idx_row + v + 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        dst[i] = (int32_t)x0[i];
        dst[4 + i] = (int32_t)x1[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) dst[i] = idx_row[min(v + i, a.dims.k_max - 1)];
    }
  };
  // selected positions of this thread's tokens in a chunk: tokens 8 t .. 8 t + 7 of it
  int32_t sel[kStageBatch];
  static_assert(kStageBatch == 8 && kStageSteps * kStep == 8 * kW * kWave, "staging layout");
  auto load_selection = [&](int cs) {
    if constexpr (kSparse) load_idx8(cs * kStep + 8 * (int)threadIdx.x, sel);
    else
#pragma unroll
      for (int j = 0; j < kStageBatch; ++j) sel[j] = 0;
  };
  // the positions of this lane's tokens in the wave's first step, so that its loads can
  // start before the block-wide staging pass (contiguous caches; a paged one needs the
  // staged translation)
  int first_v0 = 0;
  int32_t first_sel[8];
  int own_sizes = 0;  // lane 0: N_b, lane 1: T_b (if given), lane 2: the selection count
  auto locate = [&]() {
    b = pair / a.num_kv_heads;
    g = pair - b * a.num_kv_heads;
    gi = a.groups == 1 ? 0 : g;
    idx_row = kSparse ? a.idx + (int64_t)b * a.idx_sb + (int64_t)gi * a.idx_sg : nullptr;
    idx_vec = ((uintptr_t)idx_row & 15) == 0;
    first_v0 = (s_begin + wave) * kStep + 8 * lg;
  };
  // the first step's positions go first (contiguous caches): the first rows wait for them
  auto first_loads = [&]() {
    if constexpr (kStage && !kPaged) load_idx8(first_v0, first_sel);
  };
  auto prologue_loads = [&]() {
    // one gather by three lanes (read back lane by lane where first needed, so that no
    // wait for it lands among the loads below)
    {
      const int32_t* src = lane == 1 && a.dims.n_query ? a.dims.n_query + b
                           : lane == 2 && kSparse ? a.count + b * a.groups + gi
                           : a.dims.seq_lens + b;
      own_sizes = *src;
    }
    // Every query load is unconditional: a row past those in memory reads the last one,
    // and is zeroed with the rows of absent verification tokens when it is staged.
    // (Conditional loads made the compiler recompute the row address, a division and
    // 64-bit products, inside every load's branch.)
#pragma unroll
    for (int j = 0; j < kQPer; ++j) {
      const int e = min((int)threadIdx.x + j * kW * kWave, kQChunks - 1);
      const int r = e / (kD / 8), c0 = (e % (kD / 8)) * 8;
      qx[j] = load16(q_row_ptr(min(r, rows_mem - 1)) + c0);
    }
    if constexpr (kStage) load_selection(s_begin);
  };
  locate();
  if constexpr (kPaged) prologue_loads();
  else first_loads();
  // sizes of pairs 4 lane .. 4 lane + 3 (every wave).  With a contiguous cache they are
  // issued before the prologue loads, so that waiting for them leaves those in flight while
  // the schedule is planned; with a paged cache the positions go first, since they feed
  // the page-table lookups of the first rows (each order measured faster for its kind).
  // Buffer loads at 32-bit offsets computed up front: 64-bit address arithmetic between
  // the loads had the compiler reuse a register of a pending load, and the wait for it
  // (vmcnt(0)) held back the later loads until every earlier one had returned.
  // (unconditional loads: a lane past the last pair reads the last pair's sizes, which
  // count for nothing, see steps_of's callers)
  int pn[4], pt[4], pc[4];
  if (balance) {
    const int nb = small_div(a.pairs, a.num_kv_heads);  // the batch (pairs <= 256 here)
    int on[4], oc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int p = min(4 * lane + j, a.pairs - 1);
      const int pb = small_div(p, a.num_kv_heads), pg = p - pb * a.num_kv_heads;
      on[j] = pb * 4;
      oc[j] = (pb * a.groups + (a.groups == 1 ? 0 : pg)) * 4;
    }
    const auto rs_n = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(a.dims.seq_lens), 0, nb * 4, 0x00020000);
#pragma unroll
    for (int j = 0; j < 4; ++j) pn[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_n, on[j], 0, 0);
    if (a.dims.n_query) {  // kernel-uniform
      const auto rs_t = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(a.dims.n_query), 0, nb * 4, 0x00020000);
#pragma unroll
      for (int j = 0; j < 4; ++j) pt[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_t, on[j], 0, 0);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) pt[j] = a.dims.nq_max;
    }
    if constexpr (kSparse) {
      const auto rs_c = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(a.count), 0, nb * a.groups * 4,
                                                          0x00020000);
#pragma unroll
      for (int j = 0; j < 4; ++j) pc[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_c, oc[j], 0, 0);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) pc[j] = 0;
    }
  }
  if constexpr (!kPaged) prologue_loads();

  // Rows are addressed as uniform base + 32-bit byte offset phys * stride_n (the host
  // checks that every offset fits): phys is the position (contiguous) or
  // page * page_size + slot (paged, pages laid out back to back).  The loads go through
  // buffer resources over the pair's K and V rows, whose extent, (rows - 1) * stride +
  // 256 bytes, bounds every offset the kernel forms.
  const uint32_t kstride = (uint32_t)a.k.stride_n * 2u, vstride = (uint32_t)a.v.stride_n * 2u;
  auto extent = [&](int64_t nrows, uint32_t stride) -> uint32_t {
    const int64_t e = (nrows - 1) * (int64_t)stride + 256;
    return (uint32_t)(e < (int64_t)UINT32_MAX ? e : (int64_t)UINT32_MAX);
  };
  __amdgpu_buffer_rsrc_t krs, vrs;
  const char *kbase, *vbase;
  auto set_rows = [&]() {
    kbase = reinterpret_cast<const char*>(a.k.data + (kPaged ? 0 : (int64_t)b * a.k.stride_b) +
                                          (int64_t)g * a.k.stride_h);
    vbase = reinterpret_cast<const char*>(a.v.data + (kPaged ? 0 : (int64_t)b * a.v.stride_b) +
                                          (int64_t)g * a.v.stride_h);
    krs = byte_rsrc(kbase, extent(kPaged ? ((int64_t)a.k.num_pages << a.k.page_shift) : a.k.capacity, kstride));
    vrs = byte_rsrc(vbase, extent(kPaged ? ((int64_t)a.v.num_pages << a.v.page_shift) : a.v.capacity, vstride));
  };
  set_rows();
  // positions are 32-bit: N_b + T_b and the selected positions are int32 (a capacity
  // beyond that bound leaves every int32 position inside it)
  const int cap_m1 = (int)(a.k.capacity - 1 < INT32_MAX ? a.k.capacity - 1 : INT32_MAX - 1);

  // The K half and the V half of a step's loads alone (kernels that wait for K and V
  // separately; buffer form).
  auto issue_v_to = [&](const uint32_t (&ph)[8], char* vt, auto buffered) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int j = 8 * lg + i;
      if constexpr (decltype(buffered)::value) load_lds16(vrs, ph[i] * vstride + 16 * v_chunk(j, lr), vt + i * 1024);
      else load_lds16(vbase, ph[i] * vstride + 16 * v_chunk(j, lr), vt + i * 1024);
    }
  };
  auto issue_rows_to_k = [&](const uint32_t (&ph)[8], char* kt) {
#pragma unroll
    for (int i = 0; i < 8; ++i) load_lds16(krs, ph[i] * kstride + 16 * k_chunk(8 * lg + i, lr), kt + i * 1024);
  };
  // Loads of one step into a K and a V tile: this lane moves chunk lr of tokens 8 lg + i
  // (i = 0..7) of the step, whose physical rows are ph[i]; one instruction per i for K and
  // one for V.  Buffer loads in the prologue (see load_lds16), global ones in the loop.
  auto issue_rows_to = [&](const uint32_t (&ph)[8], char* kt, char* vt, auto buffered) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int j = 8 * lg + i;
      if constexpr (decltype(buffered)::value) {
        load_lds16(krs, ph[i] * kstride + 16 * k_chunk(j, lr), kt + i * 1024);
        if constexpr (!kSplitKV) load_lds16(vrs, ph[i] * vstride + 16 * v_chunk(j, lr), vt + i * 1024);
      } else {
        load_lds16(kbase, ph[i] * kstride + 16 * k_chunk(j, lr), kt + i * 1024);
        if constexpr (!kSplitKV) load_lds16(vbase, ph[i] * vstride + 16 * v_chunk(j, lr), vt + i * 1024);
      }
    }
    // split waits: the step's eight V loads follow its eight K loads
    if constexpr (kSplitKV) issue_v_to(ph, vt, buffered);
  };
  using Buffered = std::true_type;
  using Global = std::false_type;

  // With a contiguous cache every wave issues its first step before the split schedule
  // is known: the step of the guessed unit, from the positions it loaded first (the
  // selected ones, or the positions themselves when dense), clamped into the cache.  The
  // sizes, queries and row table then arrive and are staged while the step's rows are in
  // flight.  Those are the step's right rows: a sparse kernel here has a window step of
  // its own, so body tokens from the selection count on are masked, and a dense cache's
  // window positions follow its committed ones.  If the guess was wrong, the wave waits
  // for the rows to land and issues the step again.  The 16 loads are issued by every
  // wave, so that the same number of loads follows the queries and positions on every
  // path and the compiler can wait for them with a partial vmcnt.  (A paged cache needs
  // the staged page translations first, and beyond three row tiles the table shares the
  // tile area's LDS object: both issue the first step after staging, as do dense kernels
  // beyond four row tiles, where the extra live registers would spill.)
  constexpr bool kSpec = !kPaged && (kStage ? RT <= 3 : RT <= 4);
  static_assert(!kSpec || !kSparse || RT <= kAttnSepMaxRT, "speculative sparse rows need the window step");
  // the token loop's form: buffer loads where the first step is speculative, and where K and
  // V are waited for separately (the wait insertion counts FLAT loads as out of order)
  using LoopForm = std::integral_constant<bool, kSpec || kSplitKV>;
  auto issue_first = [&](auto exact_pos) {
    uint32_t ph[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if constexpr (kStage) ph[i] = (uint32_t)exact_pos(first_v0 + i, first_sel[i]);
      else ph[i] = (uint32_t)exact_pos(first_v0 + i, 0);
    }
    issue_rows_to(ph, ktile, vtile, Buffered{});
  };
  if constexpr (kSpec)
    issue_first([&](int v, int32_t selected) { return clampi(kStage ? (int)selected : v, 0, cap_m1); });
  bool relocate = false;  // the guess was wrong
  // a wave leaves only once its speculative rows have landed in its tile
  auto drain = [&]() {
    if constexpr (kSpec) wait_vmem_all();
  };

  // 32-token steps of a pair that the splits share: its selected (or all) positions, then
  // its window -- or, with a window step of its own, the positions alone (at least one step)
  // Row tiles up to which the window has a step of its own.  Beyond three the window tile
  // no longer fits beside four wave accumulators in LDS, and the second copy of the step
  // code makes the five-tile kernel spill.
  constexpr bool sep = RT <= kAttnSepMaxRT;
  auto steps_of = [&](int n, int t, int c) {
    const int Nc = clampi(n, 0, a.dims.max_len), Tc = clampi(t, 0, a.dims.nq_max);
    const int body = kSparse ? clampi(c, 0, a.dims.k_max) : Nc;
    if (Tc == 0) return 0;
    return sep ? max(1, (body + kStep - 1) / kStep) : (body + Tc + kStep - 1) / kStep;
  };
  if (balance) {
    // The smallest split size s (at least min_split_steps) whose splits fit the U slots:
    // pair p takes ceil(steps_p / s) splits of equal size.  s = ceil(W / U) (W = total steps)
    // fits when the lengths are equal; otherwise a binary search up to ceil(W / (U - pairs)),
    // which always fits (sum ceil(steps_p / s) <= W / s + pairs).  Every wave plans the same
    // schedule from the same sizes, so no wave waits for another here.
    int st[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) st[j] = 4 * lane + j < a.pairs ? steps_of(pn[j], pt[j], pc[j]) : 0;
    // k = ceil(x / s) splits of size ceil(x / k).  None of them is empty: with that size
    // ceil(x / size) = k again (size <= s gives x / size >= x / s, and size >= x / k gives
    // x / size <= k).
    auto splits_for = [](int x, int s, int& size) {
      const int k0 = x ? small_div(x + s - 1, s) : 0;
      size = k0 ? small_div(x + k0 - 1, k0) : 0;
      return k0;
    };
    const int st0 = __builtin_amdgcn_readfirstlane(st[0]);
    bool differs = false;
#pragma unroll
    for (int j = 0; j < 4; ++j) differs |= 4 * lane + j < a.pairs && st[j] != st0;
    int p_new = -1, split_new = 0;
    if (!__any(differs)) {
      // equal lengths (the common case): every pair takes the same splits, no scan
      int sz0;
      const int k = splits_for(st0, max(small_div(st0 + a.splits - 1, a.splits), a.min_split_steps), sz0);
      int my = 0;
      if (k && unit_of(a.pairs * k, my)) {
        p_new = small_div(my, k);
        split_new = my - p_new * k;
        nsplit = k;
        split_steps = sz0;
        slot0 = p_new * k;
      }
    } else {
      int kk[4], sz[4], start[4];
      int loc = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) loc += st[j];
      const int W = __builtin_amdgcn_readlane(wave_inclusive_sum(loc), 63);
      // the number of units split size s needs (one division per pair: the search's probe)
      auto units_for = [&](int s) {
        int tot = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) tot += st[j] ? small_div(st[j] + s - 1, s) : 0;
        return __builtin_amdgcn_readlane(wave_inclusive_sum(tot), 63);
      };
      // splits per pair for split size s, each pair's first unit, and the total
      auto plan = [&](int s) {
        int tot = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          kk[j] = splits_for(st[j], s, sz[j]);
          start[j] = tot;
          tot += kk[j];
        }
        const int incl = wave_inclusive_sum(tot);
#pragma unroll
        for (int j = 0; j < 4; ++j) start[j] += incl - tot;
        return __builtin_amdgcn_readlane(incl, 63);
      };
      int s = max((W + U - 1) / U, a.min_split_steps);
      if (units_for(s) > U) {
        int lo = s + 1, hi = max(lo, (W + (U - a.pairs) - 1) / (U - a.pairs));
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (units_for(mid) <= U) hi = mid;
          else lo = mid + 1;
        }
        s = lo;
      }
      const int A = plan(s);
      int my = 0;
      const bool ok = A <= U && unit_of(A, my);
      // the pair whose units contain this unit: one lane and slot holds it
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint64_t m = __ballot(ok && kk[j] && my >= start[j] && my < start[j] + kk[j]);
        if (m) {
          const int l = __builtin_ctzll(m);
          p_new = 4 * l + j;
          slot0 = __builtin_amdgcn_readlane(start[j], l);
          nsplit = __builtin_amdgcn_readlane(kk[j], l);
          split_steps = __builtin_amdgcn_readlane(sz[j], l);
          split_new = my - slot0;
        }
      }
    }
    // (wave-uniform values, so that everything derived stays scalar)
    p_new = __builtin_amdgcn_readfirstlane(p_new);
    split_new = __builtin_amdgcn_readfirstlane(split_new);
    nsplit = __builtin_amdgcn_readfirstlane(nsplit);
    split_steps = __builtin_amdgcn_readfirstlane(split_steps);
    slot0 = __builtin_amdgcn_readfirstlane(slot0);
    if (p_new < 0 || p_new >= a.pairs || slot0 < 0 || nsplit < 1 || slot0 + nsplit > U) {
      drain();
      return;
    }
    // the pair's sizes, from the lane and slot that loaded them
    const int ol = p_new >> 2, oj = p_new & 3;
    auto owner = [&](const int (&v)[4]) {
      return __builtin_amdgcn_readlane(oj == 0 ? v[0] : oj == 1 ? v[1] : oj == 2 ? v[2] : v[3], ol);
    };
    n_raw = owner(pn);
    t_raw = owner(pt);
    c_raw = owner(pc);
    if (p_new != pair || split_new * split_steps != s_begin) {  // the guess was wrong
      pair = p_new;
      s_begin = split_new * split_steps;
      relocate = true;
    }
    split = split_new;
  } else {
    if (!guess_ok) {
      drain();
      return;
    }
    n_raw = __builtin_amdgcn_readlane(own_sizes, 0);
    t_raw = a.dims.n_query ? __builtin_amdgcn_readlane(own_sizes, 1) : a.dims.nq_max;
    c_raw = kSparse ? __builtin_amdgcn_readlane(own_sizes, 2) : 0;
  }

  const int N = clampi(n_raw, 0, a.dims.max_len);
  const int T = clampi(t_raw, 0, a.dims.nq_max);
  if (T == 0) {
    drain();
    return;
  }
  const int wstart = kSparse ? clampi(c_raw, 0, a.dims.k_max) : N;
  const int total = wstart + T;        // virtual tokens: selected (or all) then window
  const int rows = T * a.group_size;   // <= RT * 16 (checked on the host via nq_max)
  const int nsteps = sep ? max(1, (wstart + kStep - 1) / kStep) : (total + kStep - 1) / kStep;
  if (s_begin >= nsteps) {
    drain();
    return;
  }
  const int s_end = min(nsteps, s_begin + split_steps);
  // the wave that takes the window step: in the pair's last split, the last wave with the
  // fewest steps of the split (wave 3, or the last wave with a step when there are fewer
  // than four)
  const bool has_window = sep && split == nsplit - 1 && wave == min(kW - 1, s_end - s_begin - 1);
  // with a window step, tokens from wstart on are the window's: body steps mask them
  const int body_limit = sep ? wstart - 1 : INT32_MAX;

  // Position of virtual token v (clamped into the cache; past-the-end -> 0) and its
  // physical row.
  auto pos_of = [&](int v, int32_t selected) -> int {
    const int pos = v < wstart ? (kSparse ? selected : v) : (v < total ? N + (v - wstart) : 0);
    return clampi(pos, 0, cap_m1);
  };
  auto page_of = [&](int pos) -> int {
    return clampi(a.k.page_table[(int64_t)b * a.k.max_pages + (pos >> a.k.page_shift)], 0,
                  a.k.num_pages - 1);
  };
  auto phys_at = [&](int pos, int page) -> uint32_t {
    if constexpr (kPaged)
      return ((uint32_t)page << a.k.page_shift) | (uint32_t)(pos & ((1 << a.k.page_shift) - 1));
    else
      return (uint32_t)pos;
  };
  // The window step's rows go to a tile of their own.
  auto issue_window = [&](auto buffered) {
    uint32_t ph[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if constexpr (kPaged) ph[i] = sm_wphys[8 * lg + i];
      else ph[i] = (uint32_t)pos_of(wstart + 8 * lg + i, 0);
    }
    issue_rows_to(ph, sm_win, sm_win + kTile, buffered);
  };
  if (relocate) {
    if constexpr (kSpec) wait_vmem_all();  // the speculative rows have landed in this wave's tile
    locate();
    set_rows();
    first_loads();
    prologue_loads();
  }
  bool first_issued = false;
  if constexpr (kSpec) {
    // the speculative step was the wrong unit's: issue it again
    if (relocate) issue_first([&](int v, int32_t selected) { return (int)phys_at(pos_of(v, selected), 0); });
    first_issued = s_begin + wave < min(s_end, s_begin + kStageSteps);
    // a wave whose first step lies beyond the first chunk issues it into the same tile
    // later: the speculative rows land first
    if (!first_issued) wait_vmem_all();
  }

  int limit[RT];  // token v is visible to this lane's row iff v <= limit
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = rt * 16 + lr;
    limit[rt] = wstart + (r < rows ? small_div(r, a.group_size) : T - 1);
  }
  // rows of absent verification tokens act as zero queries
#pragma unroll
  for (int j = 0; j < kQPer; ++j) {
    const int e = threadIdx.x + j * kW * kWave;
    const int r = e / (kD / 8), c0 = (e % (kD / 8)) * 8;
    if (e < kQChunks) *reinterpret_cast<u32x4*>(sm_q + r * kQPitch + c0) = r < rows ? qx[j] : u32x4{0u, 0u, 0u, 0u};
  }
  auto q_operand = [&](int rt, int ks) -> bf16x8 {
    if constexpr (kQReg)
      return qreg[rt][ks];
    else
      return as_bf16x8(*reinterpret_cast<const u32x4*>(sm_q + (rt * 16 + lr) * kQPitch + 8 * lg + 32 * ks));
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

  // physical rows of this lane's tokens in step st
  auto step_rows = [&](int st, uint32_t (&ph)[8]) {
    const int v0 = st * kStep + 8 * lg;
    if constexpr (kStage) {
      const u32x4* src = reinterpret_cast<const u32x4*>(sm_phys + (v0 - chunk_v0));
      const u32x4 p0 = src[0], p1 = src[1];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ph[i] = p0[i];
        ph[4 + i] = p1[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) ph[i] = v0 + i < total ? (uint32_t)(v0 + i) : 0u;
    }
  };
  auto issue = [&](int st) {
    uint32_t ph[8];
    step_rows(st, ph);
    issue_rows_to(ph, ktile, vtile, LoopForm{});
  };

  // With up to four row tiles a wave reads all of a step's operands into registers and
  // starts the next step's loads before computing.  With more, the registers are needed
  // for the accumulators: the wave computes first, reading V^T from its tile as it goes,
  // and only then starts the next step (the other waves of the CU keep loads in flight).
  constexpr bool kOverlap = RT <= 4;
  struct Operands {
    bf16x8 k[2][4];                // K rows of the step's two 16-token tiles (MFMA A layout)
    bf16x8 vt[kOverlap ? NDT : 1];  // V^T of each 16-column tile over the 32 tokens (MFMA A layout)
  };

  // V^T operand of 16-column tile dt: lane lr of a 16-lane group addresses token
  // 4 lg + lr / 4 (+16 for the second half of k), columns 16 dt + 4 (lr % 4) .. + 3; it
  // receives V[token 4 lg + e (+16)][16 dt + lr]
  auto read_vt = [&](const char* vt, int dt) -> bf16x8 {
    const int j0 = 4 * lg + (lr >> 2), j1 = j0 + 16;
    const int c = 2 * dt + ((lr >> 1) & 1);
    const v4i16 lo = lds_read_tr16(vt + tile_row(j0) * 256 + 8 * (lr & 1) + 16 * v_chunk(j0, c));
    const v4i16 hi = lds_read_tr16(vt + tile_row(j1) * 256 + 8 * (lr & 1) + 16 * v_chunk(j1, c));
    return as_bf16x8(u32x4{__builtin_bit_cast(u32x2, lo)[0], __builtin_bit_cast(u32x2, lo)[1],
                           __builtin_bit_cast(u32x2, hi)[0], __builtin_bit_cast(u32x2, hi)[1]});
  };

  // Reads a step's operands out of a K and a V tile (after their loads completed).
  auto read_tiles_from = [&](const char* kt, const char* vt, Operands& op) {
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const int j = 16 * t2 + lr;
      const char* row = kt + tile_row(j) * 256;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        op.k[t2][ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(row + 16 * k_chunk(j, 4 * ks + lg)));
    }
    if constexpr (kOverlap)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) op.vt[dt] = read_vt(vt, dt);
  };
  auto read_tiles = [&](Operands& op) { read_tiles_from(ktile, vtile, op); };

  // One 32-token step on register operands, one 16-row tile at a time (its scores,
  // probabilities and softmax decision live only while the tile is processed, which keeps
  // five row tiles inside the register file): (1) the score tile; (2) its softmax, with
  // one wave-uniform decision whether to move the tile's reference maxima; (3) its value
  // product.  Scores stay in raw units until one FMA forms (s * scale * log2 e - m) inside
  // exp2; the reference max m is in scaled units.
  // v0: the virtual token of the tile's first row; vt: its V tile; win: the window step
  // (causal mask per query row), else a body step (with a window step, tokens from wstart on
  // belong to the window step and are masked here).
  // A pair with fewer query rows than the launch's widest skips its absent row tiles (their
  // maxima stay -inf and their sums zero, which the merges below ignore).  Not up to three
  // row tiles (the branches changed that code, and it measured 0.1-0.2 us per layer slower
  // at the Qwen2.5-72B shape), nor in the dense contiguous kernels, where at five row tiles
  // they cost a spill.
  auto tile_absent = [&](int rt) { return kStage && RT > 3 && rt > 0 && rt * 16 >= rows; };
  auto compute = [&](int v0, const Operands& op, const char* vt, bool win) {
    const bool edge = win || v0 + kStep - 1 >= wstart;  // wave-uniform: masking only near the window
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      if (tile_absent(rt)) break;
      // (1) S^T tile: lane holds tokens v0 + 16 i + 4 lg + e for query row rt*16 + lr
      f32x4 sc[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) c = mfma16x16x32(op.k[i][ks], q_operand(rt, ks), c);
        sc[i] = c;
      }
      // (2) masked row maxima, lazy rescale, probabilities
      if (edge) {
        const int lim = win ? limit[rt] : min(limit[rt], body_limit);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (v0 + 16 * i + 4 * lg + e > lim) sc[i][e] = -INFINITY;
      }
      const float m = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                            fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
      const float mx = max_over_lane_groups(m) * a.scale_log2;
      if (__any(mx > m_ref[rt] + kRescaleLog2)) {  // wave-uniform, rare after the first step
        const float mn = fmaxf(m_ref[rt], mx);
        const float alpha = m_ref[rt] == -INFINITY ? 0.f : fast_exp2(m_ref[rt] - mn);
        m_ref[rt] = mn;
        accl[rt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[rt][dt] *= alpha;
      }
      const float nmu = m_ref[rt] == -INFINITY ? 0.f : -m_ref[rt];
      float p[2][4];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) p[i][e] = fast_exp2(fmaf(sc[i][e], a.scale_log2, nmu));
      // B operand of the PV product: k slot 8 lg + e <-> token 4 lg + e (e < 4, tile 0)
      // and token 16 + 4 lg + e - 4 (e >= 4, tile 1)
      const bf16x8 pT = as_bf16x8(u32x4{cvt_pk_bf16(p[0][0], p[0][1]), cvt_pk_bf16(p[0][2], p[0][3]),
                                        cvt_pk_bf16(p[1][0], p[1][1]), cvt_pk_bf16(p[1][2], p[1][3])});
      accl[rt] = mfma16x16x32(ones, pT, accl[rt]);
      // (3) O^T tiles
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        if constexpr (kOverlap) acc[rt][dt] = mfma16x16x32(op.vt[dt], pT, acc[rt][dt]);
        else acc[rt][dt] = mfma16x16x32(read_vt(vt, dt), pT, acc[rt][dt]);
      }
    }
  };
  // The same step in two halves (kernels that wait for K and V separately; body steps
  // only, as these kernels have no window step): (1) and (2) of every row tile from the
  // K rows, then (3) of every row tile from the V tile, each V^T operand read once.
  // (1) and (2) of row tile rt, the same steps as in compute(): returns the tile's
  // probabilities as the B operand of its value product, after adding their row sums.
  auto tile_probs = [&](int rt, int v0, const Operands& op, bool win, bool edge) -> bf16x8 {
    // (1) S^T tile: lane holds tokens v0 + 16 i + 4 lg + e for query row rt*16 + lr
    f32x4 sc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) c = mfma16x16x32(op.k[i][ks], q_operand(rt, ks), c);
      sc[i] = c;
    }
    // (2) masked row maxima, lazy rescale, probabilities
    if (edge) {
      const int lim = win ? limit[rt] : min(limit[rt], body_limit);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (v0 + 16 * i + 4 * lg + e > lim) sc[i][e] = -INFINITY;
    }
    const float m = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                          fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
    const float mx = max_over_lane_groups(m) * a.scale_log2;
    if (__any(mx > m_ref[rt] + kRescaleLog2)) {  // wave-uniform, rare after the first step
      const float mn = fmaxf(m_ref[rt], mx);
      const float alpha = m_ref[rt] == -INFINITY ? 0.f : fast_exp2(m_ref[rt] - mn);
      m_ref[rt] = mn;
      accl[rt] *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) acc[rt][dt] *= alpha;
    }
    const float nmu = m_ref[rt] == -INFINITY ? 0.f : -m_ref[rt];
    float p[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) p[i][e] = fast_exp2(fmaf(sc[i][e], a.scale_log2, nmu));
    const bf16x8 pT = as_bf16x8(u32x4{cvt_pk_bf16(p[0][0], p[0][1]), cvt_pk_bf16(p[0][2], p[0][3]),
                                      cvt_pk_bf16(p[1][0], p[1][1]), cvt_pk_bf16(p[1][2], p[1][3])});
    accl[rt] = mfma16x16x32(ones, pT, accl[rt]);
    return pT;
  };
  auto compute_scores = [&](int v0, const Operands& op, bf16x8 (&pT)[RT]) {
    const bool edge = v0 + kStep - 1 >= wstart;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      if (tile_absent(rt)) break;
      pT[rt] = tile_probs(rt, v0, op, false, edge);
    }
  };
  auto compute_values = [&](const char* vt, const bf16x8 (&pT)[RT]) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const bf16x8 v = read_vt(vt, dt);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        if (tile_absent(rt)) break;
        acc[rt][dt] = mfma16x16x32(v, pT[rt], acc[rt][dt]);
      }
    }
  };

  // Physical rows of this thread's tokens in chunk cs (reads sel, and the page table).
  uint32_t staged[kStageBatch];
  auto stage_rows = [&](int cs) {
    int pos[kStageBatch];
    int page[kStageBatch];
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j) pos[j] = pos_of(cs * kStep + 8 * (int)threadIdx.x + j, sel[j]);
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j) page[j] = kPaged ? page_of(pos[j]) : 0;
#pragma unroll
    for (int j = 0; j < kStageBatch; ++j) staged[j] = phys_at(pos[j], page[j]);
  };
  auto store_staged = [&](int cs, int ce) {
    chunk_v0 = cs * kStep;
    const int nv = ce * kStep - chunk_v0;  // a multiple of 32
    if (8 * (int)threadIdx.x < nv) {
      u32x4* dst = reinterpret_cast<u32x4*>(sm_phys + 8 * threadIdx.x);
      dst[0] = u32x4{staged[0], staged[1], staged[2], staged[3]};
      dst[1] = u32x4{staged[4], staged[5], staged[6], staged[7]};
    }
  };
  // the first chunk's table (and, paged, the window step's rows, by the first 32 threads
  // of the workgroup that takes it)
  const bool wg_window = sep && split == nsplit - 1;
  if constexpr (kStage) {
    stage_rows(s_begin);
    if constexpr (kPaged) {
      if (wg_window && threadIdx.x < kStep) {
        const int pos = pos_of(wstart + (int)threadIdx.x, 0);
        sm_wphys[threadIdx.x] = phys_at(pos, page_of(pos));
      }
    }
    store_staged(s_begin, min(s_end, s_begin + kStageSteps));
  }
  if constexpr (kSpec) {
    // The window's rows go after the staging (a conditional load between the queries' and
    // positions' loads and their waits would cost the compiler its count); the wave
    // computes them after its last step.
    if (has_window) issue_window(Buffered{});
  }
  if constexpr (!kSpec) {
    // every prologue load is consumed before the first global_load_lds (with those in
    // flight the compiler would wait for all loads at the first use of any)
    wait_vmem_all();
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (!kPaged && !kSpec) {
    // the table shares the tiles' LDS object: the first step goes after its stores
    if (has_window) issue_window(Global{});
    __builtin_amdgcn_sched_barrier(0);  // the window's loads stay ahead of the step's
    if (s_begin + wave < min(s_end, s_begin + kStageSteps)) {
      uint32_t ph[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) ph[i] = phys_at(pos_of(first_v0 + i, first_sel[i]), 0);
      issue_rows_to(ph, ktile, vtile, LoopForm{});
      first_issued = true;
    }
  }
  for (int cs = s_begin; cs < s_end; cs += kStageSteps) {
    const int ce = min(s_end, cs + kStageSteps);
    if constexpr (kStage) {
      if (cs != s_begin) {
        __syncthreads();  // the previous chunk's rows are no longer read
        load_selection(cs);
        stage_rows(cs);
        store_staged(cs, ce);
      }
    }
    lds_barrier();  // staged rows (and staged queries) are visible
    if constexpr (kQReg) {
      if (cs == s_begin) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int ks = 0; ks < 4; ++ks)
            qreg[rt][ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(sm_q + (rt * 16 + lr) * kQPitch + 8 * lg + 32 * ks));
      }
    }
    // this wave's steps: cs + wave + i kW
    int st = cs + wave;
    if (st >= ce) continue;
    if constexpr (kPaged) {
      if (has_window && cs == s_begin) issue_window(Global{});
      __builtin_amdgcn_sched_barrier(0);  // the window's loads stay ahead of the step's
    }
    if (!(first_issued && cs == s_begin)) issue(st);
    if (!kSpec && has_window && cs == s_begin) {
      // the window's 16 loads were issued before the step's 16: wait for them alone and
      // compute the window while the step is in flight
      __builtin_amdgcn_s_waitcnt(0x4F70);  // vmcnt(16)
      Operands opw;
      read_tiles_from(sm_win, sm_win + kTile, opw);
      compute(wstart, opw, sm_win + kTile, true);
    }
    while (true) {
      if constexpr (kSplitKV) {
        // Outstanding here: this step's K loads, then its V loads.  The K rows go to
        // registers and the next step's K loads into the freed tile; the scores are computed
        // while this step's V rows (and the next K rows) arrive; then the value products, and
        // the next step's V loads into the freed V tile.
        wait_vmem_8();  // this step's K rows are in the tile
        Operands op;
        read_tiles(op);
        const int next = st + kW;
        if (next < ce) {
          uint32_t ph[8];
          step_rows(next, ph);
          wait_lds_all();  // the K tile has been read out
          issue_rows_to_k(ph, ktile);
        }
        bf16x8 pT[RT];
        compute_scores(st * kStep, op, pT);
        if (next < ce) wait_vmem_8();  // this step's V rows are in the tile (the next K rows may not be)
        else wait_vmem_all();
        compute_values(vtile, pT);
        if (next >= ce) break;
        uint32_t ph[8];
        step_rows(next, ph);
        wait_lds_all();  // the V tile has been read out
        issue_v_to(ph, vtile, Buffered{});
        st = next;
        continue;
      }
      wait_vmem_all();  // this step's rows are in the tiles
      Operands op;
      read_tiles(op);
      const int next = st + kW;
      if constexpr (kOverlap) {
        if (next < ce) {
          wait_lds_all();  // the tiles have been read out before the next loads overwrite them
          issue(next);
        }
        compute(st * kStep, op, vtile, false);
      } else {
        compute(st * kStep, op, vtile, false);
        if (next < ce) {
          wait_lds_all();
          issue(next);
        }
      }
      if (next >= ce) break;
      st = next;
    }
  }
  if constexpr (kSpec) {
    if (has_window) {
      wait_vmem_all();
      Operands opw;
      read_tiles_from(sm_win, sm_win + kTile, opw);
      compute(wstart, opw, sm_win + kTile, true);
    }
  }

  // ---- combine the waves: each leaves its raw (max, sum, acc) in LDS; then every thread
  // merges four columns of its rows over the waves, in wave order (deterministic) ----
  __shared__ float sm_m[kW][RT * 16];
  __shared__ float sm_l[kW][RT * 16];
  __shared__ int sm_last;
  float* const bufs = reinterpret_cast<float*>(smem);  // [kNB][RT * 16][kPitch]
  auto put_acc = [&](float* buf) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
        *reinterpret_cast<f32x4*>(buf + (rt * 16 + lr) * kPitch + 16 * dt + 4 * lg) = acc[rt][dt];
  };
  auto put_stats = [&]() {
    if (lg == 0)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        sm_m[wave][rt * 16 + lr] = m_ref[rt];
        sm_l[wave][rt * 16 + lr] = accl[rt][0];
      }
  };
  put_stats();
  __syncthreads();  // every wave is past its token loop: the tiles are free
  if constexpr (kNB < kW) {
    // not enough LDS for one buffer per wave: in rounds, waves [top - kNB, top) hand their
    // partials to waves [top - 2 kNB, top - kNB) until only kNB waves hold one
    for (int top = kW; top > kNB; top -= kNB) {
      if (wave >= top - kNB && wave < top) put_acc(bufs + (wave - (top - kNB)) * kBufFloats);
      __syncthreads();
      if (wave >= top - 2 * kNB && wave < top - kNB) {
        const int p = wave + kNB;
        const float* pb = bufs + (wave - (top - 2 * kNB)) * kBufFloats;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const int r = rt * 16 + lr;
          const float mp = sm_m[p][r], lp = sm_l[p][r];
          const float M = fmaxf(m_ref[rt], mp), Mu = M == -INFINITY ? 0.f : M;
          const float fa = m_ref[rt] == -INFINITY ? 0.f : fast_exp2(m_ref[rt] - Mu);
          const float fb = mp == -INFINITY ? 0.f : fast_exp2(mp - Mu);
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
            acc[rt][dt] = acc[rt][dt] * fa + *reinterpret_cast<const f32x4*>(pb + r * kPitch + 16 * dt + 4 * lg) * fb;
          accl[rt][0] = accl[rt][0] * fa + lp * fb;
          m_ref[rt] = M;
        }
        put_stats();
      }
      __syncthreads();  // the handed-over buffers have been read, the new stats written
    }
  }
  if (wave < kNB) put_acc(bufs + wave * kBufFloats);
  __syncthreads();

  // thread element k: row e / 32, columns 4 (e % 32) .. + 3, e = threadIdx.x + 256 k
  constexpr int nthreads = kW * kWave;
  constexpr int KE = (RT * 16 * (kD / 4) + nthreads - 1) / nthreads;
  const int nel = rows * (kD / 4);
  f32x4 o[KE];
  float Mk[KE], Lk[KE];
  // Every LDS read of the merge is issued before any of its arithmetic.  (Written as one
  // loop, the compiler waited for each batch of reads in turn, some thirty LDS round trips
  // in a row.)
  float mw[KE][kNB], lw[KE][kNB];
  f32x4 xw[KE][kNB];
#pragma unroll
  for (int k = 0; k < KE; ++k) {
    const int e = min((int)threadIdx.x + k * nthreads, nel - 1);
    const int r = e / (kD / 4), c0 = (e % (kD / 4)) * 4;
#pragma unroll
    for (int w = 0; w < kNB; ++w) {
      mw[k][w] = sm_m[w][r];
      lw[k][w] = sm_l[w][r];
      xw[k][w] = *reinterpret_cast<const f32x4*>(bufs + w * kBufFloats + r * kPitch + c0);
    }
  }
#pragma unroll
  for (int k = 0; k < KE; ++k) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kNB; ++w) M = fmaxf(M, mw[k][w]);
    const float Mu = M == -INFINITY ? 0.f : M;
    float L = 0.f;
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < kNB; ++w) {
      const float f = mw[k][w] == -INFINITY ? 0.f : fast_exp2(mw[k][w] - Mu);
      L += lw[k][w] * f;
      sum += xw[k][w] * f;
    }
    o[k] = sum;
    Mk[k] = M;
    Lk[k] = L;
  }

  auto out_ptr = [&](int r) {
    const int t = r / a.group_size, hh = r - t * a.group_size;
    return a.out + (int64_t)b * a.o_sb + (int64_t)t * a.o_st + (int64_t)(g * a.group_size + hh) * a.o_sh;
  };
  auto store_out = [&](int k, const f32x4& v) {
    const int e = (int)threadIdx.x + k * nthreads;
    if (e < nel) {
      const int r = e / (kD / 4), c0 = (e % (kD / 4)) * 4;
      *reinterpret_cast<u32x2*>(out_ptr(r) + c0) = u32x2{cvt_pk_bf16(v[0], v[1]), cvt_pk_bf16(v[2], v[3])};
    }
  };
  if (nsplit == 1) {
#pragma unroll
    for (int k = 0; k < KE; ++k) store_out(k, o[k] * (Lk[k] > 0.f ? 1.f / Lk[k] : 0.f));
    return;
  }

  // ---- several splits: publish (write-through), count in; the last one merges ----
  // A split's partial is [rows][128] fp32 (unnormalised, relative to its row maxima) plus
  // (max, sum) per row, reached through buffer resources whose stores and loads carry the
  // agent-scope (sc1) cache policy, so they are coherent across XCDs without cache flushes.
  constexpr int kSC1 = 16;
  auto part_rsrc = [&](int sp) {
    return __builtin_amdgcn_make_buffer_rsrc(a.part_acc + (int64_t)(slot0 + sp) * a.rows_pad * kD, 0,
                                             a.rows_pad * kD * 4, 0x00020000);
  };
  auto ml_rsrc = [&](int sp) {
    return __builtin_amdgcn_make_buffer_rsrc(a.part_ml + (int64_t)(slot0 + sp) * a.rows_pad * 2, 0,
                                             a.rows_pad * 2 * 4, 0x00020000);
  };
  {
    const auto ra = part_rsrc(split), rm = ml_rsrc(split);
#pragma unroll
    for (int k = 0; k < KE; ++k) {
      const int e = (int)threadIdx.x + k * nthreads;
      if (e < nel) {
        const int r = e / (kD / 4), c0 = (e % (kD / 4)) * 4;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, o[k]), ra, (r * kD + c0) * 4, 0, kSC1);
        if (c0 == 0)
          __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(Mk[k]), __float_as_uint(Lk[k])}, rm, r * 8, 0,
                                                kSC1);
      }
    }
  }
  wait_vmem_all();  // this thread's write-through stores have completed
  __syncthreads();  // ... and every other thread's
  if (threadIdx.x == 0)
    sm_last = __hip_atomic_fetch_add(a.counters + pair, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nsplit - 1;
  __syncthreads();
  if (!sm_last) return;
  if (threadIdx.x == 0) __hip_atomic_store(a.counters + pair, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // merge the splits online in split order (the same order whichever workgroup is last):
  // this workgroup's own partial from registers, every other one read back with one
  // batch of loads
  f32x4 res[KE];
  float Mr[KE], Lr[KE];
  for (int sp = 0; sp < nsplit; ++sp) {
    f32x4 x[KE];
    float ms[KE], ls[KE];
    if (sp == split) {
#pragma unroll
      for (int k = 0; k < KE; ++k) {
        x[k] = o[k];
        ms[k] = Mk[k];
        ls[k] = Lk[k];
      }
    } else {
      const auto ra = part_rsrc(sp), rm = ml_rsrc(sp);
#pragma unroll
      for (int k = 0; k < KE; ++k) {
        const int e = min((int)threadIdx.x + k * nthreads, nel - 1);
        const int r = e / (kD / 4), c0 = (e % (kD / 4)) * 4;
        x[k] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, (r * kD + c0) * 4, 0, kSC1));
        const u32x2 ml = __builtin_amdgcn_raw_buffer_load_b64(rm, r * 8, 0, kSC1);
        ms[k] = __uint_as_float(ml[0]);
        ls[k] = __uint_as_float(ml[1]);
      }
    }
#pragma unroll
    for (int k = 0; k < KE; ++k) {
      if (sp == 0) {
        res[k] = x[k];
        Mr[k] = ms[k];
        Lr[k] = ls[k];
      } else {
        const float M = fmaxf(Mr[k], ms[k]), Mu = M == -INFINITY ? 0.f : M;
        const float fa = Mr[k] == -INFINITY ? 0.f : fast_exp2(Mr[k] - Mu);
        const float fb = ms[k] == -INFINITY ? 0.f : fast_exp2(ms[k] - Mu);
        res[k] = res[k] * fa + x[k] * fb;
        Lr[k] = Lr[k] * fa + ls[k] * fb;
        Mr[k] = M;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < KE; ++k) store_out(k, res[k] * (Lr[k] > 0.f ? 1.f / Lr[k] : 0.f));
}

// ------------------------------------------------------------------------- host side

template <int RT, bool kSparse, bool kPaged>
static hipError_t launch_rt(const AttnArgs& a, hipStream_t stream) {
  const int units = a.splits * a.pairs;
  const int blocks = (units + 7) / 8 * 8;
  constexpr bool kQReg = RT <= 3;
  hipLaunchKernelGGL((verify_attn_kernel<RT, kSparse, kPaged, kQReg>), dim3(blocks), dim3(kW * kWave), 0,
                     stream, a);
  return hipGetLastError();
}

template <bool kSparse, bool kPaged>
static hipError_t launch_kind(const AttnArgs& a, int rt, hipStream_t stream) {
  switch (rt) {
    case 1: return launch_rt<1, kSparse, kPaged>(a, stream);
    case 2: return launch_rt<2, kSparse, kPaged>(a, stream);
    case 3: return launch_rt<3, kSparse, kPaged>(a, stream);
    case 4: return launch_rt<4, kSparse, kPaged>(a, stream);
    case 5: return launch_rt<5, kSparse, kPaged>(a, stream);
    case 6: return launch_rt<6, kSparse, kPaged>(a, stream);
    case 7:
    case 8: return launch_rt<8, kSparse, kPaged>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_verify_attn(const AttnArgs& a, int rt, bool sparse, bool paged, hipStream_t stream) {
  if (sparse) return paged ? launch_kind<true, true>(a, rt, stream) : launch_kind<true, false>(a, rt, stream);
  return paged ? launch_kind<false, true>(a, rt, stream) : launch_kind<false, false>(a, rt, stream);
}

}  // namespace dustin
