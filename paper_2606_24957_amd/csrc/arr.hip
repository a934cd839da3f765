// arr.hip -- windowed attention recovery rate of index sets (the evaluation framework,
// Eqs. 1-4).  ARR is linear in the attention weights, so the head-averaged windowed ARR of
// a set is the sum over the set of the head-averaged window attention A-bar (Eq. 3), and
// A-bar is the Eq. 5 score over every served head and the window's queries, divided by
// (window length x heads).  One workgroup per (output group, sequence) gathers the score
// at the set's positions and sums in fp64 in a fixed order (per thread, then a butterfly
// over the wave, then the waves in order), so that the result does not depend on timing.
#include "kernels.hpp"

namespace dustin {

constexpr int kArrThreads = 256;

__global__ __launch_bounds__(kArrThreads) void arr_kernel(ArrArgs a) {
  const int go = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int N = a.dims.len(b);
  const int w = a.dims.nq(b);
  const int c = clampi(a.count[(int64_t)b * a.groups + go], 0, a.dims.k_max);
  const int32_t* ix = a.idx + (int64_t)b * a.idx_sb + (int64_t)go * a.idx_sg;
  const float* s = a.s + (int64_t)b * a.s_sb + (int64_t)go * a.s_sg;
  double acc = 0.0;
  for (int i = tid; i < c; i += kArrThreads) {
    const int n = ix[i];
    if (n >= 0 && n < N) acc += (double)s[n];
  }
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) acc += __shfl_xor(acc, off);
  __shared__ double sm[kArrThreads / kWave];
  if (lane == 0) sm[wave] = acc;
  __syncthreads();
  if (tid == 0) {
    double tot = 0.0;
    for (int i = 0; i < kArrThreads / kWave; ++i) tot += sm[i];
    a.arr[(int64_t)b * a.groups + go] = w > 0 ? tot / ((double)w * a.heads_per_group) : 0.0;
  }
}

hipError_t launch_arr(const ArrArgs& a, int B, hipStream_t stream) {
  hipLaunchKernelGGL(arr_kernel, dim3(a.groups, B), dim3(kArrThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dustin
