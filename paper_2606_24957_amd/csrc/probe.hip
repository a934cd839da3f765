// probe.hip -- a plain streaming read of a device buffer: the practical read rate of the
// GPU, against which the bandwidth-bound kernels' rates are reported.
//
// Workgroup g of G reads the g-th of G equal runs of 16-byte units of the buffer with
// 16-byte buffer loads, 16 in flight per lane, and writes the wrapping sum of the 32-bit
// words it read to sums[g] (so that no load can be dropped, and a test can check them).
#include "kernels.hpp"
#include "probe.hpp"

namespace dustin {

namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeLoads = 16;

__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const uint8_t* data, uint64_t units,
                                                                   uint64_t per_block, uint32_t* sums) {
  const uint64_t u0 = (uint64_t)blockIdx.x * per_block;
  const uint64_t u1 = u0 + per_block < units ? u0 + per_block : units;
  __shared__ uint32_t part[kProbeThreads / kWave];
  uint32_t acc = 0;
  if (u0 < u1) {
    // the run through one buffer resource (its byte size below 2^31, checked on the host);
    // loads past its end read zero
    const uint32_t bytes = (uint32_t)((u1 - u0) * 16);
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(data + u0 * 16), 0, (int)bytes, 0x00020000);
    const uint32_t step = kProbeThreads * 16 * kProbeLoads;
    for (uint32_t off = threadIdx.x * 16; off < bytes; off += step) {
      u32x4 v[kProbeLoads];
#pragma unroll
      for (int i = 0; i < kProbeLoads; ++i)
        v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(off + i * kProbeThreads * 16), 0, 0));
#pragma unroll
      for (int i = 0; i < kProbeLoads; ++i) acc += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
    }
  }
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if ((threadIdx.x & (kWave - 1)) == 0) part[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
#pragma unroll
    for (int w = 0; w < kProbeThreads / kWave; ++w) t += part[w];
    sums[blockIdx.x] = t;
  }
}

}  // namespace

hipError_t launch_read_probe(const void* data, uint64_t bytes, uint32_t* sums, int blocks, hipStream_t stream) {
  const uint64_t units = bytes / 16;
  const uint64_t per_block = (units + blocks - 1) / blocks;
  if (per_block * 16 >= (1ull << 31)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(read_probe_kernel, dim3(blocks), dim3(kProbeThreads), 0, stream,
                     static_cast<const uint8_t*>(data), units, per_block, sums);
  return hipGetLastError();
}

}  // namespace dustin
