// page.hip -- page statistics for the page estimator (the query-aware page scoring the
// paper compares its estimator with): for every page of 2^page_shift committed positions
// and every KV head, the channel-wise maximum and minimum of K over the page's positions
// below N_b.  A statistics row is [max | min], 2d bf16 values; min and max of bf16 values
// are bf16 values, so the row is exact.
//
// One thread per (page, 16-byte chunk of a K row): it reads the chunk at every position of
// its page (all loads issued before the first compare) and keeps, per channel, the value
// that compares strictly greater (smaller) than every earlier one, so that of equal values
// the earliest position's bit pattern stays (this decides only the sign of a zero).
// Only pages from the one holding position from_b onwards are rewritten: after an append,
// the pages that changed.
#include "kernels.hpp"

namespace dustin {

constexpr int kMetaThreads = 256;
constexpr int kMetaBatch = 8;  // positions loaded together

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

template <int D, bool kPaged>
__global__ __launch_bounds__(kMetaThreads) void page_meta_kernel(PageMetaArgs a) {
  constexpr int C = D / 8;  // 16-byte chunks per row
  constexpr int kPagesPerBlock = kMetaThreads / C;
  const int g = blockIdx.y, b = blockIdx.z;
  const int c = threadIdx.x % C, pl = threadIdx.x / C;
  const int N = a.dims.len(b);
  const int P = (N + (1 << a.page_shift) - 1) >> a.page_shift;
  const int from = a.from ? clampi(a.from[b], 0, N) : 0;
  const int p = (from >> a.page_shift) + blockIdx.x * kPagesPerBlock + pl;
  if (p >= P) return;
  const int n0 = p << a.page_shift, n1 = min(n0 + (1 << a.page_shift), N);

  const u32x4 first = load16(a.k.row<kPaged>(b, n0, g) + 8 * c);
  u32x4 hi = first, lo = first;  // bf16 pairs; halves updated independently
  for (int n = n0 + 1; n < n1; n += kMetaBatch) {
    u32x4 r[kMetaBatch];
#pragma unroll
    for (int u = 0; u < kMetaBatch; ++u)  // past the page: the first row again (never replaces)
      r[u] = n + u < n1 ? load16(a.k.row<kPaged>(b, n + u, g) + 8 * c) : first;
#pragma unroll
    for (int u = 0; u < kMetaBatch; ++u) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t x = r[u][i];
        const uint32_t h_lo = bf16_lo(x) > bf16_lo(hi[i]) ? x & 0xFFFFu : hi[i] & 0xFFFFu;
        const uint32_t h_hi = bf16_hi(x) > bf16_hi(hi[i]) ? x & 0xFFFF0000u : hi[i] & 0xFFFF0000u;
        const uint32_t l_lo = bf16_lo(x) < bf16_lo(lo[i]) ? x & 0xFFFFu : lo[i] & 0xFFFFu;
        const uint32_t l_hi = bf16_hi(x) < bf16_hi(lo[i]) ? x & 0xFFFF0000u : lo[i] & 0xFFFF0000u;
        hi[i] = h_hi | h_lo;
        lo[i] = l_hi | l_lo;
      }
    }
  }
  uint16_t* row = a.meta + (int64_t)b * a.m_sb + (int64_t)p * a.m_sp + (int64_t)g * (2 * D) + 8 * c;
  *reinterpret_cast<u32x4*>(row) = hi;
  *reinterpret_cast<u32x4*>(row + D) = lo;
}

hipError_t launch_page_meta(const PageMetaArgs& a, int B, int head_dim, hipStream_t stream) {
  const int ppb = kMetaThreads / (head_dim / 8);
  const dim3 grid((a.span_pages + ppb - 1) / ppb, a.num_kv_heads, B);
  const bool paged = a.k.page_table != nullptr;
  if (head_dim == 128) {
    if (paged) hipLaunchKernelGGL((page_meta_kernel<128, true>), grid, dim3(kMetaThreads), 0, stream, a);
    else hipLaunchKernelGGL((page_meta_kernel<128, false>), grid, dim3(kMetaThreads), 0, stream, a);
  } else if (head_dim == 64) {
    if (paged) hipLaunchKernelGGL((page_meta_kernel<64, true>), grid, dim3(kMetaThreads), 0, stream, a);
    else hipLaunchKernelGGL((page_meta_kernel<64, false>), grid, dim3(kMetaThreads), 0, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dustin
