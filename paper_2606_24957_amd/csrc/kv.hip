// kv.hip -- the steps on either side of verification (Sec. 3.2): the target KV of the T_b
// verification tokens is written into the cache at positions [N_b, N_b + T_b) before the
// verification attention reads it, and afterwards the accepted tokens are kept by moving
// N_b past them; the rejected rows stay beyond N_b, unseen, until the next step's window
// overwrites them.
#include "kernels.hpp"

namespace dustin {

constexpr int kKvThreads = 256;

// One 16-byte chunk per thread; rows are (cache: K then V, sequence, token, KV head).
__global__ __launch_bounds__(kKvThreads) void kv_append_kernel(KvAppendArgs a) {
  const int cpr = a.head_dim / 8;  // chunks per row
  int64_t i = (int64_t)blockIdx.x * kKvThreads + threadIdx.x;
  const int chunk = (int)(i % cpr);
  i /= cpr;
  const int h = (int)(i % a.num_kv_heads);
  i /= a.num_kv_heads;
  const int t = (int)(i % a.dims.nq_max);
  i /= a.dims.nq_max;
  const int b = (int)(i % a.batch);
  const int which = (int)(i / a.batch);
  if (which >= 2) return;
  if (t >= a.dims.nq(b)) return;
  const int64_t pos = (int64_t)a.dims.len(b) + t;
  const KvView& c = which == 0 ? a.k : a.v;
  int64_t row;
  if (c.page_table) {
    const int64_t slot = pos >> c.page_shift;
    if (slot >= c.max_pages) return;  // no page for this position: nothing is written
    const int page = clampi(c.page_table[(int64_t)b * c.max_pages + slot], 0, c.num_pages - 1);
    row = (int64_t)page * c.stride_page + (pos & ((1 << c.page_shift) - 1)) * c.stride_n;
  } else {
    if (pos >= c.capacity) return;
    row = (int64_t)b * c.stride_b + pos * c.stride_n;
  }
  const uint16_t* src = (which == 0 ? a.k_new : a.v_new) + (int64_t)b * (which == 0 ? a.k_sb : a.v_sb) +
                        (int64_t)t * (which == 0 ? a.k_st : a.v_st) + (int64_t)h * (which == 0 ? a.k_sh : a.v_sh);
  uint16_t* dst = const_cast<uint16_t*>(c.data) + row + (int64_t)h * c.stride_h;
  *reinterpret_cast<u32x4*>(dst + 8 * chunk) = *reinterpret_cast<const u32x4*>(src + 8 * chunk);
}

hipError_t launch_kv_append(const KvAppendArgs& a, hipStream_t stream) {
  const int64_t threads = 2 * (int64_t)a.batch * a.dims.nq_max * a.num_kv_heads * (a.head_dim / 8);
  if (threads == 0) return hipSuccess;
  const int64_t blocks = (threads + kKvThreads - 1) / kKvThreads;
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)blocks), dim3(kKvThreads), 0, stream, a);
  return hipGetLastError();
}

__global__ __launch_bounds__(kKvThreads) void kv_commit_kernel(int32_t* seq_lens, const int32_t* accepted,
                                                               const int32_t* n_query, int nq_max, int batch) {
  const int b = blockIdx.x * kKvThreads + threadIdx.x;
  if (b >= batch) return;
  const int T = n_query ? clampi(n_query[b], 0, nq_max) : nq_max;
  seq_lens[b] += clampi(accepted[b], 0, T);
}

hipError_t launch_kv_commit(int32_t* seq_lens, const int32_t* accepted, const int32_t* n_query, int nq_max,
                            int batch, hipStream_t stream) {
  if (batch == 0) return hipSuccess;
  hipLaunchKernelGGL(kv_commit_kernel, dim3((batch + kKvThreads - 1) / kKvThreads), dim3(kKvThreads), 0, stream,
                     seq_lens, accepted, n_query, nq_max, batch);
  return hipGetLastError();
}

}  // namespace dustin
