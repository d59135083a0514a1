// Paged KV append: the chunk's keys and values are copied bit for bit into
// cache positions L_b .. L_b + n_b - 1 (append-only growth, Theorem 2).
//
// One thread moves one 16-byte chunk of one (token, kv head) row for both K and
// V, so a 64-lane wave writes whole rows with 16-byte stores.  The whole ragged
// batch is one launch; a thread finds its sequence by binary search over
// cu_seqlens_q.  Nothing outside the destination slots is written.
#include "kernels.h"

namespace csr {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int find_sequence(const int32_t* __restrict__ cu, int batch, int tok) {
  int lo = 0, hi = batch - 1;  // largest b with cu[b] <= tok
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (__ldg(cu + mid) <= tok) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__global__ void __launch_bounds__(256) kv_append_kernel(AppendArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per_token = (int64_t)a.Hkv * a.row_chunks;
  const int64_t total = (int64_t)a.total_q * per_token;
  if (gid >= total) return;
  const int tok = (int)(gid / per_token);
  const int64_t within = gid - (int64_t)tok * per_token;  // kv head * row_chunks + chunk
  const int b = find_sequence(a.cu_q, a.batch, tok);
  const int64_t pos = (int64_t)(a.cache_len ? __ldg(a.cache_len + b) : 0) + (tok - __ldg(a.cu_q + b));
  const int64_t pidx = pos >> a.log2P;
  const int64_t page = a.block_table ? (int64_t)__ldg(a.block_table + (int64_t)b * a.bt_stride + pidx)
                                     : (int64_t)b * a.bt_stride + pidx;
  if (page < 0 || page >= a.num_pages) return;  // caller contract violated: drop the row
  const int64_t slot = (page << a.log2P) + (pos & ((1 << a.log2P) - 1));
  const int64_t dst = slot * per_token + within;           // in 16-byte chunks
  const int64_t src = (int64_t)tok * per_token + within;
  const u32x4 kx = reinterpret_cast<const u32x4*>(a.k_new)[src];
  const u32x4 vx = reinterpret_cast<const u32x4*>(a.v_new)[src];
  reinterpret_cast<u32x4*>(a.k_pool)[dst] = kx;
  reinterpret_cast<u32x4*>(a.v_pool)[dst] = vx;
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, hipStream_t stream) {
  const int64_t total = (int64_t)a.total_q * a.Hkv * a.row_chunks;
  if (total == 0) return hipSuccess;
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace csr
