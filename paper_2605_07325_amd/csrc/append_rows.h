// Paged KV append body shared by the stand-alone append launch and the split-K
// merge launch that carries the append of short chunks (chunk keys and values
// copied bit for bit into cache positions L_b .. L_b + n_b - 1: append-only
// growth, Theorem 2).
//
// Work item `gid` moves one 16-byte chunk of one (token, kv head) row of K and
// of V, so a 64-lane wave writes whole rows with 16-byte stores.  A token finds
// its sequence by binary search over cu_seqlens_q.  Nothing outside the
// destination slots is written; a row whose page id is out of range (a broken
// caller contract) is dropped.
#pragma once

#include "kernels.h"

namespace csr {

__device__ __forceinline__ int append_find_sequence(const int32_t* __restrict__ cu, int batch, int tok) {
  int lo = 0, hi = batch - 1;  // largest b with cu[b] <= tok
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (__ldg(cu + mid) <= tok) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Work items of one append: total_q * Hkv * row_chunks.
__host__ __device__ __forceinline__ int64_t append_items(const AppendArgs& a) {
  return (int64_t)a.total_q * a.Hkv * a.row_chunks;
}

__device__ __forceinline__ void append_item(const AppendArgs& a, int64_t gid) {
  typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
  const int64_t per_token = (int64_t)a.Hkv * a.row_chunks;
  if (gid >= (int64_t)a.total_q * per_token) return;
  const int tok = (int)(gid / per_token);
  const int64_t within = gid - (int64_t)tok * per_token;  // kv head * row_chunks + chunk
  // the source chunks do not depend on the slot lookup: load them first
  const int64_t src = (int64_t)tok * per_token + within;
  const u32x4_t kx = reinterpret_cast<const u32x4_t*>(a.k_new)[src];
  const u32x4_t vx = reinterpret_cast<const u32x4_t*>(a.v_new)[src];
  const int b = append_find_sequence(a.cu_q, a.batch, tok);
  const int64_t pos = (int64_t)(a.cache_len ? __ldg(a.cache_len + b) : 0) + (tok - __ldg(a.cu_q + b));
  const int64_t pidx = pos >> a.log2P;
  const int64_t page = a.block_table ? (int64_t)__ldg(a.block_table + (int64_t)b * a.bt_stride + pidx)
                                     : (int64_t)b * a.bt_stride + pidx;
  if (page < 0 || page >= a.num_pages) return;
  const int64_t slot = (page << a.log2P) + (pos & ((1 << a.log2P) - 1));
  const int64_t dst = slot * per_token + within;  // in 16-byte chunks
  reinterpret_cast<u32x4_t*>(a.k_pool)[dst] = kx;
  reinterpret_cast<u32x4_t*>(a.v_pool)[dst] = vx;
}

}  // namespace csr
