// Work order for ragged batches: which attention unit each workgroup runs.
//
// A unit is (sequence b, kv head g, key split s, row tile m); its run time is
// proportional to the key tiles it scans, ceil((L_b + rows seen) / 64) / nsplit,
// so in a ragged batch units differ by an order of magnitude.  The lengths are
// device-side (cache_seqlens, cu_seqlens_q), so the order is formed on the
// device, by one workgroup, before the attention launch:
//  * the row tiles of a group (b, g) share one K/V stream; they are cut into
//    subgroups of up to K consecutive row tiles, and a subgroup stays on one
//    XCD (its L2 serves every row tile of the subgroup).  Whole groups would be
//    too coarse: one long sequence's group can exceed an XCD's fair share;
//  * subgroups are ranked by per-unit length, longest first, and each goes to
//    the XCD with the least work so far among those with room left (greedy
//    longest-processing-time assignment);
//  * workgroup slot w runs on XCD w % 8 (the hardware deals workgroups to the
//    XCDs round robin); XCD x's slots w = 8i + x take its subgroups' units in
//    rank order, so every XCD dispatches its longest units first;
//  * slots left over hold -1 and their workgroups exit at once.
#include "kernels.h"

namespace csr {

namespace {

constexpr int kPlanThreads = 256;

// Subgroups the shared-memory arrays are sized for.
__host__ __device__ __forceinline__ int subgroup_cap(int batch, int Hkv, int mtiles, int K) {
  return batch * Hkv * ((mtiles + K - 1) / K);
}

__global__ void __launch_bounds__(kPlanThreads) plan_units_kernel(PlanArgs p) {
  extern __shared__ int smem[];
  const int ng = p.batch * p.Hkv;
  const int K = p.rt_per_sub;
  const int cap = subgroup_cap(p.batch, p.Hkv, p.mtiles, K);
  int* gfirst = smem;             // [ng + 1] first subgroup of each group (prefix sums)
  int* slen = gfirst + ng + 1;    // per-unit key tiles of the subgroup's longest row tile
  int* sunits = slen + cap;       // units of each subgroup
  int* sgrp = sunits + cap;       // group of each subgroup
  int* by_rank = sgrp + cap;      // subgroup of each rank
  int* sslot = by_rank + cap;     // first slot of the subgroup in its XCD's queue
  int* sxcd = sslot + cap;
  const int tid = threadIdx.x;

  for (int w = tid; w < p.slots * 8; w += kPlanThreads) p.order[w] = -1;

  for (int i = tid; i < ng; i += kPlanThreads) {
    const int b = i / p.Hkv;
    const int rows = (p.cu_q[b + 1] - p.cu_q[b]) * p.G;
    const int mt_active = (rows + p.bm - 1) / p.bm;
    gfirst[i + 1] = (mt_active + K - 1) / K;
  }
  __syncthreads();
  if (tid == 0) {
    gfirst[0] = 0;
    for (int i = 1; i <= ng; ++i) gfirst[i] += gfirst[i - 1];
  }
  __syncthreads();
  const int nsg = gfirst[ng];  // <= cap: mt_active <= mtiles

  for (int i = tid; i < ng; i += kPlanThreads) {
    const int b = i / p.Hkv;
    const int n = p.cu_q[b + 1] - p.cu_q[b];
    const int L = p.cache_len ? p.cache_len[b] : 0;
    const int rows = n * p.G;
    const int mt_active = (rows + p.bm - 1) / p.bm;
    for (int c = 0; c < gfirst[i + 1] - gfirst[i]; ++c) {
      const int sg = gfirst[i] + c;
      const int r1 = min((c + 1) * K, mt_active);  // row tiles [c K, r1), counted from the first
      const int m_last = min(r1 * p.bm, rows) - 1;
      const int tiles = (L + m_last / p.G + 1 + 63) / 64;
      slen[sg] = (tiles + p.nsplit - 1) / p.nsplit;
      sunits[sg] = (r1 - c * K) * p.nsplit;
      sgrp[sg] = i;
    }
  }
  __syncthreads();
  // Rank: longer first, ties by subgroup index (a permutation of 0 .. nsg-1).
  for (int s = tid; s < nsg; s += kPlanThreads) {
    int r = 0;
    for (int j = 0; j < nsg; ++j) r += (slen[j] > slen[s]) || (slen[j] == slen[s] && j < s);
    by_rank[r] = s;
  }
  __syncthreads();
  if (tid == 0) {
    long long load[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int count[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int r = 0; r < nsg; ++r) {
      const int s = by_rank[r];
      int best = -1;
      for (int x = 0; x < 8; ++x)
        if (count[x] + sunits[s] <= p.slots && (best < 0 || load[x] < load[best])) best = x;
      if (best < 0) best = 0;  // unreachable with the host's slot bound; writes below stay in range
      sxcd[s] = best;
      sslot[s] = count[best];
      count[best] += sunits[s];
      load[best] += (long long)sunits[s] * slen[s];
    }
  }
  __syncthreads();
  // Units of each subgroup, later row tiles first (they see a few more keys).
  for (int s = tid; s < nsg; s += kPlanThreads) {
    const int i = sgrp[s];
    const int b = i / p.Hkv, g = i - b * p.Hkv;
    const int r0 = (s - gfirst[i]) * K;
    const int nrt = sunits[s] / p.nsplit;
    for (int k = 0; k < sunits[s]; ++k) {
      const int slot = sslot[s] + k;
      if (slot >= p.slots) break;
      const int mt = r0 + nrt - 1 - k / p.nsplit;  // row tile, counted from the first
      const int sp = k % p.nsplit;
      // the attention kernel's unit numbering (row tiles stored reversed)
      p.order[8 * slot + sxcd[s]] = ((b * p.Hkv + g) * p.nsplit + sp) * p.mtiles + (p.mtiles - 1 - mt);
    }
  }
}

}  // namespace

int plan_subgroup_rows(int batch, int Hkv, int mtiles) {
  // at most ~1024 + batch * Hkv subgroups: the shared arrays stay under 64 KB
  const int64_t need = ((int64_t)batch * Hkv * mtiles + 1023) / 1024;
  return (int)(need > 8 ? need : 8);
}

int plan_smem_bytes(int batch, int Hkv, int mtiles, int rt_per_sub) {
  return (batch * Hkv + 1 + 6 * subgroup_cap(batch, Hkv, mtiles, rt_per_sub)) * (int)sizeof(int);
}

hipError_t launch_plan(const PlanArgs& p, hipStream_t stream) {
  hipLaunchKernelGGL(plan_units_kernel, dim3(1), dim3(kPlanThreads),
                     plan_smem_bytes(p.batch, p.Hkv, p.mtiles, p.rt_per_sub), stream, p);
  return hipGetLastError();
}

}  // namespace csr
