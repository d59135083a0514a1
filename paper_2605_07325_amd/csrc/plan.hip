// Work order for ragged batches: which attention unit each workgroup runs.
//
// A unit is (sequence b, kv head g, key split s, row tile m); its run time is
// proportional to the key tiles it scans, ceil((L_b + rows seen) / 64) / nsplit,
// so in a ragged batch units differ by an order of magnitude.  The lengths are
// device-side (cache_seqlens, cu_seqlens_q), so the order is formed on the
// device, by one workgroup, before the attention launch:
//  * the row tiles of a group (b, g) share one K/V stream; they are cut into
//    subgroups of up to K consecutive row tiles (K = 4 unless the batch is
//    very large), and a subgroup stays on one XCD (its L2 serves every row
//    tile of the subgroup).  Whole groups would be too coarse: one long
//    sequence's group can exceed an XCD's fair share;
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
  int* rk_units = sxcd + cap;     // units and per-unit length in rank order
  int* rk_len = rk_units + cap;
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
    const int ls = slen[s];
    int r = 0;
#pragma unroll 8
    for (int j = 0; j < nsg; ++j) r += (slen[j] > ls) || (slen[j] == ls && j < s);
    by_rank[r] = s;
    rk_units[r] = sunits[s];
    rk_len[r] = ls;
  }
  __syncthreads();
  if (tid < 8) {
    // Greedy assignment, one lane per XCD: lane x holds XCD x's unit count
    // and work; each subgroup goes to the lane with the least work among
    // those with room (ties: the lower XCD), found with three xor shuffles
    // over keys (work << 3 | x).
    const int x = tid;
    int count = 0;
    unsigned long long load = 0;
    for (int r = 0; r < nsg; ++r) {
      const int su = rk_units[r];
      const unsigned long long key =
          count + su <= p.slots ? (load << 3) | (unsigned long long)x : ~0ull;
      unsigned long long m = key;
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) {
        const unsigned long long other = __shfl_xor(m, o, 8);
        m = other < m ? other : m;
      }
      // (no XCD with room is unreachable with the host's slot bound: XCD 0 then)
      const int best = m == ~0ull ? 0 : (int)(m & 7);
      if (x == best) {
        const int s = by_rank[r];
        sxcd[s] = best;
        sslot[s] = count;
        count += su;
        load += (unsigned long long)su * (unsigned long long)rk_len[r];
      }
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
  // 4 row tiles (measured on the 8-sequence ragged batch: 4 beat 1, 2, 8, 16
  // and 32), more when needed to keep at most 768 + batch * Hkv <= 1792
  // subgroups (the host plans batches of at most 1024 groups): the shared
  // arrays (8 ints per subgroup) then stay under 64 KB and the ranking's cost,
  // quadratic in the subgroup count, stays small
  const int64_t need = ((int64_t)batch * Hkv * mtiles + 767) / 768;
  return (int)(need > 4 ? need : 4);
}

int plan_smem_bytes(int batch, int Hkv, int mtiles, int rt_per_sub) {
  return (batch * Hkv + 1 + 8 * subgroup_cap(batch, Hkv, mtiles, rt_per_sub)) * (int)sizeof(int);
}

hipError_t launch_plan(const PlanArgs& p, hipStream_t stream) {
  hipLaunchKernelGGL(plan_units_kernel, dim3(1), dim3(kPlanThreads),
                     plan_smem_bytes(p.batch, p.Hkv, p.mtiles, p.rt_per_sub), stream, p);
  return hipGetLastError();
}

}  // namespace csr
