// Work order for ragged batches: which attention unit each workgroup runs.
//
// A unit is (sequence b, kv head g, key split s, row tile m); its run time is
// proportional to the key tiles it scans, ceil((L_b + rows seen) / 64) / nsplit,
// so in a ragged batch units differ by an order of magnitude.  The lengths are
// device-side (cache_seqlens, cu_seqlens_q), so the order is formed on the
// device, by one workgroup, before the attention launch:
//  * groups (b, g) share one K/V stream and stay on one XCD (its L2 serves
//    every row tile of the group); groups are ranked by per-unit length,
//    longest first, and each goes to the XCD with the least work so far among
//    those with room left (greedy longest-processing-time assignment);
//  * workgroup slot w runs on XCD w % 8 (the hardware deals workgroups to the
//    XCDs round robin); XCD x's slots w = 8i + x take its groups' units in
//    rank order, so every XCD dispatches its longest units first;
//  * slots left over hold -1 and their workgroups exit at once.
#include "kernels.h"

namespace csr {

namespace {

constexpr int kPlanThreads = 256;

__global__ void __launch_bounds__(kPlanThreads) plan_units_kernel(PlanArgs p) {
  extern __shared__ int smem[];
  const int ng = p.batch * p.Hkv;
  int* glen = smem;            // per-unit key tiles of each group
  int* gunits = glen + ng;     // units of each group
  int* by_rank = gunits + ng;  // group of each rank
  int* gslot = by_rank + ng;   // first slot of the group in its XCD's queue
  int* gxcd = gslot + ng;
  const int tid = threadIdx.x;

  for (int w = tid; w < p.slots * 8; w += kPlanThreads) p.order[w] = -1;

  for (int i = tid; i < ng; i += kPlanThreads) {
    const int b = i / p.Hkv;
    const int n = p.cu_q[b + 1] - p.cu_q[b];
    const int L = p.cache_len ? p.cache_len[b] : 0;
    const int rows = n * p.G;
    const int mt_active = (rows + p.bm - 1) / p.bm;
    const int tiles = (L + n + 63) / 64;
    glen[i] = (tiles + p.nsplit - 1) / p.nsplit;
    gunits[i] = mt_active * p.nsplit;
  }
  __syncthreads();
  // Rank: longer first, ties by group index (a permutation of 0 .. ng-1).
  for (int i = tid; i < ng; i += kPlanThreads) {
    int r = 0;
    for (int j = 0; j < ng; ++j) r += (glen[j] > glen[i]) || (glen[j] == glen[i] && j < i);
    by_rank[r] = i;
  }
  __syncthreads();
  if (tid == 0) {
    long long load[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int count[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int r = 0; r < ng; ++r) {
      const int i = by_rank[r];
      int best = -1;
      for (int x = 0; x < 8; ++x)
        if (count[x] + gunits[i] <= p.slots && (best < 0 || load[x] < load[best])) best = x;
      if (best < 0) best = 0;  // unreachable with the host's slot bound; writes below stay in range
      gxcd[i] = best;
      gslot[i] = count[best];
      count[best] += gunits[i];
      load[best] += (long long)gunits[i] * glen[i];
    }
  }
  __syncthreads();
  // Units of each group, later row tiles first (they see a few more keys).
  for (int i = tid; i < ng; i += kPlanThreads) {
    const int b = i / p.Hkv, g = i - b * p.Hkv;
    for (int k = 0; k < gunits[i]; ++k) {
      const int slot = gslot[i] + k;
      if (slot >= p.slots) break;
      const int mt = gunits[i] / p.nsplit - 1 - k / p.nsplit;  // row tile, counted from the first
      const int s = k % p.nsplit;
      // the attention kernel's unit numbering (row tiles stored reversed)
      p.order[8 * slot + gxcd[i]] = ((b * p.Hkv + g) * p.nsplit + s) * p.mtiles + (p.mtiles - 1 - mt);
    }
  }
}

}  // namespace

int plan_smem_bytes(int batch, int Hkv) { return 5 * batch * Hkv * (int)sizeof(int); }

hipError_t launch_plan(const PlanArgs& p, hipStream_t stream) {
  hipLaunchKernelGGL(plan_units_kernel, dim3(1), dim3(kPlanThreads), plan_smem_bytes(p.batch, p.Hkv), stream, p);
  return hipGetLastError();
}

}  // namespace csr
