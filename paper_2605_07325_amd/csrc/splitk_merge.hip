// Split-K merge.  Each key split s produced a normalised partial output o_s
// and its log-sum-exp lse_s over that split's keys.  Softmax over the union
// of the key sets is exactly
//     lse = ln sum_s exp(lse_s),   o = sum_s exp(lse_s - lse) * o_s,
// so the merge is a rearrangement of the paper's attention sums, not an
// approximation.  Splits with no visible key carry lse_s = -inf and drop out
// (their weight is 0; the select keeps whatever their partial holds out).
//
// splitk_merge_kernel: one thread produces 4 consecutive output elements of
// one (token, head) row (many rows); splitk_merge_wide_kernel below covers the
// case of few rows and many splits.  Both merge online: a thread issues the
// loads of KB splits (lse and partial; KB = 4, 8 or 16, the fewest that cover
// the splits one thread handles) before using any of them, then moves its
// running maximum and rescales what it has summed so far, so it waits for one
// memory round trip per KB splits and needs no separate pass for the maximum.
//
// A call that appends and merges carries the append in the same launch:
// workgroups past the merge's own run the append body (append_rows.h).
#include "append_rows.h"

namespace csr {

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// Online weighted sum over splits s0, s0 + step, ... (< nsplit) of one output
// quad: acc = sum_s exp(lse_s - m) o_s and wsum = sum_s exp(lse_s - m) for the
// running maximum m (-inf while every split seen so far is empty).
template <int KB>
__device__ __forceinline__ void accumulate(const MergeArgs& a, int64_t rows, int64_t row, int q, int s0, int step,
                                           float& m, f32x4& acc, float& wsum) {
  for (int sb = s0; sb < a.nsplit; sb += KB * step) {
    float ls[KB];
    f32x4 p[KB];
#pragma unroll
    for (int i = 0; i < KB; ++i) {
      const int s = sb + i * step;
      const bool ok = s < a.nsplit;
      ls[i] = ok ? a.part_lse[(int64_t)s * rows + row] : -INFINITY;
      p[i] = ok ? *reinterpret_cast<const f32x4*>(a.part_o + ((int64_t)s * rows + row) * a.d + 4 * q)
                : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    float mb = m;
#pragma unroll
    for (int i = 0; i < KB; ++i) mb = fmaxf(mb, ls[i]);
    if (mb == -INFINITY) continue;  // nothing but empty splits so far
    const float r = m == -INFINITY ? 0.f : expf(m - mb);
    acc *= r;
    wsum *= r;
    m = mb;
#pragma unroll
    for (int i = 0; i < KB; ++i) {
      const float w = expf(ls[i] - mb);
      const f32x4 c = w * p[i];
      acc += w == 0.f ? f32x4{0.f, 0.f, 0.f, 0.f} : c;
      wsum += w;
    }
  }
}

__device__ __forceinline__ void write_row(const MergeArgs& a, int64_t row, int q, f32x4 acc, float wsum, float m,
                                          bool bf16) {
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  acc *= inv;
  if (bf16) {
    const u32x2 w = {pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
    *reinterpret_cast<u32x2*>(static_cast<char*>(a.out) + (row * a.d + 4 * q) * 2) = w;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + row * a.d + 4 * q) = acc;
  }
  if (q == 0 && a.lse) a.lse[row] = wsum > 0.f ? m + logf(wsum) : -INFINITY;
}

template <bool BF16, int KB>
__global__ void __launch_bounds__(256) splitk_merge_kernel(MergeArgs a, int merge_blocks) {
  if ((int)blockIdx.x >= merge_blocks) {
    append_item(a.append, (int64_t)(blockIdx.x - merge_blocks) * blockDim.x + threadIdx.x);
    return;
  }
  const int quads = a.d >> 2;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t rows = (int64_t)a.total_q * a.Hq;
  if (gid >= rows * quads) return;
  const int64_t row = gid / quads;
  const int q = (int)(gid - row * quads);
  float m = -INFINITY, wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  accumulate<KB>(a, rows, row, q, 0, 1, m, acc, wsum);
  write_row(a, row, q, acc, wsum, m, BF16);
}

// Few rows, many splits (short chunks over a long prefix): one workgroup per
// (token, head) row.  Thread t takes output quad t % (d/4) and every
// (256/(d/4))-th split from t / (d/4); the split groups' running maxima and
// partial sums are combined through LDS.
template <bool BF16, int KB>
__global__ void __launch_bounds__(256) splitk_merge_wide_kernel(MergeArgs a, int merge_blocks) {
  if ((int)blockIdx.x >= merge_blocks) {
    append_item(a.append, (int64_t)(blockIdx.x - merge_blocks) * blockDim.x + threadIdx.x);
    return;
  }
  __shared__ float gmax[256], gsum[256];
  __shared__ f32x4 part[256];
  const int quads = a.d >> 2;
  const int groups = 256 / quads;
  const int t = threadIdx.x;
  const int q = t % quads, g = t / quads;
  const int64_t rows = (int64_t)a.total_q * a.Hq;
  const int64_t row = blockIdx.x;
  float m = -INFINITY, wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  accumulate<KB>(a, rows, row, q, g, groups, m, acc, wsum);
  part[t] = acc;
  if (q == 0) {
    gmax[g] = m;
    gsum[g] = wsum;
  }
  __syncthreads();
  if (g != 0) return;
  float mt = -INFINITY;
  for (int i = 0; i < groups; ++i) mt = fmaxf(mt, gmax[i]);
  float wtot = 0.f;
  f32x4 tot = {0.f, 0.f, 0.f, 0.f};
  if (mt != -INFINITY) {
    for (int i = 0; i < groups; ++i) {
      if (gmax[i] == -INFINITY) continue;  // that group saw only empty splits
      const float r = expf(gmax[i] - mt);
      tot += r * part[i * quads + q];
      wtot += r * gsum[i];
    }
  }
  write_row(a, row, q, tot, wtot, mt, BF16);
}

template <bool WIDE, int KB>
void launch_kb(const MergeArgs& a, int dtype_bf16, unsigned grid, int mb, hipStream_t stream) {
  if constexpr (WIDE) {
    if (dtype_bf16) hipLaunchKernelGGL((splitk_merge_wide_kernel<true, KB>), dim3(grid), dim3(256), 0, stream, a, mb);
    else hipLaunchKernelGGL((splitk_merge_wide_kernel<false, KB>), dim3(grid), dim3(256), 0, stream, a, mb);
  } else {
    if (dtype_bf16) hipLaunchKernelGGL((splitk_merge_kernel<true, KB>), dim3(grid), dim3(256), 0, stream, a, mb);
    else hipLaunchKernelGGL((splitk_merge_kernel<false, KB>), dim3(grid), dim3(256), 0, stream, a, mb);
  }
}

// The batch that covers `per` splits per thread in one round trip (16 at most).
template <bool WIDE>
void launch_sized(const MergeArgs& a, int dtype_bf16, int per, unsigned grid, int mb, hipStream_t stream) {
  if (per <= 4) launch_kb<WIDE, 4>(a, dtype_bf16, grid, mb, stream);
  else if (per <= 8) launch_kb<WIDE, 8>(a, dtype_bf16, grid, mb, stream);
  else launch_kb<WIDE, 16>(a, dtype_bf16, grid, mb, stream);
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int dtype_bf16, hipStream_t stream) {
  const int64_t rows = (int64_t)a.total_q * a.Hq;
  const int64_t total = rows * (a.d / 4);
  const int64_t app_blocks = (append_items(a.append) + 255) / 256;
  if (total == 0 && app_blocks == 0) return hipSuccess;
  if (total < 32768 && a.nsplit >= 8 && rows < (1ll << 31)) {
    // too few output quads to hide the per-split loads one thread at a time
    const int groups = 256 / (a.d / 4);
    launch_sized<true>(a, dtype_bf16, (a.nsplit + groups - 1) / groups, (unsigned)(rows + app_blocks), (int)rows,
                       stream);
    return hipGetLastError();
  }
  const int mb = (int)((total + 255) / 256);
  launch_sized<false>(a, dtype_bf16, a.nsplit, (unsigned)(mb + app_blocks), mb, stream);
  return hipGetLastError();
}

}  // namespace csr
