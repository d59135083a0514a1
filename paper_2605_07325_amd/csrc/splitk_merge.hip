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
// case of few rows and many splits.  Both read the partials of 8 splits with
// independent loads before using any of them, so a thread waits for one
// memory round trip per 8 splits, not two per split.
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

constexpr int kBatch = 8;  // splits whose loads are in flight together

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// Weighted sum over splits s0, s0 + step, ... (< nsplit) of one output quad.
__device__ __forceinline__ void accumulate(const MergeArgs& a, int64_t rows, int64_t row, int q, int s0, int step,
                                           float ref, f32x4& acc, float& wsum) {
  for (int sb = s0; sb < a.nsplit; sb += kBatch * step) {
    float ls[kBatch];
    f32x4 p[kBatch];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int s = sb + i * step;
      const bool ok = s < a.nsplit;
      ls[i] = ok ? a.part_lse[(int64_t)s * rows + row] : -INFINITY;
      p[i] = ok ? *reinterpret_cast<const f32x4*>(a.part_o + ((int64_t)s * rows + row) * a.d + 4 * q)
                : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const float w = expf(ls[i] - ref);
      const f32x4 c = w * p[i];
      acc += w == 0.f ? f32x4{0.f, 0.f, 0.f, 0.f} : c;
      wsum += w;
    }
  }
}

__device__ __forceinline__ void write_row(const MergeArgs& a, int64_t row, int q, f32x4 acc, float wsum, float ref,
                                          bool bf16) {
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  acc *= inv;
  if (bf16) {
    const u32x2 w = {pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
    *reinterpret_cast<u32x2*>(static_cast<char*>(a.out) + (row * a.d + 4 * q) * 2) = w;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + row * a.d + 4 * q) = acc;
  }
  if (q == 0 && a.lse) a.lse[row] = wsum > 0.f ? ref + logf(wsum) : -INFINITY;
}

template <bool BF16>
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
  float mx = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) mx = fmaxf(mx, a.part_lse[(int64_t)s * rows + row]);
  const float ref = mx == -INFINITY ? 0.f : mx;
  float wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  accumulate(a, rows, row, q, 0, 1, ref, acc, wsum);
  write_row(a, row, q, acc, wsum, ref, BF16);
}

// Few rows, many splits (short chunks over a long prefix): one workgroup per
// (token, head) row.  Thread t takes output quad t % (d/4) and every
// (256/(d/4))-th split from t / (d/4); the maximum lse (wave shuffles, then
// LDS across the 4 waves) and the partial sums are combined through LDS.
template <bool BF16>
__global__ void __launch_bounds__(256) splitk_merge_wide_kernel(MergeArgs a, int merge_blocks) {
  if ((int)blockIdx.x >= merge_blocks) {
    append_item(a.append, (int64_t)(blockIdx.x - merge_blocks) * blockDim.x + threadIdx.x);
    return;
  }
  __shared__ float red[256];
  __shared__ f32x4 part[256];
  const int quads = a.d >> 2;
  const int groups = 256 / quads;
  const int t = threadIdx.x;
  const int q = t % quads, g = t / quads;
  const int64_t rows = (int64_t)a.total_q * a.Hq;
  const int64_t row = blockIdx.x;
  float mx = -INFINITY;
  for (int s = t; s < a.nsplit; s += 256) mx = fmaxf(mx, a.part_lse[(int64_t)s * rows + row]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if ((t & 63) == 0) red[t >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float ref = mx == -INFINITY ? 0.f : mx;
  __syncthreads();
  float wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  accumulate(a, rows, row, q, g, groups, ref, acc, wsum);
  part[t] = acc;
  if (q == 0) red[g] = wsum;
  __syncthreads();
  if (g != 0) return;
  float wtot = 0.f;
  for (int i = 0; i < groups; ++i) wtot += red[i];
  for (int i = 1; i < groups; ++i) acc += part[i * quads + q];
  write_row(a, row, q, acc, wtot, ref, BF16);
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int dtype_bf16, hipStream_t stream) {
  const int64_t rows = (int64_t)a.total_q * a.Hq;
  const int64_t total = rows * (a.d / 4);
  const int64_t app_blocks = (append_items(a.append) + 255) / 256;
  if (total == 0 && app_blocks == 0) return hipSuccess;
  if (total < 32768 && a.nsplit >= 8 && rows < (1ll << 31)) {
    // too few output quads to hide the per-split loads one thread at a time
    const int mb = (int)rows;
    const unsigned grid = (unsigned)(rows + app_blocks);
    if (dtype_bf16) hipLaunchKernelGGL(splitk_merge_wide_kernel<true>, dim3(grid), dim3(256), 0, stream, a, mb);
    else hipLaunchKernelGGL(splitk_merge_wide_kernel<false>, dim3(grid), dim3(256), 0, stream, a, mb);
    return hipGetLastError();
  }
  const int mb = (int)((total + 255) / 256);
  const unsigned grid = (unsigned)(mb + app_blocks);
  if (dtype_bf16) hipLaunchKernelGGL(splitk_merge_kernel<true>, dim3(grid), dim3(256), 0, stream, a, mb);
  else hipLaunchKernelGGL(splitk_merge_kernel<false>, dim3(grid), dim3(256), 0, stream, a, mb);
  return hipGetLastError();
}

}  // namespace csr
