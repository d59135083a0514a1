// Split-K merge.  Each key split s produced a normalised partial output o_s
// and its log-sum-exp lse_s over that split's keys.  Softmax over the union
// of the key sets is exactly
//     lse = ln sum_s exp(lse_s),   o = sum_s exp(lse_s - lse) * o_s,
// so the merge is a rearrangement of the paper's attention sums, not an
// approximation.  Splits with no visible key carry lse_s = -inf and drop out.
//
// splitk_merge_kernel: one thread produces 4 consecutive output elements of
// one (token, head) row (many rows); splitk_merge_wide_kernel below covers the
// case of few rows and many splits.
#include "kernels.h"

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

template <bool BF16>
__global__ void __launch_bounds__(256) splitk_merge_kernel(MergeArgs a) {
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
  for (int s = 0; s < a.nsplit; ++s) {
    const float ls = a.part_lse[(int64_t)s * rows + row];
    const float w = expf(ls - ref);
    if (w == 0.f) continue;  // split saw no key of this row: its partial is never read
    const f32x4 p = *reinterpret_cast<const f32x4*>(a.part_o + ((int64_t)s * rows + row) * a.d + 4 * q);
    acc += w * p;
    wsum += w;
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  acc *= inv;
  if (BF16) {
    const u32x2 w = {pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
    *reinterpret_cast<u32x2*>(static_cast<char*>(a.out) + (row * a.d + 4 * q) * 2) = w;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + row * a.d + 4 * q) = acc;
  }
  if (q == 0 && a.lse) a.lse[row] = wsum > 0.f ? ref + logf(wsum) : -INFINITY;
}

// Few rows, many splits (short chunks over a long prefix): one workgroup per
// (token, head) row.  Thread t takes output quad t % (d/4) and every
// (256/(d/4))-th split from t / (d/4); the maximum lse and the partial sums are
// combined through LDS, so no thread walks all splits one load after another.
template <bool BF16>
__global__ void __launch_bounds__(256) splitk_merge_wide_kernel(MergeArgs a) {
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
  red[t] = mx;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] = fmaxf(red[t], red[t + w]);
    __syncthreads();
  }
  const float ref = red[0] == -INFINITY ? 0.f : red[0];
  __syncthreads();
  float wsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = g; s < a.nsplit; s += groups) {
    const float w = expf(a.part_lse[(int64_t)s * rows + row] - ref);
    if (w == 0.f) continue;  // split saw no key of this row
    const f32x4 p = *reinterpret_cast<const f32x4*>(a.part_o + ((int64_t)s * rows + row) * a.d + 4 * q);
    acc += w * p;
    wsum += w;
  }
  part[t] = acc;
  if (q == 0) red[g] = wsum;
  __syncthreads();
  if (g != 0) return;
  float wtot = 0.f;
  for (int i = 0; i < groups; ++i) wtot += red[i];
  for (int i = 1; i < groups; ++i) acc += part[i * quads + q];
  const float inv = wtot > 0.f ? 1.f / wtot : 0.f;
  acc *= inv;
  if (BF16) {
    const u32x2 w = {pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
    *reinterpret_cast<u32x2*>(static_cast<char*>(a.out) + (row * a.d + 4 * q) * 2) = w;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + row * a.d + 4 * q) = acc;
  }
  if (q == 0 && a.lse) a.lse[row] = wtot > 0.f ? ref + logf(wtot) : -INFINITY;
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int dtype_bf16, hipStream_t stream) {
  const int64_t rows = (int64_t)a.total_q * a.Hq;
  const int64_t total = rows * (a.d / 4);
  if (total == 0) return hipSuccess;
  if (total < 32768 && a.nsplit >= 8 && rows < (1ll << 31)) {
    // too few output quads to hide the per-split loads one thread at a time
    if (dtype_bf16) hipLaunchKernelGGL(splitk_merge_wide_kernel<true>, dim3((unsigned)rows), dim3(256), 0, stream, a);
    else hipLaunchKernelGGL(splitk_merge_wide_kernel<false>, dim3((unsigned)rows), dim3(256), 0, stream, a);
    return hipGetLastError();
  }
  const unsigned blocks = (unsigned)((total + 255) / 256);
  if (dtype_bf16) hipLaunchKernelGGL(splitk_merge_kernel<true>, dim3(blocks), dim3(256), 0, stream, a);
  else hipLaunchKernelGGL(splitk_merge_kernel<false>, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace csr
