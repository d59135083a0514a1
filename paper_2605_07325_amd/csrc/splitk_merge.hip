// Split-K merge.  Each key split s produced a normalised partial output o_s
// and its log-sum-exp lse_s over that split's keys.  Softmax over the union
// of the key sets is exactly
//     lse = ln sum_s exp(lse_s),   o = sum_s exp(lse_s - lse) * o_s,
// so the merge is a rearrangement of the paper's attention sums, not an
// approximation.  Splits with no visible key carry lse_s = -inf and drop out.
//
// One thread produces 4 consecutive output elements of one (token, head) row.
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

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int dtype_bf16, hipStream_t stream) {
  const int64_t total = (int64_t)a.total_q * a.Hq * (a.d / 4);
  if (total == 0) return hipSuccess;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  if (dtype_bf16) hipLaunchKernelGGL(splitk_merge_kernel<true>, dim3(blocks), dim3(256), 0, stream, a);
  else hipLaunchKernelGGL(splitk_merge_kernel<false>, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace csr
