// Measured dense-MFMA ceiling of the device and its shader clock under that
// load: the attention kernel's throughput is quoted against this figure
// beside the published peak.  Benchmark support only; not part of libcsr.
//
// Every wave keeps four independent accumulator chains of
// v_mfma_f32_32x32x16_bf16 busy (two waves per SIMD, one 8-wave workgroup per
// CU, the attention kernel's occupancy).  Each workgroup reads the shader
// clock counter and the 100 MHz constant counter at its start and end, so
// cycles / ticks gives the clock it ran at.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <vector>

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

constexpr int kChains = 4;
constexpr double kFlopsPerMfma = 2.0 * 32 * 32 * 16;

__global__ void __launch_bounds__(512, 1) mfma_loop_kernel(int iters, unsigned long long* cycles,
                                                          unsigned long long* ticks, float* sink) {
  const int lane = threadIdx.x & 63;
  s16x8 ai, bi;
  for (int e = 0; e < 8; ++e) {
    ai[e] = (short)(0x3c00 + ((lane + e) & 7));  // small bf16 values, different per lane
    bi[e] = (short)(0x3b80 + ((lane * 3 + e) & 7));
  }
  const bf16x8 a = __builtin_bit_cast(bf16x8, ai), b = __builtin_bit_cast(bf16x8, bi);
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x16{};
  __syncthreads();
  const unsigned long long c0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  __syncthreads();
  const unsigned long long c1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  if (s == 1234.5f) sink[blockIdx.x] = s;  // keeps the products live
  if (threadIdx.x == 0) {
    cycles[blockIdx.x] = c1 - c0;
    ticks[blockIdx.x] = r1 - r0;
  }
}

}  // namespace

// Runs the loop on `workgroups` workgroups of 8 waves for `iters` iterations
// (after one warm-up launch) on the current device and stream 0.  Outputs: the
// launch time in ms (hipEvents), its dense bf16 FLOP/s, and the median shader
// clock in GHz over the workgroups.  Returns 0, or the HIP error code.
extern "C" int csr_bench_mfma_peak(int workgroups, int iters, double* ms_out, double* flops_per_s_out,
                                   double* clock_ghz_out) {
  if (workgroups < 1 || iters < 1 || !ms_out || !flops_per_s_out || !clock_ghz_out) return (int)hipErrorInvalidValue;
  unsigned long long *cyc = nullptr, *tck = nullptr;
  float* sink = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t err = hipMalloc(&cyc, sizeof(unsigned long long) * workgroups);
  if (err == hipSuccess) err = hipMalloc(&tck, sizeof(unsigned long long) * workgroups);
  if (err == hipSuccess) err = hipMalloc(&sink, sizeof(float) * workgroups);
  if (err == hipSuccess) err = hipEventCreate(&e0);
  if (err == hipSuccess) err = hipEventCreate(&e1);
  float ms = 0.f;
  std::vector<unsigned long long> hc(workgroups), ht(workgroups);
  if (err == hipSuccess) {
    hipLaunchKernelGGL(mfma_loop_kernel, dim3(workgroups), dim3(512), 0, 0, iters / 4 + 1, cyc, tck, sink);
    err = hipGetLastError();
  }
  if (err == hipSuccess) err = hipEventRecord(e0, 0);
  if (err == hipSuccess) {
    hipLaunchKernelGGL(mfma_loop_kernel, dim3(workgroups), dim3(512), 0, 0, iters, cyc, tck, sink);
    err = hipGetLastError();
  }
  if (err == hipSuccess) err = hipEventRecord(e1, 0);
  if (err == hipSuccess) err = hipEventSynchronize(e1);
  if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
  if (err == hipSuccess) err = hipMemcpy(hc.data(), cyc, sizeof(unsigned long long) * workgroups, hipMemcpyDeviceToHost);
  if (err == hipSuccess) err = hipMemcpy(ht.data(), tck, sizeof(unsigned long long) * workgroups, hipMemcpyDeviceToHost);
  if (err == hipSuccess) {
    std::vector<double> ghz(workgroups);
    for (int i = 0; i < workgroups; ++i) ghz[i] = ht[i] ? 0.1 * (double)hc[i] / (double)ht[i] : 0.0;
    std::sort(ghz.begin(), ghz.end());
    *clock_ghz_out = ghz[workgroups / 2];
    *ms_out = ms;
    *flops_per_s_out = (double)workgroups * 8 * (double)iters * kChains * kFlopsPerMfma / (ms * 1e-3);
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (cyc) (void)hipFree(cyc);
  if (tck) (void)hipFree(tck);
  if (sink) (void)hipFree(sink);
  return (int)err;
}
