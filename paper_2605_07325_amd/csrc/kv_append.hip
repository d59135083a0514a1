// Paged KV append as a launch of its own (the per-item body is shared with the
// split-K merge launch, which carries the append when a call merges splits).
// The whole ragged batch is one launch.
#include "append_rows.h"

namespace csr {

namespace {

__global__ void __launch_bounds__(256) kv_append_kernel(AppendArgs a) {
  append_item(a, (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, hipStream_t stream) {
  const int64_t total = append_items(a);
  if (total == 0) return hipSuccess;
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace csr
