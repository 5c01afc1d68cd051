// Extend (chunked prefill) attention over the paged cache: kernel entry
// point.  The algorithm lives in extend_mfma_body (mfma_body.h).
#include "mfma_body.h"

namespace pa {
namespace {

template <int G>
__global__ void __launch_bounds__(64 * mfma::kWaves) __attribute__((amdgpu_waves_per_eu(2, 8)))
extend_mfma_kernel(const ExtendParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[mfma::kExtendLdsBytes];
  mfma::extend_mfma_body<G>(p, blockIdx.x, (lds_u8_t*)smem);
}

}  // namespace

hipError_t launch_extend(const ExtendParams& p, int group, hipStream_t stream) {
  const int64_t grid = (int64_t)p.batch * p.groups * p.num_kv_heads;
  if (grid == 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  if (group == 4)
    hipLaunchKernelGGL(extend_mfma_kernel<4>, dim3((unsigned)grid), dim3(64 * mfma::kWaves), 0, stream, p);
  else if (group == 8)
    hipLaunchKernelGGL(extend_mfma_kernel<8>, dim3((unsigned)grid), dim3(64 * mfma::kWaves), 0, stream, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa
