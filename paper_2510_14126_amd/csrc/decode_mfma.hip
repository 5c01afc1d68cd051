// MFMA decode kernels (GQA groups of 8): kernel entry points.  The
// algorithms live in mfma_body.h; the shared-prefix pass runs inside the
// cascade kernel (cascade.hip).
#include "mfma_body.h"

namespace pa {
namespace {

using mfma::kWaves;

template <bool TRACE, bool STREAM>
__global__ void __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 8)))
decode_mfma_g8_kernel(const DecodeParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[mfma::kLdsBytes];
  mfma::decode_mfma_body<TRACE, STREAM>(p, blockIdx.x, (lds_u8_t*)smem);
}

}  // namespace

hipError_t launch_decode_mfma(const DecodeParams& p, bool trace, hipStream_t stream) {
  const int64_t grid = decode_items(p) * p.num_kv_heads;
  if (grid == 0) return hipSuccess;
  // The trace kernel keeps the default cache policy (the hint changes no index).
  if (trace)
    hipLaunchKernelGGL((decode_mfma_g8_kernel<true, false>), dim3((unsigned)grid), dim3(64 * kWaves),
                       0, stream, p);
  else if (p.stream_tiles)
    hipLaunchKernelGGL((decode_mfma_g8_kernel<false, true>), dim3((unsigned)grid), dim3(64 * kWaves),
                       0, stream, p);
  else
    hipLaunchKernelGGL((decode_mfma_g8_kernel<false, false>), dim3((unsigned)grid),
                       dim3(64 * kWaves), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pa
