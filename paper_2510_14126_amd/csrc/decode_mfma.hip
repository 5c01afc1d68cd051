// MFMA decode kernels (GQA groups of 8) and the shared-prefix pass: kernel
// entry points.  The algorithms live in mfma_body.h.
#include "mfma_body.h"

namespace pa {
namespace {

using mfma::kWaves;

template <bool TRACE>
__global__ void __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 8)))
decode_mfma_g8_kernel(const DecodeParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[mfma::kLdsBytes];
  mfma::decode_mfma_body<TRACE>(p, blockIdx.x, (lds_u8_t*)smem);
}

template <int G>
__global__ void __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 8)))
prefix_mfma_kernel(const PrefixParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[mfma::kPrefixLdsBytes];
  mfma::prefix_mfma_body<G>(p, blockIdx.x, (lds_u8_t*)smem);
}

}  // namespace

hipError_t launch_prefix_mfma(const PrefixParams& p, int group, hipStream_t stream) {
  const int64_t rows = (int64_t)p.batch * group;
  const int64_t row_groups = (rows + mfma::kPrefixRowsPerWg - 1) / mfma::kPrefixRowsPerWg;
  const int64_t grid = (int64_t)p.prefix_parts * row_groups * p.num_kv_heads;
  if (grid == 0) return hipSuccess;
  if (group == 4)
    hipLaunchKernelGGL(prefix_mfma_kernel<4>, dim3((unsigned)grid), dim3(64 * kWaves), 0, stream, p);
  else if (group == 8)
    hipLaunchKernelGGL(prefix_mfma_kernel<8>, dim3((unsigned)grid), dim3(64 * kWaves), 0, stream, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_decode_mfma(const DecodeParams& p, bool trace, hipStream_t stream) {
  const int64_t grid = decode_items(p) * p.num_kv_heads;
  if (grid == 0) return hipSuccess;
  if (trace)
    hipLaunchKernelGGL(decode_mfma_g8_kernel<true>, dim3((unsigned)grid), dim3(64 * kWaves), 0,
                       stream, p);
  else
    hipLaunchKernelGGL(decode_mfma_g8_kernel<false>, dim3((unsigned)grid), dim3(64 * kWaves), 0,
                       stream, p);
  return hipGetLastError();
}

}  // namespace pa
