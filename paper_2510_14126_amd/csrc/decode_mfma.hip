// MFMA decode kernels (GQA groups of 8): kernel entry points.  The
// algorithms live in mfma_body.h; the shared-prefix pass runs inside the
// cascade kernel (cascade.hip).
#include "mfma_body.h"

namespace pa {
namespace {

using mfma::kWaves;

template <bool TRACE, bool STREAM, bool APPEND>
__global__ void __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 8)))
decode_mfma_g8_kernel(const DecodeParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[mfma::kLdsBytes];
  mfma::decode_mfma_body<TRACE, STREAM, APPEND>(p, blockIdx.x, (lds_u8_t*)smem);
}

}  // namespace

hipError_t launch_decode_mfma(const DecodeParams& p, bool trace, hipStream_t stream) {
  const int64_t grid = decode_items(p) * p.num_kv_heads;
  if (grid == 0) return hipSuccess;
  // The trace kernel keeps the default cache policy (the hint changes no
  // index) and has no fused append.
  const dim3 grd((unsigned)grid), blk(64 * kWaves);
  const bool append = p.k_new != nullptr;
  if (trace)
    hipLaunchKernelGGL((decode_mfma_g8_kernel<true, false, false>), grd, blk, 0, stream, p);
  else if (p.stream_tiles && append)
    hipLaunchKernelGGL((decode_mfma_g8_kernel<false, true, true>), grd, blk, 0, stream, p);
  else if (p.stream_tiles)
    hipLaunchKernelGGL((decode_mfma_g8_kernel<false, true, false>), grd, blk, 0, stream, p);
  else if (append)
    hipLaunchKernelGGL((decode_mfma_g8_kernel<false, false, true>), grd, blk, 0, stream, p);
  else
    hipLaunchKernelGGL((decode_mfma_g8_kernel<false, false, false>), grd, blk, 0, stream, p);
  return hipGetLastError();
}

}  // namespace pa
