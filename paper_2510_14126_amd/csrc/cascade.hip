// One-launch shared-prefix (cascade) step: the first `prefix_wgs` workgroups
// run the shared-prefix pass (matrix-core tiles over all query rows), the
// rest run the per-sequence decode over the tokens after the prefix.  Both
// halves write disjoint (o, lse) partials, so they need no synchronisation;
// running them in one grid lets the latency-bound prefix work overlap the
// bandwidth-bound per-sequence work instead of preceding it.
#include "mfma_body.h"
#include "valu_body.h"

namespace pa {
namespace {

constexpr int kCascadeLds =
    mfma::kLdsBytes > valu::valu_lds_bytes<128, 4, PA_VALU_WAVES>()
        ? mfma::kLdsBytes
        : valu::valu_lds_bytes<128, 4, PA_VALU_WAVES>();

static_assert(PA_VALU_WAVES == mfma::kWaves, "both halves use the same workgroup size");

template <int G>
__global__ void __launch_bounds__(64 * mfma::kWaves) __attribute__((amdgpu_waves_per_eu(2, 8)))
cascade_kernel(const PrefixParams pp, const DecodeParams dp, int prefix_wgs) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kCascadeLds];
  lds_u8_t* lds = (lds_u8_t*)smem;
  const int wg = blockIdx.x;
  if (wg < prefix_wgs) {
    mfma::prefix_mfma_body<G>(pp, wg, lds);
  } else if constexpr (G == 4) {
    valu::decode_valu_body<128, 4, PA_VALU_WAVES, PA_VALU_NBUF, false>(dp, wg - prefix_wgs, lds);
  } else {
    mfma::decode_mfma_body<false>(dp, wg - prefix_wgs, lds);
  }
}

}  // namespace

hipError_t launch_cascade(const PrefixParams& pp, const DecodeParams& dp, int group,
                          hipStream_t stream) {
  const int64_t rows = (int64_t)pp.batch * group;
  const int64_t row_groups = (rows + mfma::kPrefixRowsPerWg - 1) / mfma::kPrefixRowsPerWg;
  const int64_t prefix_wgs = (int64_t)pp.prefix_parts * row_groups * pp.num_kv_heads;
  const int64_t decode_wgs = (int64_t)dp.num_parts * dp.batch * dp.num_kv_heads;
  const int64_t grid = prefix_wgs + decode_wgs;
  if (grid == 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  if (group == 4)
    hipLaunchKernelGGL(cascade_kernel<4>, dim3((unsigned)grid), dim3(64 * mfma::kWaves), 0, stream,
                       pp, dp, (int)prefix_wgs);
  else if (group == 8)
    hipLaunchKernelGGL(cascade_kernel<8>, dim3((unsigned)grid), dim3(64 * mfma::kWaves), 0, stream,
                       pp, dp, (int)prefix_wgs);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa
