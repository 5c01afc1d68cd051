// Split-KV paged decode attention on VALU dot products: kernel entry points.
// The algorithm lives in valu_body.h.
#include "valu_body.h"

namespace pa {
namespace {

template <int D, int G, int W, int NBUF, bool TRACE, bool STREAM, bool APPEND>
__global__ void __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(PA_VALU_MIN_WAVES, 8)))
decode_valu_kernel(const DecodeParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[valu::valu_lds_bytes<D, G, W>()];
  valu::decode_valu_body<D, G, W, NBUF, TRACE, STREAM, APPEND>(p, blockIdx.x, (lds_u8_t*)smem);
}

// The trace kernels keep the default cache policy (the hint changes no index)
// and have no fused append.
template <int D, int G, bool TRACE>
hipError_t launch_t(const DecodeParams& p, hipStream_t stream) {
  constexpr int W = PA_VALU_WAVES;
  constexpr int NBUF = PA_VALU_NBUF;
  const int64_t grid = decode_items(p) * p.num_kv_heads;
  if (grid == 0) return hipSuccess;
  const dim3 grd((unsigned)grid), blk(64 * W);
  if constexpr (TRACE) {
    hipLaunchKernelGGL((decode_valu_kernel<D, G, W, NBUF, true, false, false>), grd, blk, 0, stream, p);
  } else {
    const bool append = p.k_new != nullptr;
    if (p.stream_tiles && append)
      hipLaunchKernelGGL((decode_valu_kernel<D, G, W, NBUF, false, true, true>), grd, blk, 0, stream, p);
    else if (p.stream_tiles)
      hipLaunchKernelGGL((decode_valu_kernel<D, G, W, NBUF, false, true, false>), grd, blk, 0, stream, p);
    else if (append)
      hipLaunchKernelGGL((decode_valu_kernel<D, G, W, NBUF, false, false, true>), grd, blk, 0, stream, p);
    else
      hipLaunchKernelGGL((decode_valu_kernel<D, G, W, NBUF, false, false, false>), grd, blk, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace

// GQA groups of 8 at head_dim 128 run on matrix cores (decode_mfma.hip).
hipError_t launch_decode_valu(const DecodeParams& p, int head_dim, int group, bool trace,
                              hipStream_t stream) {
  if (head_dim == 128 && group == 4)
    return trace ? launch_t<128, 4, true>(p, stream) : launch_t<128, 4, false>(p, stream);
  if (head_dim == 64 && group == 4)
    return trace ? launch_t<64, 4, true>(p, stream) : launch_t<64, 4, false>(p, stream);
  if (head_dim == 64 && group == 8)
    return trace ? launch_t<64, 8, true>(p, stream) : launch_t<64, 8, false>(p, stream);
  return hipErrorInvalidValue;
}

}  // namespace pa
