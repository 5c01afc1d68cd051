// Launchers that launch nothing, for the host-only sanitizer build of the C
// ABI layer: every call reports "not supported", so an entry point whose
// validation passes returns PA_EHIP without touching a GPU.
#include "kernels.h"

namespace pa {
hipError_t launch_decode_valu(const DecodeParams&, int, int, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_decode_mfma(const DecodeParams&, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_cascade(const PrefixParams&, const DecodeParams&, int, bool, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_reduce(const ReduceParams&, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_extend(const ExtendParams&, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_append(const AppendParams&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_stream_copy(const void*, void*, size_t, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_gather_tiles(const void*, const void*, int, int, int, const int32_t*, int, int,
                               const int32_t*, int, int, uint32_t*, hipStream_t) {
  return hipErrorNotSupported;
}
}  // namespace pa
