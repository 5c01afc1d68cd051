// One-launch shared-prefix (cascade) step: some workgroups run the
// shared-prefix pass (matrix-core tiles over all query rows) and, with a
// second level, the pass over each group's shared tokens (tiles over the
// group's rows); the others run the per-sequence decode over the tokens
// after what is shared.  All write disjoint (o, lse) partials, so they need
// no synchronisation.  Shared and per-sequence work
// alternate in runs of num_kv_heads workgroups (with a phase flip every 8
// runs, see below), so every CU holds some of each at once: the L2-fed prefix work overlaps the HBM-fed per-sequence work
// instead of preceding it, and workgroup i still serves KV head
// i % num_kv_heads, which keeps each head on one XCD (the dispatcher deals
// workgroups to the XCDs round-robin).
#include "mfma_body.h"
#include "valu_body.h"

namespace pa {
namespace {

constexpr int kMax(int a, int b) { return a > b ? a : b; }
constexpr int kCascadeLds = kMax(kMax(mfma::kPrefixLdsBytes, mfma::kLdsBytes),
                                 valu::valu_lds_bytes<128, 4, PA_VALU_WAVES>());

static_assert(PA_VALU_WAVES == mfma::kWaves, "both halves use the same workgroup size");

// Tiles in flight per wavefront of the per-sequence half: its work items are
// the short tails after the prefix, where a 2-deep ring measured ~2% faster
// than the 3-deep ring of the standalone kernel.
constexpr int kCascadeValuNbuf = 2;

template <int G, bool TRACE, bool APPEND>
__global__ void __launch_bounds__(64 * mfma::kWaves) __attribute__((amdgpu_waves_per_eu(2, 8)))
cascade_kernel(const PrefixParams pp, const DecodeParams dp, int prefix_runs, int group_runs,
               int decode_runs) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kCascadeLds];
  lds_u8_t* lds = (lds_u8_t*)smem;
  // Run r = blockIdx / Hkv: while both kinds remain, even runs are shared
  // runs (the prefix partitions, then the groups) and odd runs decode runs;
  // then the longer kind continues alone.
  const int hkv = dp.num_kv_heads;
  const int run = blockIdx.x / hkv;
  const int g = blockIdx.x - run * hkv;
  const int shared_runs = prefix_runs + group_runs;
  const int both = min(shared_runs, decode_runs);
  bool shared;
  int idx;
  if (3 * shared_runs >= decode_runs) {
    // Shared work at least a third of the decode runs (the fixer batch with
    // its request groups): all shared runs first measured 2% faster than
    // interleaving them; a run of consecutive shared runs reaches every
    // shader engine.
    shared = run < shared_runs;
    idx = shared ? run : run - shared_runs;
  } else if (run < 2 * both) {
    // Alternate, flipping the phase every 8 runs.  Each XCD hands its
    // workgroups to its four shader engines in a fixed cycle and waits for
    // the next engine in the cycle to have room, so a plain alternation would
    // put every shared run on two engines of each XCD and every decode run on
    // the other two (measured: dispatch then stalls on the engines that hold
    // the longest items while the others sit half empty).
    const int blk = run >> 3, w = run & 7;
    shared = ((w ^ blk) & 1) == 0;
    idx = (blk << 2) + (w >> 1);
  } else {
    shared = shared_runs > decode_runs;
    idx = both + (run - 2 * both);
  }
  if (shared) {
    if (idx < prefix_runs)
      mfma::prefix_mfma_body<G, TRACE>(pp, idx * hkv + g, lds);
    else
      mfma::group_mfma_body<G, TRACE>(pp, (idx - prefix_runs) * hkv + g, lds);
    return;
  }
  const int wg = idx * hkv + g;
  if constexpr (G == 4) {
    valu::decode_valu_body<128, 4, PA_VALU_WAVES, kCascadeValuNbuf, TRACE, /*STREAM=*/true, APPEND>(
        dp, wg, lds);
  } else {
    mfma::decode_mfma_body<TRACE, /*STREAM=*/true, APPEND>(dp, wg, lds);
  }
}

}  // namespace

hipError_t launch_cascade(const PrefixParams& pp, const DecodeParams& dp, int group, bool trace,
                          hipStream_t stream) {
  const int64_t rows = (int64_t)pp.batch * group;
  const int64_t row_groups = (rows + mfma::kPrefixRowsPerWg - 1) / mfma::kPrefixRowsPerWg;
  // Both grids are whole runs of num_kv_heads workgroups (the KV head is the
  // fastest index of both).
  if (pp.num_kv_heads != dp.num_kv_heads) return hipErrorInvalidValue;
  const int64_t prefix_runs = (int64_t)pp.prefix_parts * row_groups;
  const int64_t group_runs = pp.num_groups > 0 ? pp.num_groups : 0;
  const int64_t decode_runs = decode_items(dp);
  const int64_t grid = (prefix_runs + group_runs + decode_runs) * dp.num_kv_heads;
  if (grid == 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(64 * mfma::kWaves), 0, stream, pp, dp,
                       (int)prefix_runs, (int)group_runs, (int)decode_runs);
  };
  // The trace kernels have no fused append.
  const bool append = dp.k_new != nullptr && !trace;
  if (group == 4)
    trace ? go(cascade_kernel<4, true, false>)
          : (append ? go(cascade_kernel<4, false, true>) : go(cascade_kernel<4, false, false>));
  else if (group == 8)
    trace ? go(cascade_kernel<8, true, false>)
          : (append ? go(cascade_kernel<8, false, true>) : go(cascade_kernel<8, false, false>));
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa
