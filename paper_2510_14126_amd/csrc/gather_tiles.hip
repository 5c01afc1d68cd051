// Data-movement reference for the decode kernels: reads the K and V tiles of
// a list of token spans the way a decode work item does, with no arithmetic.
// One workgroup per (span, KV head), the head fastest (so a head stays on one
// XCD, as in the decode grids); its four wavefronts take the span's 16-token
// blocks round-robin through a ring that keeps NIF tiles of K and V in flight
// each (two suit short spans, where deeper rings only lengthen the memory
// queues; four suit long ones), and fold every 32-bit word they read with XOR so that no load
// is dead.  Every tile is read once, 1 KiB of contiguous rows per load
// instruction, with the streaming cache hint (kLoadStreaming), like the
// tiles a decode step reads once.  The time of one launch over the tiles a
// decode step reads is what that access pattern costs on the memory system
// alone.
#include "kernels.h"
#include "pa_device.h"

namespace pa {
namespace {

constexpr int kWavesPerGroup = 4;
constexpr int kIdChunk = 1024;     // block ids staged in LDS at a time

template <int D, int NIF>
__global__ void __launch_bounds__(64 * kWavesPerGroup)
gather_tiles_kernel(const uint16_t* __restrict__ kp, const uint16_t* __restrict__ vp,
                    int num_blocks, int num_kv_heads, const int32_t* __restrict__ block_tables,
                    int bt_stride, int batch, const int32_t* __restrict__ spans,
                    uint32_t* __restrict__ sink) {
  constexpr int kTileBytes = 16 * D * 2;
  constexpr int kPerLane = kTileBytes / (64 * 16);   // 16-byte loads per lane: 2 (D = 64), 4 (D = 128)
  __shared__ int32_t ids[kIdChunk];
  const int g = blockIdx.x % num_kv_heads;
  const int s = blockIdx.x / num_kv_heads;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // device data: clamped into the batch and the table row
  const int row_tokens = 16 * bt_stride;
  int seq = spans[3 * s];
  seq = seq < 0 ? 0 : (seq >= batch ? batch - 1 : seq);
  int start = spans[3 * s + 1];
  start = (start < 0 ? 0 : (start > row_tokens ? row_tokens : start)) & ~15;
  int end = spans[3 * s + 2];
  end = end < start ? start : (end > row_tokens ? row_tokens : end);
  const int nblk = (end - start + 15) >> 4;
  const int32_t* bt = block_tables + (size_t)seq * bt_stride + (start >> 4);
  const size_t blk_stride = (size_t)num_kv_heads * kTileBytes;
  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(kp) + (size_t)g * kTileBytes;
  const uint8_t* vbase = reinterpret_cast<const uint8_t*>(vp) + (size_t)g * kTileBytes;

  uint32_t acc = 0;
  for (int c0 = 0; c0 < nblk; c0 += kIdChunk) {
    const int cn = min(kIdChunk, nblk - c0);
    __syncthreads();                           // the previous chunk's ids are no longer read
    for (int t = threadIdx.x; t < cn; t += 64 * kWavesPerGroup) {
      const int id = bt[c0 + t];
      ids[t] = id < 0 ? 0 : (id >= num_blocks ? num_blocks - 1 : id);
    }
    __syncthreads();
    // Tile i of the chunk; past the chunk the descriptor is empty (0 bytes),
    // so the load returns zeros without touching memory and every path
    // through the ring issues the same loads.
    auto load = [&](uint4 (&dst)[2][kPerLane], int i) {
      const bool ok = i < cn;
      const size_t id = (size_t)__builtin_amdgcn_readfirstlane(ids[ok ? i : 0]);
      const int bytes = ok ? kTileBytes : 0;
      const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint8_t*>(kbase + id * blk_stride), 0, bytes, kBufferDescWord3);
      const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint8_t*>(vbase + id * blk_stride), 0, bytes, kBufferDescWord3);
#pragma unroll
      for (int u = 0; u < kPerLane; ++u) {
        const auto k = __builtin_amdgcn_raw_buffer_load_b128(rk, (u * 64 + lane) * 16, 0, kLoadStreaming);
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(rv, (u * 64 + lane) * 16, 0, kLoadStreaming);
        dst[0][u] = make_uint4(k[0], k[1], k[2], k[3]);
        dst[1][u] = make_uint4(v[0], v[1], v[2], v[3]);
      }
    };
    auto fold = [&](const uint4 (&src)[2][kPerLane]) {
#pragma unroll
      for (int kv = 0; kv < 2; ++kv)
#pragma unroll
        for (int u = 0; u < kPerLane; ++u)
          acc ^= src[kv][u].x ^ src[kv][u].y ^ src[kv][u].z ^ src[kv][u].w;
    };
    int i = wave;
    if (i >= cn) continue;
    uint4 ring[NIF][2][kPerLane];
    int ld = i;
#pragma unroll
    for (int r = 0; r < NIF - 1; ++r) {
      load(ring[r], ld);
      ld += kWavesPerGroup;
    }
    bool done = false;
    while (!done) {
#pragma unroll
      for (int r = 0; r < NIF; ++r) {
        if (!done) {
          load(ring[(r + NIF - 1) % NIF], ld);
          ld += kWavesPerGroup;
          fold(ring[r]);
          i += kWavesPerGroup;
          done = i >= cn;
        }
      }
    }
  }
  // XOR over the wavefront's lanes.
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, m, 64);
  if (lane == 0) sink[(size_t)blockIdx.x * kWavesPerGroup + wave] = acc;
}

}  // namespace

hipError_t launch_gather_tiles(const void* k_pool, const void* v_pool, int num_blocks,
                               int num_kv_heads, int head_dim, const int32_t* block_tables,
                               int bt_stride, int batch, const int32_t* spans, int num_spans,
                               int tiles_in_flight, uint32_t* sink, hipStream_t stream) {
  const int64_t grid = (int64_t)num_spans * num_kv_heads;
  if (grid == 0) return hipSuccess;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  const auto* kp = static_cast<const uint16_t*>(k_pool);
  const auto* vp = static_cast<const uint16_t*>(v_pool);
  const dim3 grd((unsigned)grid), blk(64 * kWavesPerGroup);
#define PA_GATHER_LAUNCH(D, NIF)                                                              \
  hipLaunchKernelGGL((gather_tiles_kernel<D, NIF>), grd, blk, 0, stream, kp, vp, num_blocks, \
                     num_kv_heads, block_tables, bt_stride, batch, spans, sink)
  if (head_dim == 128 && tiles_in_flight == 2)
    PA_GATHER_LAUNCH(128, 2);
  else if (head_dim == 128 && tiles_in_flight == 4)
    PA_GATHER_LAUNCH(128, 4);
  else if (head_dim == 64 && tiles_in_flight == 2)
    PA_GATHER_LAUNCH(64, 2);
  else if (head_dim == 64 && tiles_in_flight == 4)
    PA_GATHER_LAUNCH(64, 4);
  else
    return hipErrorInvalidValue;
#undef PA_GATHER_LAUNCH
  return hipGetLastError();
}

}  // namespace pa
