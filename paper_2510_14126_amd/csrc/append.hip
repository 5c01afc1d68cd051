// Append a decode step's K and V rows to the paged pools.
//
// Token t = ctx_b - 1 of sequence b lives in row t % 16 of physical block
// block_tables[b][t / 16]; for every KV head g its D-wide K row and V row
// are copied from k_new[b][g] / v_new[b][g].  One workgroup per sequence
// moves the 2 * Hkv * D bf16 values in 16-byte chunks: each destination row
// is D * 2 contiguous bytes of the pool, so every chunk store is a full
// aligned 16-byte vector store.
#include "kernels.h"

namespace pa {
namespace {

constexpr int kAppendThreads = 128;

__global__ void __launch_bounds__(kAppendThreads) append_kernel(const AppendParams p) {
  const int b = blockIdx.x;
  const int cap = 16 * p.bt_stride;
  int n = p.context_lens[b];
  n = n < 0 ? 0 : (n > cap ? cap : n);
  if (n == 0) return;
  const int t = n - 1;
  int phys = p.block_tables[(size_t)b * p.bt_stride + t / 16];
  phys = phys < 0 ? 0 : (phys >= p.num_blocks ? p.num_blocks - 1 : phys);

  const int chunks = p.head_dim / 8;                // 16-byte chunks per row
  const int per_pool = p.num_kv_heads * chunks;
  for (int i = threadIdx.x; i < 2 * per_pool; i += kAppendThreads) {
    const bool is_v = i >= per_pool;
    const int j = is_v ? i - per_pool : i;
    const int g = j / chunks;
    const int c = j - g * chunks;
    const uint16_t* src = (is_v ? p.v_new : p.k_new) + ((size_t)b * p.num_kv_heads + g) * p.head_dim;
    uint16_t* dst = (is_v ? p.v_pool : p.k_pool) +
                    (((size_t)phys * p.num_kv_heads + g) * 16 + (t & 15)) * p.head_dim;
    reinterpret_cast<uint4*>(dst)[c] = reinterpret_cast<const uint4*>(src)[c];
  }
}

}  // namespace

hipError_t launch_append(const AppendParams& p, hipStream_t stream) {
  if (p.batch == 0) return hipSuccess;
  hipLaunchKernelGGL(append_kernel, dim3((unsigned)p.batch), dim3(kAppendThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pa
