// A decode step that allocates nothing, for callers that cannot allocate
// device memory (code under graph capture, tight serving loops).
//
// paged_attn_decode needs caller-provided buffers for its split-KV partials
// whenever a batch splits.  This entry point keeps them instead in `scratch`,
// a device array of the library's own (PA_NOALLOC_SCRATCH_BYTES per GPU,
// held from the first call on a GPU until the process ends), and runs the
// decode and the reduce back to back on the caller's stream.  It calls no
// hipMalloc or hipFree.  In host code `scratch` names a host-side stand-in,
// not the device array: every host use goes through the device address that
// hipGetSymbolAddress returns, looked up once per GPU with that GPU current.
#include "kernels.h"
#include "paged_attn.h"

#include <hip/hip_runtime.h>

#include <mutex>

static __device__ __align__(256) uint8_t scratch[PA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this GPU's `scratch` (the current device), or NULL with
// the error recorded.
void* scratch_on_current_device(int* rc, const char* fn) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *rc = pa::fail(PA_EHIP, "%s: hipGetDevice failed: %s", fn, hipGetErrorString(e));
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    *rc = pa::fail(PA_EUNSUPPORTED, "%s: device %d outside [0, %d)", fn, dev, kMaxDevices);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      *rc = pa::fail(PA_EHIP, "%s: hipGetSymbolAddress(scratch) on device %d failed: %s", fn, dev,
                     hipGetErrorString(e));
      return nullptr;
    }
    g_scratch[dev] = ptr;
  }
  return g_scratch[dev];
}

}  // namespace

extern "C" int paged_attn_decode_noalloc(const pa_kv_pool* pool, const void* q,
                                         const int32_t* block_tables, int32_t bt_stride,
                                         const int32_t* context_lens, int32_t batch,
                                         int32_t num_q_heads, float scale, int32_t max_context_len,
                                         int32_t partition_size, void* out, void* stream) {
  const char* fn = "paged_attn_decode_noalloc";
  if (!pool) return pa::fail(PA_EINVAL, "%s: pool is NULL", fn);
  int64_t strides[4];
  int rc = kv_pool_layout(pool, strides, nullptr);
  if (rc) return rc;
  const int32_t head_dim = (int32_t)strides[2];
  size_t o_bytes = 0, lse_bytes = 0;
  rc = paged_attn_workspace_size(batch, num_q_heads, head_dim, max_context_len, partition_size,
                                 &o_bytes, &lse_bytes);
  if (rc) return rc;
  const size_t lse_at = (o_bytes + 255) / 256 * 256;
  if (lse_at + lse_bytes > (size_t)PA_NOALLOC_SCRATCH_BYTES)
    return pa::fail(PA_EINVAL, "%s: the split-KV partials need %zu bytes, more than the %zu-byte "
                    "scratch array", fn, lse_at + lse_bytes, (size_t)PA_NOALLOC_SCRATCH_BYTES);
  int32_t parts = 1;
  rc = paged_attn_num_partitions(max_context_len, partition_size, &parts);
  if (rc) return rc;
  float* part_o = nullptr;
  float* part_lse = nullptr;
  if (parts > 1 && batch > 0) {
    uint8_t* base = static_cast<uint8_t*>(scratch_on_current_device(&rc, fn));
    if (!base) return rc;
    part_o = reinterpret_cast<float*>(base);
    part_lse = reinterpret_cast<float*>(base + lse_at);
  }
  rc = paged_attn_decode(pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                         max_context_len, partition_size, out, part_o, part_lse, stream);
  if (rc || parts == 1 || batch == 0) return rc;
  return paged_attn_reduce(part_o, part_lse, context_lens, batch, num_q_heads, head_dim,
                           partition_size, parts, out, stream);
}
