// C ABI of the paged decode-attention library: KV block pool allocator,
// argument validation and launch planning.  Every check runs on the host
// before any HIP call, so all validation paths work without a GPU.
#include "paged_attn.h"
#include "kernels.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

struct pa_kv_pool {
  int32_t num_blocks;
  int32_t num_kv_heads;
  int32_t head_dim;
  uint16_t* k;                     // caller-owned device pools (the append writes them)
  uint16_t* v;
  std::vector<int32_t> refcount;  // 0 = free
  std::vector<int32_t> free_stack; // top = back(); ids pop in ascending order initially
  int64_t shared_blocks = 0;       // blocks whose reference count is 2 or more
};

namespace {
thread_local std::string g_err = "no error";
}  // namespace

namespace pa {
// Records the message that pa_last_error() returns and passes the code on.
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}
}  // namespace pa

namespace {
using pa::fail;

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Rebuild the free stack from refcounts (ascending ids pop first).
void rebuild_free(pa_kv_pool* pool) {
  pool->free_stack.clear();
  for (int32_t id = pool->num_blocks - 1; id >= 0; --id)
    if (pool->refcount[id] == 0) pool->free_stack.push_back(id);
}

int check_ids(const pa_kv_pool* pool, int32_t n, const int32_t* ids, const char* fn) {
  if (!pool) return fail(PA_EINVAL, "%s: pool is NULL", fn);
  if (n < 0) return fail(PA_EINVAL, "%s: n = %d < 0", fn, n);
  if (n > 0 && !ids) return fail(PA_EINVAL, "%s: ids is NULL", fn);
  for (int32_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= pool->num_blocks)
      return fail(PA_EINVAL, "%s: id %d at position %d outside [0, %d)", fn, ids[i], i,
                  pool->num_blocks);
  return PA_OK;
}

struct Plan {
  int32_t group;
  int32_t part_tokens;
  int32_t num_parts;
};

int plan(int32_t max_context_len, int32_t partition_size, Plan* out, const char* fn) {
  if (max_context_len < 0) return fail(PA_EINVAL, "%s: max_context_len = %d < 0", fn, max_context_len);
  if (partition_size < 0 || partition_size % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: partition_size = %d is not a non-negative multiple of %d", fn,
                partition_size, PA_BLOCK_SIZE);
  const int64_t whole = ((int64_t)max_context_len + PA_BLOCK_SIZE - 1) / PA_BLOCK_SIZE * PA_BLOCK_SIZE;
  if (partition_size == 0 || whole <= partition_size) {
    out->part_tokens = (int32_t)(whole > 0 ? whole : PA_BLOCK_SIZE);
    out->num_parts = 1;
  } else {
    out->part_tokens = partition_size;
    out->num_parts = (int32_t)(((int64_t)max_context_len + partition_size - 1) / partition_size);
  }
  return PA_OK;
}

struct DecodeArgs {
  const pa_kv_pool* pool;
  const void* q;
  const int32_t* block_tables;
  int32_t bt_stride;
  const int32_t* context_lens;
  int32_t batch;
  int32_t num_q_heads;
  float scale;
  int32_t max_context_len;
  const void* k_new = nullptr;     // fused KV append: [batch][num_kv_heads][head_dim] bf16, or NULL
  const void* v_new = nullptr;
};

// Checks shared by every decode entry point; fills the group size.
int validate_decode(const DecodeArgs& a, int32_t* group, const char* fn) {
  if (!a.pool) return fail(PA_EINVAL, "%s: pool is NULL", fn);
  if (a.batch < 0) return fail(PA_EINVAL, "%s: batch = %d < 0", fn, a.batch);
  if (a.num_q_heads <= 0 || a.num_q_heads % a.pool->num_kv_heads != 0)
    return fail(PA_EINVAL, "%s: num_q_heads = %d is not a positive multiple of num_kv_heads = %d",
                fn, a.num_q_heads, a.pool->num_kv_heads);
  *group = a.num_q_heads / a.pool->num_kv_heads;
  if (*group != 4 && *group != 8)
    return fail(PA_EUNSUPPORTED, "%s: query heads per KV head = %d (supported: 4, 8)", fn, *group);
  if (!(a.scale == a.scale) || a.scale == __builtin_inff() || a.scale == -__builtin_inff())
    return fail(PA_EINVAL, "%s: scale is not finite", fn);
  if (a.max_context_len < 0)
    return fail(PA_EINVAL, "%s: max_context_len = %d < 0", fn, a.max_context_len);
  const int64_t need_bt = ((int64_t)a.max_context_len + PA_BLOCK_SIZE - 1) / PA_BLOCK_SIZE;
  if (a.bt_stride < need_bt || a.bt_stride < 0)
    return fail(PA_EINVAL, "%s: bt_stride = %d < ceil(max_context_len / 16) = %lld", fn,
                a.bt_stride, (long long)need_bt);
  if (a.batch == 0) return PA_OK;
  if (!a.q || !a.block_tables || !a.context_lens)
    return fail(PA_EINVAL, "%s: q, block_tables and context_lens must be non-NULL", fn);
  if (!aligned(a.q, 16)) return fail(PA_EINVAL, "%s: q is not 16-byte aligned", fn);
  if (!aligned(a.block_tables, 4) || !aligned(a.context_lens, 4))
    return fail(PA_EINVAL, "%s: block_tables/context_lens are not 4-byte aligned", fn);
  if ((a.k_new != nullptr) != (a.v_new != nullptr))
    return fail(PA_EINVAL, "%s: k_new and v_new must both be given or both be NULL", fn);
  if (a.k_new && (!aligned(a.k_new, 16) || !aligned(a.v_new, 16)))
    return fail(PA_EINVAL, "%s: k_new/v_new are not 16-byte aligned", fn);
  return PA_OK;
}

// Workgroup order of a decode grid.  With many partitions per sequence the
// partitions of one sequence are dispatched together, so the end of the grid
// is a mix of sequences instead of the last partitions of the longest ones
// (measured: +3% on contexts of 8k-32k tokens in 512- or 1024-token
// partitions, while partition-major is faster for a few partitions).
int32_t item_order_for(int32_t num_parts) { return num_parts >= 16 ? 1 : 0; }

pa::DecodeParams decode_params(const DecodeArgs& a) {
  pa::DecodeParams p{};
  p.k_pool = a.pool->k;
  p.v_pool = a.pool->v;
  p.q = static_cast<const uint16_t*>(a.q);
  p.block_tables = a.block_tables;
  p.context_lens = a.context_lens;
  p.num_blocks = a.pool->num_blocks;
  p.num_kv_heads = a.pool->num_kv_heads;
  p.num_q_heads = a.num_q_heads;
  p.batch = a.batch;
  p.bt_stride = a.bt_stride;
  p.max_ctx = a.max_context_len;
  // With no block shared by two tables every tile is read once per step:
  // stream it past the caches.
  p.stream_tiles = a.pool->shared_blocks == 0 ? 1 : 0;
  p.scale_log2 = a.scale * 1.4426950408889634f;
  if (a.k_new) {
    p.k_new = static_cast<const uint16_t*>(a.k_new);
    p.v_new = static_cast<const uint16_t*>(a.v_new);
    p.k_pool_w = a.pool->k;
    p.v_pool_w = a.pool->v;
  }
  return p;
}

hipError_t launch_decode(const pa::DecodeParams& p, const pa_kv_pool* pool, int32_t group,
                         bool tracing, void* stream) {
  // GQA groups of 8 at head_dim 128 form dense 16x16 tiles: matrix cores;
  // everything else runs on VALU dot products.
  return (group == 8 && pool->head_dim == 128)
             ? pa::launch_decode_mfma(p, tracing, static_cast<hipStream_t>(stream))
             : pa::launch_decode_valu(p, pool->head_dim, group, tracing,
                                      static_cast<hipStream_t>(stream));
}

// Checks of an optional host-built work list (items = part * batch + b).
int validate_items(const int32_t* items, int32_t num_items, int64_t max_items, const char* fn) {
  if (num_items < 0 || num_items > max_items)
    return fail(PA_EINVAL, "%s: num_items = %d outside [0, %lld]", fn, num_items, (long long)max_items);
  if (num_items > 0 && (!items || !aligned(items, 4)))
    return fail(PA_EINVAL, "%s: items is NULL or not 4-byte aligned", fn);
  return PA_OK;
}

int decode_impl(const DecodeArgs& a, int32_t partition_size, void* out, float* partial_out,
                float* partial_lse, int32_t* trace, int64_t trace_capacity, bool tracing,
                void* stream, const char* fn, bool scheduled = false,
                const int32_t* items = nullptr, int32_t num_items = 0) {
  int32_t group = 0;
  int rc = validate_decode(a, &group, fn);
  if (rc) return rc;
  Plan pl;
  rc = plan(a.max_context_len, partition_size, &pl, fn);
  if (rc) return rc;
  const int64_t grid = (int64_t)pl.num_parts * a.batch * a.pool->num_kv_heads;
  if (grid > 0x7fffffffLL) return fail(PA_EINVAL, "%s: grid of %lld workgroups is too large", fn, (long long)grid);
  if (scheduled) {
    rc = validate_items(items, num_items, (int64_t)pl.num_parts * a.batch, fn);
    if (rc) return rc;
  }
  if (a.batch == 0) return PA_OK;
  const bool split = pl.num_parts > 1;
  if (!split) {
    if (!out) return fail(PA_EINVAL, "%s: out is NULL (single partition)", fn);
    if (!aligned(out, 4)) return fail(PA_EINVAL, "%s: out is not 4-byte aligned", fn);
  } else {
    if (!partial_out || !partial_lse)
      return fail(PA_EINVAL, "%s: %d partitions need partial_out and partial_lse", fn, pl.num_parts);
    if (!aligned(partial_out, 16) || !aligned(partial_lse, 4))
      return fail(PA_EINVAL, "%s: partial buffers are misaligned", fn);
  }
  const int32_t trace_tiles = pl.part_tokens / PA_BLOCK_SIZE;
  if (tracing) {
    const int64_t need = grid * trace_tiles * 3;
    if (!trace || !aligned(trace, 4)) return fail(PA_EINVAL, "%s: trace buffer is NULL or misaligned", fn);
    if (trace_capacity < need)
      return fail(PA_EINVAL, "%s: trace_capacity %lld < %lld int32 values", fn,
                  (long long)trace_capacity, (long long)need);
  }
  pa::DecodeParams p = decode_params(a);
  p.out = static_cast<uint16_t*>(out);
  p.part_o = partial_out;
  p.part_lse = partial_lse;
  p.trace = trace;
  p.part_tokens = pl.part_tokens;
  p.num_parts = pl.num_parts;
  p.item_order = item_order_for(pl.num_parts);
  p.token_offset = 0;
  p.part_offset = 0;
  p.part_stride = pl.num_parts;
  p.write_partials = split ? 1 : 0;
  p.trace_tiles = trace_tiles;
  if (scheduled) {
    p.items = items;
    p.num_items = num_items;
  }
  hipError_t e = launch_decode(p, a.pool, group, tracing, stream);
  if (e != hipSuccess) return fail(PA_EHIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return PA_OK;
}

// Partition plan of a shared-prefix (cascade) step.
struct CascadePlan {
  int32_t pre_parts, pre_tokens;  // prefix partitions and their size
  int32_t group_parts;            // 1 with a second level of groups, else 0
  int32_t shared_len;             // prefix_len + group_len: where the per-sequence part starts
  int32_t suf_parts, suf_tokens;  // partitions of the rest of the longest context
  int32_t stride;                 // partitions per (sequence, head)
};

int plan_cascade(int32_t max_context_len, int32_t partition_size, int32_t prefix_len,
                 int32_t prefix_partition_size, int32_t group_len, CascadePlan* out, const char* fn) {
  if (max_context_len < 0) return fail(PA_EINVAL, "%s: max_context_len = %d < 0", fn, max_context_len);
  if (partition_size <= 0 || partition_size % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: partition_size = %d is not a positive multiple of %d", fn,
                partition_size, PA_BLOCK_SIZE);
  if (prefix_len < 0 || prefix_len % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: prefix_len = %d is not a non-negative multiple of %d", fn,
                prefix_len, PA_BLOCK_SIZE);
  if (prefix_len > max_context_len)
    return fail(PA_EINVAL, "%s: prefix_len = %d exceeds max_context_len = %d", fn, prefix_len,
                max_context_len);
  if (prefix_partition_size < PA_BLOCK_SIZE || prefix_partition_size > 64 * PA_BLOCK_SIZE ||
      prefix_partition_size % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: prefix_partition_size = %d not a multiple of 16 in [16, 1024]", fn,
                prefix_partition_size);
  if (group_len < 0 || group_len % PA_BLOCK_SIZE != 0 || group_len > 64 * PA_BLOCK_SIZE)
    return fail(PA_EINVAL, "%s: group_len = %d not a multiple of 16 in [0, 1024]", fn, group_len);
  if ((int64_t)prefix_len + group_len > max_context_len)
    return fail(PA_EINVAL, "%s: prefix_len + group_len = %d exceeds max_context_len = %d", fn,
                prefix_len + group_len, max_context_len);
  out->pre_tokens = prefix_partition_size;
  out->pre_parts = (prefix_len + prefix_partition_size - 1) / prefix_partition_size;
  out->group_parts = group_len > 0 ? 1 : 0;
  out->shared_len = prefix_len + group_len;
  out->suf_tokens = partition_size;
  const int64_t rest = (int64_t)max_context_len - out->shared_len;
  out->suf_parts = (int32_t)((rest + partition_size - 1) / partition_size);
  const int64_t stride = (int64_t)out->pre_parts + out->group_parts + out->suf_parts;
  out->stride = (int32_t)(stride > 0 ? stride : 1);
  return PA_OK;
}

// Where the index trace of a cascade step puts each kind of work item, in
// int32 values (three per tile): the prefix partitions' tiles, then the
// groups', then the per-sequence partitions'.
struct TraceLayout {
  int64_t prefix_offset, prefix_tiles;
  int64_t group_offset, group_tiles;
  int64_t decode_offset, decode_tiles;
  int64_t total;
};

void cascade_trace_layout(int32_t num_kv_heads, int32_t batch, int32_t group, const CascadePlan& cp,
                          int32_t num_groups, int32_t group_len, TraceLayout* t) {
  const int64_t row_groups = ((int64_t)batch * group + pa::kSharedRowsPerWg - 1) / pa::kSharedRowsPerWg;
  t->prefix_tiles = cp.pre_tokens / PA_BLOCK_SIZE;
  t->group_tiles = group_len / PA_BLOCK_SIZE;
  t->decode_tiles = cp.suf_tokens / PA_BLOCK_SIZE;
  t->prefix_offset = 0;
  t->group_offset = t->prefix_offset + 3 * (int64_t)cp.pre_parts * row_groups * num_kv_heads * t->prefix_tiles;
  const int64_t groups = group_len > 0 ? num_groups : 0;
  t->decode_offset = t->group_offset + 3 * groups * num_kv_heads * t->group_tiles;
  t->total = t->decode_offset + 3 * (int64_t)cp.suf_parts * batch * num_kv_heads * t->decode_tiles;
}

}  // namespace

extern "C" {

const char* pa_last_error(void) { return g_err.c_str(); }

int32_t pa_version(void) { return 100; }

int kv_pool_create(int32_t num_blocks, int32_t block_size, int32_t num_kv_heads, int32_t head_dim,
                   void* k_pool, void* v_pool, pa_kv_pool** out) {
  if (!out) return fail(PA_EINVAL, "kv_pool_create: out is NULL");
  if (num_blocks <= 0) return fail(PA_EINVAL, "kv_pool_create: num_blocks = %d <= 0", num_blocks);
  if (block_size != PA_BLOCK_SIZE)
    return fail(PA_EINVAL, "kv_pool_create: block_size = %d (must be %d)", block_size, PA_BLOCK_SIZE);
  if (num_kv_heads < 1 || num_kv_heads > 64)
    return fail(PA_EINVAL, "kv_pool_create: num_kv_heads = %d outside [1, 64]", num_kv_heads);
  if (head_dim != 64 && head_dim != 128)
    return fail(PA_EUNSUPPORTED, "kv_pool_create: head_dim = %d (supported: 64, 128)", head_dim);
  if (!k_pool || !v_pool) return fail(PA_EINVAL, "kv_pool_create: pool pointers must be non-NULL");
  if (!aligned(k_pool, 16) || !aligned(v_pool, 16))
    return fail(PA_EINVAL, "kv_pool_create: pool pointers must be 16-byte aligned");
  pa_kv_pool* p = new (std::nothrow) pa_kv_pool;
  if (!p) return fail(PA_ENOMEM, "kv_pool_create: host allocation failed");
  p->num_blocks = num_blocks;
  p->num_kv_heads = num_kv_heads;
  p->head_dim = head_dim;
  p->k = static_cast<uint16_t*>(k_pool);
  p->v = static_cast<uint16_t*>(v_pool);
  p->refcount.assign(num_blocks, 0);
  rebuild_free(p);
  *out = p;
  return PA_OK;
}

int kv_pool_destroy(pa_kv_pool* pool) {
  delete pool;
  return PA_OK;
}

int kv_pool_alloc(pa_kv_pool* pool, int32_t n, int32_t* ids_out) {
  if (!pool) return fail(PA_EINVAL, "kv_pool_alloc: pool is NULL");
  if (n < 0) return fail(PA_EINVAL, "kv_pool_alloc: n = %d < 0", n);
  if (n > 0 && !ids_out) return fail(PA_EINVAL, "kv_pool_alloc: ids_out is NULL");
  if ((size_t)n > pool->free_stack.size())
    return fail(PA_ENOMEM, "kv_pool_alloc: %d blocks requested, %zu free", n, pool->free_stack.size());
  for (int32_t i = 0; i < n; ++i) {
    const int32_t id = pool->free_stack.back();
    pool->free_stack.pop_back();
    pool->refcount[id] = 1;
    ids_out[i] = id;
  }
  return PA_OK;
}

int kv_pool_claim(pa_kv_pool* pool, int32_t n, const int32_t* ids) {
  int rc = check_ids(pool, n, ids, "kv_pool_claim");
  if (rc) return rc;
  std::vector<char> seen(pool->num_blocks, 0);
  for (int32_t i = 0; i < n; ++i) {
    if (pool->refcount[ids[i]] != 0)
      return fail(PA_ESTATE, "kv_pool_claim: block %d is already in use", ids[i]);
    if (seen[ids[i]]) return fail(PA_ESTATE, "kv_pool_claim: block %d listed twice", ids[i]);
    seen[ids[i]] = 1;
  }
  for (int32_t i = 0; i < n; ++i) pool->refcount[ids[i]] = 1;
  rebuild_free(pool);
  return PA_OK;
}

int kv_pool_retain(pa_kv_pool* pool, int32_t n, const int32_t* ids) {
  int rc = check_ids(pool, n, ids, "kv_pool_retain");
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i)
    if (pool->refcount[ids[i]] == 0)
      return fail(PA_ESTATE, "kv_pool_retain: block %d is free", ids[i]);
  for (int32_t i = 0; i < n; ++i) {
    if (pool->refcount[ids[i]] == 0x7fffffff)
      return fail(PA_ESTATE, "kv_pool_retain: reference count of block %d overflows", ids[i]);
  }
  for (int32_t i = 0; i < n; ++i)
    if (++pool->refcount[ids[i]] == 2) ++pool->shared_blocks;
  return PA_OK;
}

int kv_pool_release(pa_kv_pool* pool, int32_t n, const int32_t* ids) {
  int rc = check_ids(pool, n, ids, "kv_pool_release");
  if (rc) return rc;
  std::vector<int32_t> count(pool->num_blocks, 0);
  for (int32_t i = 0; i < n; ++i)
    if (++count[ids[i]] > pool->refcount[ids[i]])
      return fail(PA_ESTATE, "kv_pool_release: block %d released more often than retained", ids[i]);
  bool freed = false;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t left = --pool->refcount[ids[i]];
    if (left == 0) freed = true;
    if (left == 1) --pool->shared_blocks;
  }
  if (freed) rebuild_free(pool);
  return PA_OK;
}

int kv_pool_num_free(const pa_kv_pool* pool, int32_t* n_out) {
  if (!pool || !n_out) return fail(PA_EINVAL, "kv_pool_num_free: NULL argument");
  *n_out = (int32_t)pool->free_stack.size();
  return PA_OK;
}

int kv_pool_num_shared(const pa_kv_pool* pool, int64_t* n_out) {
  if (!pool || !n_out) return fail(PA_EINVAL, "kv_pool_num_shared: NULL argument");
  *n_out = pool->shared_blocks;
  return PA_OK;
}

int kv_pool_refcount(const pa_kv_pool* pool, int32_t id, int32_t* count_out) {
  if (!pool || !count_out) return fail(PA_EINVAL, "kv_pool_refcount: NULL argument");
  if (id < 0 || id >= pool->num_blocks)
    return fail(PA_EINVAL, "kv_pool_refcount: id %d outside [0, %d)", id, pool->num_blocks);
  *count_out = pool->refcount[id];
  return PA_OK;
}

int kv_pool_layout(const pa_kv_pool* pool, int64_t elem_strides_out[4], int64_t* pool_bytes_out) {
  if (!pool || !elem_strides_out) return fail(PA_EINVAL, "kv_pool_layout: NULL argument");
  const int64_t d = pool->head_dim;
  elem_strides_out[3] = 1;
  elem_strides_out[2] = d;
  elem_strides_out[1] = PA_BLOCK_SIZE * d;
  elem_strides_out[0] = (int64_t)pool->num_kv_heads * PA_BLOCK_SIZE * d;
  if (pool_bytes_out) *pool_bytes_out = elem_strides_out[0] * pool->num_blocks * 2;
  return PA_OK;
}

int paged_attn_num_partitions(int32_t max_context_len, int32_t partition_size, int32_t* p_out) {
  if (!p_out) return fail(PA_EINVAL, "paged_attn_num_partitions: p_out is NULL");
  Plan pl;
  int rc = plan(max_context_len, partition_size, &pl, "paged_attn_num_partitions");
  if (rc) return rc;
  *p_out = pl.num_parts;
  return PA_OK;
}

int paged_attn_workspace_size(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                              int32_t max_context_len, int32_t partition_size,
                              size_t* partial_out_bytes, size_t* partial_lse_bytes) {
  if (!partial_out_bytes || !partial_lse_bytes)
    return fail(PA_EINVAL, "paged_attn_workspace_size: NULL output pointer");
  if (batch < 0 || num_q_heads <= 0 || head_dim <= 0)
    return fail(PA_EINVAL, "paged_attn_workspace_size: bad geometry");
  Plan pl;
  int rc = plan(max_context_len, partition_size, &pl, "paged_attn_workspace_size");
  if (rc) return rc;
  if (pl.num_parts == 1) {
    *partial_out_bytes = 0;
    *partial_lse_bytes = 0;
  } else {
    const size_t rows = (size_t)batch * num_q_heads * pl.num_parts;
    *partial_out_bytes = rows * head_dim * sizeof(float);
    *partial_lse_bytes = rows * sizeof(float);
  }
  return PA_OK;
}

int paged_attn_decode(const pa_kv_pool* pool, const void* q, const int32_t* block_tables,
                      int32_t bt_stride, const int32_t* context_lens, int32_t batch,
                      int32_t num_q_heads, float scale, int32_t max_context_len,
                      int32_t partition_size, void* out, float* partial_out, float* partial_lse,
                      void* stream) {
  const DecodeArgs a{pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                     max_context_len};
  return decode_impl(a, partition_size, out, partial_out, partial_lse, nullptr, 0, false, stream,
                     "paged_attn_decode");
}

int paged_attn_decode_trace(const pa_kv_pool* pool, const void* q, const int32_t* block_tables,
                            int32_t bt_stride, const int32_t* context_lens, int32_t batch,
                            int32_t num_q_heads, float scale, int32_t max_context_len,
                            int32_t partition_size, void* out, float* partial_out,
                            float* partial_lse, int32_t* trace, int64_t trace_capacity,
                            void* stream) {
  const DecodeArgs a{pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                     max_context_len};
  return decode_impl(a, partition_size, out, partial_out, partial_lse, trace, trace_capacity, true,
                     stream, "paged_attn_decode_trace");
}

namespace {
int cascade_workspace_impl(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                           int32_t max_context_len, int32_t partition_size, int32_t prefix_len,
                           int32_t prefix_partition_size, int32_t group_len,
                           size_t* partial_out_bytes, size_t* partial_lse_bytes,
                           int32_t* max_partitions_out, const char* fn) {
  if (!partial_out_bytes || !partial_lse_bytes || !max_partitions_out)
    return fail(PA_EINVAL, "%s: NULL output pointer", fn);
  if (batch < 0 || num_q_heads <= 0 || head_dim <= 0) return fail(PA_EINVAL, "%s: bad geometry", fn);
  CascadePlan cp;
  int rc = plan_cascade(max_context_len, partition_size, prefix_len, prefix_partition_size,
                        group_len, &cp, fn);
  if (rc) return rc;
  const size_t rows = (size_t)batch * num_q_heads * cp.stride;
  *partial_out_bytes = rows * head_dim * sizeof(float);
  *partial_lse_bytes = rows * sizeof(float);
  *max_partitions_out = cp.stride;
  return PA_OK;
}
}  // namespace

int paged_attn_cascade_workspace_size(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                                      int32_t max_context_len, int32_t partition_size,
                                      int32_t prefix_len, int32_t prefix_partition_size,
                                      size_t* partial_out_bytes, size_t* partial_lse_bytes,
                                      int32_t* max_partitions_out) {
  return cascade_workspace_impl(batch, num_q_heads, head_dim, max_context_len, partition_size,
                                prefix_len, prefix_partition_size, 0, partial_out_bytes,
                                partial_lse_bytes, max_partitions_out,
                                "paged_attn_cascade_workspace_size");
}

int paged_attn_cascade_groups_workspace_size(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                                             int32_t max_context_len, int32_t partition_size,
                                             int32_t prefix_len, int32_t prefix_partition_size,
                                             int32_t group_len, size_t* partial_out_bytes,
                                             size_t* partial_lse_bytes, int32_t* max_partitions_out) {
  return cascade_workspace_impl(batch, num_q_heads, head_dim, max_context_len, partition_size,
                                prefix_len, prefix_partition_size, group_len, partial_out_bytes,
                                partial_lse_bytes, max_partitions_out,
                                "paged_attn_cascade_groups_workspace_size");
}

namespace {

int cascade_impl(const pa_kv_pool* pool, const void* q, const int32_t* block_tables,
                 int32_t bt_stride, const int32_t* context_lens, int32_t batch,
                 int32_t num_q_heads, float scale, int32_t max_context_len,
                 int32_t partition_size, int32_t prefix_len, int32_t prefix_partition_size,
                 float* partial_out, float* partial_lse, void* stream, const char* fn,
                 bool scheduled, const int32_t* items, int32_t num_items,
                 const int32_t* group_start = nullptr, int32_t num_groups = 0,
                 int32_t max_group_size = 0, int32_t group_len = 0, int32_t* trace = nullptr,
                 int64_t trace_capacity = 0, bool tracing = false, const void* k_new = nullptr,
                 const void* v_new = nullptr) {
  const DecodeArgs a{pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                     max_context_len, k_new, v_new};
  int32_t group = 0;
  int rc = validate_decode(a, &group, fn);
  if (rc) return rc;
  CascadePlan cp;
  rc = plan_cascade(max_context_len, partition_size, prefix_len, prefix_partition_size, group_len,
                    &cp, fn);
  if (rc) return rc;
  if ((prefix_len > 0 || group_len > 0) && pool->head_dim != 128)
    return fail(PA_EUNSUPPORTED, "%s: the shared passes need head_dim 128", fn);
  if (group_len > 0 && batch > 0) {
    if (num_groups < 1 || num_groups > batch)
      return fail(PA_EINVAL, "%s: num_groups = %d outside [1, batch]", fn, num_groups);
    if (max_group_size < 1 || (int64_t)max_group_size * group > 64)
      return fail(PA_EINVAL, "%s: max_group_size = %d: groups of 1 .. %d sequences at %d heads per "
                  "KV head", fn, max_group_size, 64 / group, group);
    if (!group_start || !aligned(group_start, 4))
      return fail(PA_EINVAL, "%s: group_start is NULL or not 4-byte aligned", fn);
  }
  const int64_t rows = (int64_t)batch * num_q_heads;
  // Upper bound on the fused grid: a prefix workgroup covers at least 16 query
  // rows of one KV head, a suffix workgroup one (sequence, KV head) pair.
  const int64_t g_pre = (int64_t)cp.pre_parts * ((rows / pool->num_kv_heads + 15) / 16) * pool->num_kv_heads;
  const int64_t g_suf = (int64_t)cp.suf_parts * batch * pool->num_kv_heads;
  const int64_t g_grp = group_len > 0 ? (int64_t)num_groups * pool->num_kv_heads : 0;
  if (g_pre + g_grp + g_suf > 0x7fffffffLL)
    return fail(PA_EINVAL, "%s: grid too large", fn);
  if (scheduled) {
    rc = validate_items(items, num_items, (int64_t)cp.suf_parts * batch, fn);
    if (rc) return rc;
  }
  TraceLayout tl;
  if (tracing) {
    cascade_trace_layout(pool->num_kv_heads, batch, group, cp, num_groups, group_len, &tl);
    if (!trace || !aligned(trace, 4)) return fail(PA_EINVAL, "%s: trace buffer is NULL or misaligned", fn);
    if (trace_capacity < tl.total)
      return fail(PA_EINVAL, "%s: trace_capacity %lld < %lld int32 values", fn,
                  (long long)trace_capacity, (long long)tl.total);
  }
  if (batch == 0) return PA_OK;
  if (!partial_out || !partial_lse) return fail(PA_EINVAL, "%s: partial buffers are NULL", fn);
  if (!aligned(partial_out, 16) || !aligned(partial_lse, 4))
    return fail(PA_EINVAL, "%s: partial buffers are misaligned", fn);
  hipStream_t st = static_cast<hipStream_t>(stream);
  pa::PrefixParams pp{};
  pp.k_pool = pool->k;
  pp.v_pool = pool->v;
  pp.q = static_cast<const uint16_t*>(q);
  pp.block_tables = block_tables;
  pp.context_lens = context_lens;
  pp.part_o = partial_out;
  pp.part_lse = partial_lse;
  pp.num_blocks = pool->num_blocks;
  pp.num_kv_heads = pool->num_kv_heads;
  pp.num_q_heads = num_q_heads;
  pp.batch = batch;
  pp.bt_stride = bt_stride;
  pp.prefix_len = prefix_len;
  pp.part_tokens = cp.pre_tokens;
  pp.prefix_parts = cp.pre_parts;
  pp.part_stride = cp.stride;
  pp.max_ctx = max_context_len;
  if (group_len > 0) {
    pp.group_start = group_start;
    pp.num_groups = num_groups;
    pp.max_group_size = max_group_size;
    pp.group_len = group_len;
  }
  pp.scale_log2 = scale * 1.4426950408889634f;
  if (tracing) {
    pp.trace_prefix = trace + tl.prefix_offset;
    pp.trace_group = trace + tl.group_offset;
    pp.prefix_trace_tiles = tl.prefix_tiles;
    pp.group_trace_tiles = tl.group_tiles;
  }
  pa::DecodeParams p = decode_params(a);
  p.part_o = partial_out;
  p.part_lse = partial_lse;
  p.part_tokens = cp.suf_tokens;
  p.num_parts = cp.suf_parts;
  p.item_order = item_order_for(cp.suf_parts);
  p.token_offset = cp.shared_len;
  p.part_offset = cp.pre_parts + cp.group_parts;
  p.part_stride = cp.stride;
  p.write_partials = 1;
  p.trace_tiles = cp.suf_tokens / PA_BLOCK_SIZE;
  if (tracing) p.trace = trace + tl.decode_offset;
  if (scheduled) {
    p.items = items;
    p.num_items = num_items;
  }
  if (pool->head_dim == 128) {
    // prefix pass and per-sequence decode in one grid
    hipError_t e = pa::launch_cascade(pp, p, group, tracing, st);
    if (e != hipSuccess) return fail(PA_EHIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
    return PA_OK;
  }
  if (cp.suf_parts > 0) {  // no shared pass (head_dim 64 requires prefix_len 0, no groups)
    hipError_t e = launch_decode(p, pool, group, tracing, stream);
    if (e != hipSuccess) return fail(PA_EHIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  }
  return PA_OK;
}

// Lengths of the work items of a decode plan, for the host schedule.
struct ItemLen {
  int32_t len;
  int32_t item;   // part * batch + b
};

}  // namespace

int paged_attn_decode_cascade(const pa_kv_pool* pool, const void* q, const int32_t* block_tables,
                              int32_t bt_stride, const int32_t* context_lens, int32_t batch,
                              int32_t num_q_heads, float scale, int32_t max_context_len,
                              int32_t partition_size, int32_t prefix_len,
                              int32_t prefix_partition_size, float* partial_out,
                              float* partial_lse, void* stream) {
  return cascade_impl(pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                      max_context_len, partition_size, prefix_len, prefix_partition_size,
                      partial_out, partial_lse, stream, "paged_attn_decode_cascade", false, nullptr, 0);
}

int paged_attn_decode_cascade_scheduled(const pa_kv_pool* pool, const void* q,
                                        const int32_t* block_tables, int32_t bt_stride,
                                        const int32_t* context_lens, int32_t batch,
                                        int32_t num_q_heads, float scale, int32_t max_context_len,
                                        int32_t partition_size, int32_t prefix_len,
                                        int32_t prefix_partition_size, const int32_t* items,
                                        int32_t num_items, float* partial_out, float* partial_lse,
                                        void* stream) {
  return cascade_impl(pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                      max_context_len, partition_size, prefix_len, prefix_partition_size,
                      partial_out, partial_lse, stream, "paged_attn_decode_cascade_scheduled", true,
                      items, num_items);
}

int paged_attn_decode_cascade_groups(const pa_kv_pool* pool, const void* q,
                                     const int32_t* block_tables, int32_t bt_stride,
                                     const int32_t* context_lens, int32_t batch, int32_t num_q_heads,
                                     float scale, int32_t max_context_len, int32_t partition_size,
                                     int32_t prefix_len, int32_t prefix_partition_size,
                                     const int32_t* group_start, int32_t num_groups,
                                     int32_t max_group_size, int32_t group_len, const int32_t* items,
                                     int32_t num_items, float* partial_out, float* partial_lse,
                                     void* stream) {
  const char* fn = "paged_attn_decode_cascade_groups";
  if (group_len <= 0) return fail(PA_EINVAL, "%s: group_len = %d <= 0", fn, group_len);
  return cascade_impl(pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                      max_context_len, partition_size, prefix_len, prefix_partition_size,
                      partial_out, partial_lse, stream, fn, items != nullptr, items, num_items,
                      group_start, num_groups, max_group_size, group_len);
}

int paged_attn_decode_append(const pa_kv_pool* pool, const void* q, const void* k_new,
                             const void* v_new, const int32_t* block_tables, int32_t bt_stride,
                             const int32_t* context_lens, int32_t batch, int32_t num_q_heads,
                             float scale, int32_t max_context_len, int32_t partition_size,
                             const int32_t* items, int32_t num_items, void* out, float* partial_out,
                             float* partial_lse, void* stream) {
  const char* fn = "paged_attn_decode_append";
  if (!k_new || !v_new) return fail(PA_EINVAL, "%s: k_new and v_new must be non-NULL", fn);
  const DecodeArgs a{pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                     max_context_len, k_new, v_new};
  return decode_impl(a, partition_size, out, partial_out, partial_lse, nullptr, 0, false, stream, fn,
                     items != nullptr, items, num_items);
}

int paged_attn_decode_cascade_append(const pa_kv_pool* pool, const void* q, const void* k_new,
                                     const void* v_new, const int32_t* block_tables,
                                     int32_t bt_stride, const int32_t* context_lens, int32_t batch,
                                     int32_t num_q_heads, float scale, int32_t max_context_len,
                                     int32_t partition_size, int32_t prefix_len,
                                     int32_t prefix_partition_size, const int32_t* group_start,
                                     int32_t num_groups, int32_t max_group_size, int32_t group_len,
                                     const int32_t* items, int32_t num_items, float* partial_out,
                                     float* partial_lse, void* stream) {
  const char* fn = "paged_attn_decode_cascade_append";
  if (!k_new || !v_new) return fail(PA_EINVAL, "%s: k_new and v_new must be non-NULL", fn);
  if (group_len < 0) return fail(PA_EINVAL, "%s: group_len = %d < 0", fn, group_len);
  return cascade_impl(pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                      max_context_len, partition_size, prefix_len, prefix_partition_size,
                      partial_out, partial_lse, stream, fn, items != nullptr, items, num_items,
                      group_start, group_len > 0 ? num_groups : 0, max_group_size, group_len,
                      nullptr, 0, false, k_new, v_new);
}

int paged_attn_decode_scheduled(const pa_kv_pool* pool, const void* q, const int32_t* block_tables,
                                int32_t bt_stride, const int32_t* context_lens, int32_t batch,
                                int32_t num_q_heads, float scale, int32_t max_context_len,
                                int32_t partition_size, const int32_t* items, int32_t num_items,
                                void* out, float* partial_out, float* partial_lse, void* stream) {
  const DecodeArgs a{pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                     max_context_len};
  return decode_impl(a, partition_size, out, partial_out, partial_lse, nullptr, 0, false, stream,
                     "paged_attn_decode_scheduled", true, items, num_items);
}

int paged_attn_decode_scheduled_trace(const pa_kv_pool* pool, const void* q,
                                      const int32_t* block_tables, int32_t bt_stride,
                                      const int32_t* context_lens, int32_t batch, int32_t num_q_heads,
                                      float scale, int32_t max_context_len, int32_t partition_size,
                                      const int32_t* items, int32_t num_items, void* out,
                                      float* partial_out, float* partial_lse, int32_t* trace,
                                      int64_t trace_capacity, void* stream) {
  const DecodeArgs a{pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                     max_context_len};
  return decode_impl(a, partition_size, out, partial_out, partial_lse, trace, trace_capacity, true,
                     stream, "paged_attn_decode_scheduled_trace", true, items, num_items);
}

int paged_attn_cascade_trace_layout(const pa_kv_pool* pool, int32_t batch, int32_t num_q_heads,
                                    int32_t max_context_len, int32_t partition_size,
                                    int32_t prefix_len, int32_t prefix_partition_size,
                                    int32_t num_groups, int32_t group_len, int64_t layout_out[7]) {
  const char* fn = "paged_attn_cascade_trace_layout";
  if (!pool || !layout_out) return fail(PA_EINVAL, "%s: NULL argument", fn);
  if (batch < 0) return fail(PA_EINVAL, "%s: batch = %d < 0", fn, batch);
  if (num_q_heads <= 0 || num_q_heads % pool->num_kv_heads != 0)
    return fail(PA_EINVAL, "%s: num_q_heads = %d is not a positive multiple of num_kv_heads = %d", fn,
                num_q_heads, pool->num_kv_heads);
  if (group_len > 0 && (num_groups < 1 || num_groups > batch))
    return fail(PA_EINVAL, "%s: num_groups = %d outside [1, batch]", fn, num_groups);
  CascadePlan cp;
  const int rc = plan_cascade(max_context_len, partition_size, prefix_len, prefix_partition_size,
                              group_len, &cp, fn);
  if (rc) return rc;
  TraceLayout t;
  cascade_trace_layout(pool->num_kv_heads, batch, num_q_heads / pool->num_kv_heads, cp, num_groups,
                       group_len, &t);
  const int64_t v[7] = {t.prefix_offset, t.prefix_tiles, t.group_offset, t.group_tiles,
                        t.decode_offset, t.decode_tiles, t.total};
  for (int i = 0; i < 7; ++i) layout_out[i] = v[i];
  return PA_OK;
}

int paged_attn_decode_cascade_trace(const pa_kv_pool* pool, const void* q,
                                    const int32_t* block_tables, int32_t bt_stride,
                                    const int32_t* context_lens, int32_t batch, int32_t num_q_heads,
                                    float scale, int32_t max_context_len, int32_t partition_size,
                                    int32_t prefix_len, int32_t prefix_partition_size,
                                    const int32_t* group_start, int32_t num_groups,
                                    int32_t max_group_size, int32_t group_len, const int32_t* items,
                                    int32_t num_items, float* partial_out, float* partial_lse,
                                    int32_t* trace, int64_t trace_capacity, void* stream) {
  const char* fn = "paged_attn_decode_cascade_trace";
  if (group_len < 0) return fail(PA_EINVAL, "%s: group_len = %d < 0", fn, group_len);
  return cascade_impl(pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale,
                      max_context_len, partition_size, prefix_len, prefix_partition_size,
                      partial_out, partial_lse, stream, fn, items != nullptr, items, num_items,
                      group_len > 0 ? group_start : nullptr, group_len > 0 ? num_groups : 0,
                      max_group_size, group_len, trace, trace_capacity, true);
}

int paged_attn_check_tables(const pa_kv_pool* pool, const int32_t* block_tables, int32_t bt_stride,
                            const int32_t* context_lens, int32_t batch, int32_t prefix_len,
                            const int32_t* group_start, int32_t num_groups, int32_t group_len,
                            int32_t* bad_seq_out) {
  const char* fn = "paged_attn_check_tables";
  if (bad_seq_out) *bad_seq_out = -1;
  if (!pool) return fail(PA_EINVAL, "%s: pool is NULL", fn);
  if (batch < 0) return fail(PA_EINVAL, "%s: batch = %d < 0", fn, batch);
  if (bt_stride < 1 || (int64_t)bt_stride * PA_BLOCK_SIZE > 0x7fffffffLL)
    return fail(PA_EINVAL, "%s: bt_stride = %d outside [1, 2^27)", fn, bt_stride);
  if (prefix_len < 0 || prefix_len % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: prefix_len = %d is not a non-negative multiple of %d", fn, prefix_len,
                PA_BLOCK_SIZE);
  if (group_len < 0 || group_len % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: group_len = %d is not a non-negative multiple of %d", fn, group_len,
                PA_BLOCK_SIZE);
  if (batch == 0) return PA_OK;
  if (!block_tables || !context_lens) return fail(PA_EINVAL, "%s: NULL table or lengths", fn);
  auto bad = [&](int32_t b) {
    if (bad_seq_out) *bad_seq_out = b;
    return PA_EINVAL;
  };
  const int64_t cap = (int64_t)bt_stride * PA_BLOCK_SIZE;
  // every entry a sequence's own context uses is a block of the pool
  for (int32_t b = 0; b < batch; ++b) {
    const int64_t n = context_lens[b];
    if (n < 0 || n > cap) {
      fail(PA_EINVAL, "%s: context_lens[%d] = %lld outside [0, 16 * bt_stride = %lld]", fn, b,
           (long long)n, (long long)cap);
      return bad(b);
    }
    const int32_t* row = block_tables + (size_t)b * bt_stride;
    for (int64_t j = 0; j < (n + PA_BLOCK_SIZE - 1) / PA_BLOCK_SIZE; ++j)
      if (row[j] < 0 || row[j] >= pool->num_blocks) {
        fail(PA_EINVAL, "%s: block_tables[%d][%lld] = %d is not a block of the pool (0 .. %d)", fn, b,
             (long long)j, row[j], pool->num_blocks - 1);
        return bad(b);
      }
  }
  // Sequence b's tokens t < min(ctx_b, end) of a shared span [begin, end)
  // are read through row `owner` instead of row b: those entries must match.
  auto shared = [&](int32_t b, int32_t owner, int64_t begin, int64_t end, const char* what) {
    const int64_t n = std::min<int64_t>(context_lens[b], end);
    const int32_t* row = block_tables + (size_t)b * bt_stride;
    const int32_t* own = block_tables + (size_t)owner * bt_stride;
    for (int64_t j = begin / PA_BLOCK_SIZE; j < (n + PA_BLOCK_SIZE - 1) / PA_BLOCK_SIZE; ++j)
      if (row[j] != own[j]) {
        fail(PA_EINVAL, "%s: block_tables[%d][%lld] = %d differs from %s block %d in row %d", fn, b,
             (long long)j, row[j], what, own[j], owner);
        return false;
      }
    return true;
  };
  if (prefix_len > 0) {
    if (prefix_len > cap) return fail(PA_EINVAL, "%s: prefix_len exceeds the table", fn);
    for (int32_t b = 1; b < batch; ++b)
      if (!shared(b, 0, 0, prefix_len, "the shared-prefix")) return bad(b);
  }
  if (group_len > 0) {
    if ((int64_t)prefix_len + group_len > cap) return fail(PA_EINVAL, "%s: prefix_len + group_len exceeds the table", fn);
    if (!group_start || num_groups < 1 || num_groups > batch)
      return fail(PA_EINVAL, "%s: group_start is NULL or num_groups = %d outside [1, batch]", fn, num_groups);
    if (group_start[0] != 0 || group_start[num_groups] != batch)
      return fail(PA_EINVAL, "%s: group_start must run from 0 to batch = %d", fn, batch);
    for (int32_t k = 0; k < num_groups; ++k) {
      const int32_t s0 = group_start[k], s1 = group_start[k + 1];
      if (s1 < s0) return fail(PA_EINVAL, "%s: group_start decreases at group %d", fn, k);
      for (int32_t b = s0 + 1; b < s1; ++b)
        if (!shared(b, s0, prefix_len, (int64_t)prefix_len + group_len, "its group's")) return bad(b);
    }
  }
  return PA_OK;
}

int paged_attn_schedule(const int32_t* context_lens, int32_t batch, int32_t max_context_len,
                        int32_t partition_size, int32_t prefix_len, int32_t* items,
                        int32_t capacity, int32_t* num_items) {
  const char* fn = "paged_attn_schedule";
  if (!num_items) return fail(PA_EINVAL, "%s: num_items is NULL", fn);
  if (batch < 0) return fail(PA_EINVAL, "%s: batch = %d < 0", fn, batch);
  if (max_context_len < 0) return fail(PA_EINVAL, "%s: max_context_len = %d < 0", fn, max_context_len);
  if (partition_size < 0 || partition_size % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: partition_size = %d is not a non-negative multiple of %d", fn,
                partition_size, PA_BLOCK_SIZE);
  if (prefix_len < 0 || prefix_len > max_context_len)
    return fail(PA_EINVAL, "%s: prefix_len = %d outside [0, max_context_len]", fn, prefix_len);
  if (batch > 0 && !context_lens) return fail(PA_EINVAL, "%s: context_lens is NULL", fn);
  // The partitioning of the call that will use the list.
  int64_t size, parts;
  if (prefix_len == 0) {
    Plan pl;
    const int rc = plan(max_context_len, partition_size, &pl, fn);
    if (rc) return rc;
    size = pl.part_tokens;
    parts = pl.num_parts;
  } else {
    if (partition_size == 0)
      return fail(PA_EINVAL, "%s: a cascade needs partition_size > 0", fn);
    size = partition_size;
    parts = ((int64_t)max_context_len - prefix_len + size - 1) / size;
  }
  if (parts * batch > 0x7fffffffLL) return fail(PA_EINVAL, "%s: too many work items", fn);
  // A single-partition decode without a prefix writes the output row of every
  // sequence (zeros for an empty one), so every sequence keeps its item; any
  // split launch skips empty partitions and the reduce covers them.
  const bool keep_empty = prefix_len == 0 && parts == 1;
  std::vector<ItemLen> list;
  list.reserve((size_t)(parts * batch));
  const bool seq_major = item_order_for((int32_t)parts) == 1;
  for (int64_t i = 0; i < parts * batch; ++i) {
    const int64_t part = seq_major ? i % parts : i / batch;
    const int32_t b = (int32_t)(seq_major ? i / parts : i % batch);
    int64_t n = context_lens[b];
    n = n < 0 ? 0 : (n > max_context_len ? max_context_len : n);
    const int64_t len = std::min<int64_t>(size, n - prefix_len - part * size);
    if (len > 0 || keep_empty)
      list.push_back({(int32_t)std::max<int64_t>(len, 0), (int32_t)(part * batch + b)});
  }
  // Longest first; ties in the order of the unscheduled grid (sequence-major
  // from 16 partitions on, else partition-major), so the list is deterministic.
  std::stable_sort(list.begin(), list.end(),
                   [](const ItemLen& x, const ItemLen& y) { return x.len > y.len; });
  *num_items = (int32_t)list.size();
  if ((int64_t)list.size() > capacity)
    return fail(PA_EINVAL, "%s: %d work items exceed capacity %d", fn, (int32_t)list.size(), capacity);
  if (!list.empty() && !items) return fail(PA_EINVAL, "%s: items is NULL", fn);
  for (size_t i = 0; i < list.size(); ++i) items[i] = list[i].item;
  return PA_OK;
}

namespace {
int reduce_impl(const float* partial_out, const float* partial_lse, const int32_t* context_lens,
                int32_t batch, int32_t num_q_heads, int32_t head_dim, int32_t partition_size,
                int32_t max_partitions, int32_t prefix_parts, int32_t prefix_len, void* out,
                void* stream, const char* fn) {
  if (batch < 0) return fail(PA_EINVAL, "%s: batch = %d < 0", fn, batch);
  if (num_q_heads <= 0) return fail(PA_EINVAL, "%s: num_q_heads = %d <= 0", fn, num_q_heads);
  if (head_dim != 64 && head_dim != 128)
    return fail(PA_EUNSUPPORTED, "%s: head_dim = %d (supported: 64, 128)", fn, head_dim);
  if (partition_size <= 0 || partition_size % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: partition_size = %d is not a positive multiple of %d", fn,
                partition_size, PA_BLOCK_SIZE);
  if (max_partitions <= 0) return fail(PA_EINVAL, "%s: max_partitions = %d <= 0", fn, max_partitions);
  if (prefix_parts > max_partitions)
    return fail(PA_EINVAL, "%s: %d prefix partitions exceed max_partitions = %d", fn, prefix_parts,
                max_partitions);
  if ((int64_t)batch * num_q_heads > 0x7fffffffLL) return fail(PA_EINVAL, "%s: grid too large", fn);
  if (batch == 0) return PA_OK;
  if (!partial_out || !partial_lse || !context_lens || !out)
    return fail(PA_EINVAL, "%s: NULL buffer", fn);
  if (!aligned(partial_out, 8) || !aligned(partial_lse, 4) || !aligned(context_lens, 4) ||
      !aligned(out, 4))
    return fail(PA_EINVAL, "%s: misaligned buffer", fn);
  pa::ReduceParams p{};
  p.part_o = partial_out;
  p.part_lse = partial_lse;
  p.context_lens = context_lens;
  p.out = static_cast<uint16_t*>(out);
  p.batch = batch;
  p.num_q_heads = num_q_heads;
  p.part_tokens = partition_size;
  p.part_stride = max_partitions;
  p.prefix_parts = prefix_parts;
  p.prefix_len = prefix_len;
  hipError_t e = pa::launch_reduce(p, head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(PA_EHIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return PA_OK;
}
}  // namespace

int paged_attn_reduce(const float* partial_out, const float* partial_lse,
                      const int32_t* context_lens, int32_t batch, int32_t num_q_heads,
                      int32_t head_dim, int32_t partition_size, int32_t max_partitions, void* out,
                      void* stream) {
  return reduce_impl(partial_out, partial_lse, context_lens, batch, num_q_heads, head_dim,
                     partition_size, max_partitions, 0, 0, out, stream, "paged_attn_reduce");
}

int paged_attn_reduce_cascade(const float* partial_out, const float* partial_lse,
                              const int32_t* context_lens, int32_t batch, int32_t num_q_heads,
                              int32_t head_dim, int32_t partition_size, int32_t prefix_len,
                              int32_t prefix_partition_size, int32_t max_partitions, void* out,
                              void* stream) {
  const char* fn = "paged_attn_reduce_cascade";
  if (prefix_len < 0 || prefix_len % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: prefix_len = %d is not a non-negative multiple of %d", fn,
                prefix_len, PA_BLOCK_SIZE);
  if (prefix_partition_size < PA_BLOCK_SIZE || prefix_partition_size > 64 * PA_BLOCK_SIZE ||
      prefix_partition_size % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: prefix_partition_size = %d not a multiple of 16 in [16, 1024]", fn,
                prefix_partition_size);
  const int32_t pre_parts = (prefix_len + prefix_partition_size - 1) / prefix_partition_size;
  return reduce_impl(partial_out, partial_lse, context_lens, batch, num_q_heads, head_dim,
                     partition_size, max_partitions, pre_parts, prefix_len, out, stream, fn);
}

int paged_attn_reduce_cascade_groups(const float* partial_out, const float* partial_lse,
                                     const int32_t* context_lens, int32_t batch,
                                     int32_t num_q_heads, int32_t head_dim, int32_t partition_size,
                                     int32_t prefix_len, int32_t prefix_partition_size,
                                     int32_t group_len, int32_t max_partitions, void* out,
                                     void* stream) {
  const char* fn = "paged_attn_reduce_cascade_groups";
  if (prefix_len < 0 || prefix_len % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: prefix_len = %d is not a non-negative multiple of %d", fn,
                prefix_len, PA_BLOCK_SIZE);
  if (prefix_partition_size < PA_BLOCK_SIZE || prefix_partition_size > 64 * PA_BLOCK_SIZE ||
      prefix_partition_size % PA_BLOCK_SIZE != 0)
    return fail(PA_EINVAL, "%s: prefix_partition_size = %d not a multiple of 16 in [16, 1024]", fn,
                prefix_partition_size);
  if (group_len <= 0 || group_len % PA_BLOCK_SIZE != 0 || group_len > 64 * PA_BLOCK_SIZE)
    return fail(PA_EINVAL, "%s: group_len = %d not a multiple of 16 in [16, 1024]", fn, group_len);
  // every sequence has the prefix partitions and its group's partition
  const int32_t shared_parts = (prefix_len + prefix_partition_size - 1) / prefix_partition_size + 1;
  return reduce_impl(partial_out, partial_lse, context_lens, batch, num_q_heads, head_dim,
                     partition_size, max_partitions, shared_parts, prefix_len + group_len, out,
                     stream, fn);
}

int paged_attn_extend(const pa_kv_pool* pool, const void* q, const int32_t* q_start, int32_t total_q,
                      const int32_t* block_tables, int32_t bt_stride, const int32_t* context_lens,
                      int32_t batch, int32_t num_q_heads, float scale, int32_t max_context_len,
                      int32_t max_chunk, void* out, void* stream) {
  const char* fn = "paged_attn_extend";
  DecodeArgs a{pool, q, block_tables, bt_stride, context_lens, batch, num_q_heads, scale, max_context_len};
  int32_t group = 0;
  int rc = validate_decode(a, &group, fn);
  if (rc) return rc;
  if (pool->head_dim != 128)
    return fail(PA_EUNSUPPORTED, "%s: head_dim = %d (the extend tiles need 128)", fn, pool->head_dim);
  if (max_context_len > pa::kExtendMaxTokens)
    return fail(PA_EUNSUPPORTED, "%s: max_context_len = %d exceeds %d", fn, max_context_len,
                pa::kExtendMaxTokens);
  if (total_q < 0) return fail(PA_EINVAL, "%s: total_q = %d < 0", fn, total_q);
  if (max_chunk < 0 || max_chunk > max_context_len)
    return fail(PA_EINVAL, "%s: max_chunk = %d outside [0, max_context_len = %d]", fn, max_chunk,
                max_context_len);
  const int64_t groups = ((int64_t)max_chunk * group + pa::kExtendRowsPerWg - 1) / pa::kExtendRowsPerWg;
  if ((int64_t)batch * groups * pool->num_kv_heads > 0x7fffffffLL)
    return fail(PA_EINVAL, "%s: grid too large", fn);
  if (batch == 0 || total_q == 0 || max_chunk == 0) return PA_OK;
  if (!q_start || !out) return fail(PA_EINVAL, "%s: q_start and out must be non-NULL", fn);
  if (!aligned(q_start, 4)) return fail(PA_EINVAL, "%s: q_start is not 4-byte aligned", fn);
  if (!aligned(out, 16)) return fail(PA_EINVAL, "%s: out is not 16-byte aligned", fn);
  pa::ExtendParams p{};
  p.k_pool = pool->k;
  p.v_pool = pool->v;
  p.q = static_cast<const uint16_t*>(q);
  p.q_start = q_start;
  p.block_tables = block_tables;
  p.context_lens = context_lens;
  p.out = static_cast<uint16_t*>(out);
  p.num_blocks = pool->num_blocks;
  p.num_kv_heads = pool->num_kv_heads;
  p.num_q_heads = num_q_heads;
  p.batch = batch;
  p.bt_stride = bt_stride;
  p.max_ctx = max_context_len;
  p.max_chunk = max_chunk;
  p.total_q = total_q;
  p.groups = (int32_t)groups;
  p.scale_log2 = scale * 1.4426950408889634f;
  hipError_t e = pa::launch_extend(p, group, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(PA_EHIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return PA_OK;
}

int paged_attn_append_kv(const pa_kv_pool* pool, const void* k_new, const void* v_new,
                         const int32_t* block_tables, int32_t bt_stride, const int32_t* context_lens,
                         int32_t batch, void* stream) {
  const char* fn = "paged_attn_append_kv";
  if (!pool) return fail(PA_EINVAL, "%s: pool is NULL", fn);
  if (batch < 0) return fail(PA_EINVAL, "%s: batch = %d < 0", fn, batch);
  if (bt_stride < 1) return fail(PA_EINVAL, "%s: bt_stride = %d < 1", fn, bt_stride);
  if ((int64_t)bt_stride * PA_BLOCK_SIZE > 0x7fffffffLL)
    return fail(PA_EINVAL, "%s: bt_stride = %d too large", fn, bt_stride);
  if (batch == 0) return PA_OK;
  if (!k_new || !v_new || !block_tables || !context_lens)
    return fail(PA_EINVAL, "%s: k_new, v_new, block_tables and context_lens must be non-NULL", fn);
  if (!aligned(k_new, 16) || !aligned(v_new, 16))
    return fail(PA_EINVAL, "%s: k_new/v_new are not 16-byte aligned", fn);
  if (!aligned(block_tables, 4) || !aligned(context_lens, 4))
    return fail(PA_EINVAL, "%s: block_tables/context_lens are not 4-byte aligned", fn);
  pa::AppendParams p{};
  p.k_pool = pool->k;
  p.v_pool = pool->v;
  p.k_new = static_cast<const uint16_t*>(k_new);
  p.v_new = static_cast<const uint16_t*>(v_new);
  p.block_tables = block_tables;
  p.context_lens = context_lens;
  p.num_blocks = pool->num_blocks;
  p.num_kv_heads = pool->num_kv_heads;
  p.head_dim = pool->head_dim;
  p.bt_stride = bt_stride;
  p.batch = batch;
  hipError_t e = pa::launch_append(p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(PA_EHIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return PA_OK;
}

int pa_stream_copy(const void* src, void* dst, size_t bytes, void* stream) {
  if (!src || !dst) return fail(PA_EINVAL, "pa_stream_copy: NULL pointer");
  if (bytes % 16 != 0 || !aligned(src, 16) || !aligned(dst, 16))
    return fail(PA_EINVAL, "pa_stream_copy: size and pointers must be 16-byte multiples/aligned");
  hipError_t e = pa::launch_stream_copy(src, dst, bytes, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(PA_EHIP, "pa_stream_copy: kernel launch failed: %s", hipGetErrorString(e));
  return PA_OK;
}

int pa_gather_tiles(const pa_kv_pool* pool, const int32_t* block_tables, int32_t bt_stride,
                    int32_t batch, const int32_t* spans, int32_t num_spans,
                    int32_t tiles_in_flight, uint32_t* sink, void* stream) {
  const char* fn = "pa_gather_tiles";
  if (!pool) return fail(PA_EINVAL, "%s: NULL pool", fn);
  if (num_spans < 0) return fail(PA_EINVAL, "%s: num_spans %d < 0", fn, num_spans);
  if (tiles_in_flight != 2 && tiles_in_flight != 4)
    return fail(PA_EINVAL, "%s: tiles_in_flight %d must be 2 or 4", fn, tiles_in_flight);
  if (num_spans == 0) return PA_OK;
  if (!block_tables || !spans || !sink) return fail(PA_EINVAL, "%s: NULL pointer", fn);
  if (!aligned(block_tables, 4) || !aligned(spans, 4) || !aligned(sink, 4))
    return fail(PA_EINVAL, "%s: block_tables/spans/sink are not 4-byte aligned", fn);
  if (batch < 1 || bt_stride < 1)
    return fail(PA_EINVAL, "%s: batch %d and bt_stride %d must be >= 1", fn, batch, bt_stride);
  if ((int64_t)bt_stride * PA_BLOCK_SIZE > 0x7fffffffLL)
    return fail(PA_EINVAL, "%s: bt_stride %d: the table row spans more than 2^31 tokens", fn, bt_stride);
  if ((int64_t)num_spans * pool->num_kv_heads > 0x7fffffffLL)
    return fail(PA_EINVAL, "%s: %d spans x %d KV heads exceed the grid limit", fn, num_spans,
                pool->num_kv_heads);
  hipError_t e = pa::launch_gather_tiles(pool->k, pool->v, pool->num_blocks, pool->num_kv_heads,
                                         pool->head_dim, block_tables, bt_stride, batch, spans,
                                         num_spans, tiles_in_flight, sink,
                                         static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(PA_EHIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return PA_OK;
}

}  // extern "C"
