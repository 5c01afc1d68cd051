// Kernel parameter blocks and launchers shared by the C-ABI layer and the
// HIP kernels.  Host code fills these after validating every argument.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

// Sets the C ABI's thread-local error message (pa_last_error) and returns code.
int fail(int code, const char* fmt, ...);

struct DecodeParams {
  const uint16_t* k_pool;        // bf16 [num_blocks][num_kv_heads][16][D]
  const uint16_t* v_pool;        // same layout
  const uint16_t* q;             // bf16 [batch][num_q_heads][D]
  const int32_t* block_tables;   // [batch][bt_stride]
  const int32_t* context_lens;   // [batch]
  uint16_t* out;                 // bf16 [batch][num_q_heads][D] (single partition)
  float* part_o;                 // fp32 [batch][num_q_heads][num_parts][D] (split)
  float* part_lse;               // fp32 [batch][num_q_heads][num_parts]
  int32_t* trace;                // index trace (trace variant only)
  int32_t num_blocks;
  int32_t num_kv_heads;
  int32_t num_q_heads;
  int32_t batch;
  int32_t bt_stride;
  int32_t max_ctx;
  int32_t part_tokens;           // tokens per work item (a multiple of 16)
  int32_t num_parts;             // partitions in the grid
  int32_t token_offset;          // first token of partition 0 (a multiple of 16)
  int32_t part_offset;           // index of partition 0 in the partial buffers
  int32_t part_stride;           // partitions per (sequence, head) in the partial buffers
  int32_t write_partials;        // 1: write (o, lse) partials; 0: write the bf16 output
  int32_t trace_tiles;           // trace slots per work item
  int32_t item_order;            // workgroup -> work item order (decode_item)
  const int32_t* items;          // optional work list: item = part * batch + b, or NULL
  int32_t num_items;             // entries of items
  int32_t stream_tiles;          // 1: load the tiles with the streaming cache hint (plain decode)
  float scale_log2;              // softmax scale * log2(e)
  // Fused KV append (append kernels only): token ctx_b - 1 of every sequence
  // takes K and V from k_new / v_new [batch][num_kv_heads][D] bf16, and the
  // work item that holds it writes them into the pools.
  const uint16_t* k_new;
  const uint16_t* v_new;
  uint16_t* k_pool_w;            // the same pools as k_pool / v_pool, written
  uint16_t* v_pool_w;
};

// Work items (partition, sequence) of a decode grid; one workgroup per item
// and KV head.
__host__ __device__ inline int64_t decode_items(const DecodeParams& p) {
  return p.items ? (int64_t)p.num_items : (int64_t)p.num_parts * p.batch;
}

// Work item (KV head g, sequence b, partition part) of decode workgroup wg.
// The KV head varies fastest, so consecutive workgroups, which the
// dispatcher deals to the XCDs round-robin, keep one KV head per XCD.  Then
// the host's work list when there is one, else either all sequences'
// partition 0, then partition 1, ... (item_order 0), or all partitions of
// sequence 0, then sequence 1, ... (item_order 1).
__device__ __forceinline__ void decode_item(const DecodeParams& p, int wg, int& g, int& b, int& part) {
  g = wg % p.num_kv_heads;
  wg /= p.num_kv_heads;
  if (p.items) {                 // host-built list (device data: clamped into the grid)
    int it = p.items[wg];
    const int last = p.num_parts * p.batch - 1;
    it = it < 0 ? 0 : (it > last ? last : it);
    b = it % p.batch;
    part = it / p.batch;
  } else if (p.item_order == 0) {
    b = wg % p.batch;
    part = wg / p.batch;
  } else {
    part = wg % p.num_parts;
    b = wg / p.num_parts;
  }
}

// Attention of every query row of the batch over a prefix that all
// sequences share (same physical blocks, read from sequence 0's table), and
// optionally, one level down, of each group of sequences over the tokens
// that the group shares after the prefix (read from the group's first
// sequence's table).
struct PrefixParams {
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const uint16_t* q;
  const int32_t* block_tables;   // [batch][bt_stride]
  const int32_t* context_lens;
  float* part_o;                 // partitions [0, prefix_parts (+1)) of the partial buffers
  float* part_lse;
  int32_t num_blocks;
  int32_t num_kv_heads;
  int32_t num_q_heads;
  int32_t batch;
  int32_t bt_stride;
  int32_t prefix_len;            // shared tokens (a multiple of 16)
  int32_t part_tokens;           // tokens per prefix partition (a multiple of 16)
  int32_t prefix_parts;          // ceil(prefix_len / part_tokens)
  int32_t part_stride;
  int32_t max_ctx;
  // Second level (num_groups > 0): group k is sequences group_start[k] ..
  // group_start[k+1]-1 (at most max_group_size of them), sharing group_len
  // tokens after the prefix; its partial is partition prefix_parts.
  const int32_t* group_start;    // device [num_groups + 1]
  int32_t num_groups;
  int32_t max_group_size;        // max_group_size * G <= 64 (one workgroup per group)
  int32_t group_len;             // a multiple of 16, at most 1024
  float scale_log2;
  // Index trace (trace launches only): the tiles of prefix partition part,
  // row group rg, KV head g at trace_prefix + ((part * row_groups + rg) *
  // num_kv_heads + g) * prefix_trace_tiles triples; those of group k at
  // trace_group + (k * num_kv_heads + g) * group_trace_tiles triples.
  int32_t* trace_prefix;
  int32_t* trace_group;
  int32_t prefix_trace_tiles;    // part_tokens / 16
  int32_t group_trace_tiles;     // group_len / 16
};

// Query rows (sequence x head of one KV head) per workgroup of the shared
// passes: four wavefronts, one 16-row tile each.
constexpr int kSharedRowsPerWg = 64;

struct ReduceParams {
  const float* part_o;
  const float* part_lse;
  const int32_t* context_lens;
  uint16_t* out;
  int32_t batch;
  int32_t num_q_heads;
  int32_t part_tokens;           // suffix partition size
  int32_t part_stride;           // partitions per (sequence, head) in the buffers
  int32_t prefix_parts;          // leading partitions that every sequence has
  int32_t prefix_len;            // tokens covered by those partitions
};

// VALU split-KV decode (group size 4 or 8, head_dim 64 or 128).
hipError_t launch_decode_valu(const DecodeParams& p, int head_dim, int group, bool trace,
                              hipStream_t stream);
// MFMA split-KV decode for group size 8, head_dim 128.
hipError_t launch_decode_mfma(const DecodeParams& p, bool trace, hipStream_t stream);
// Shared-prefix pass and per-sequence decode in one launch (head_dim 128;
// the decode half uses VALU for group 4 and MFMA for group 8).
hipError_t launch_cascade(const PrefixParams& pp, const DecodeParams& dp, int group, bool trace,
                          hipStream_t stream);
// Log-sum-exp merge of split-KV partials into the bf16 output.
hipError_t launch_reduce(const ReduceParams& p, int head_dim, hipStream_t stream);
// Causal attention of a chunk of new tokens per sequence over its paged
// context (extend / chunked prefill).
struct ExtendParams {
  const uint16_t* k_pool;        // bf16 [num_blocks][num_kv_heads][16][128]
  const uint16_t* v_pool;
  const uint16_t* q;             // bf16 [total_q][num_q_heads][128], chunks packed
  const int32_t* q_start;        // [batch + 1]: chunk b is rows q_start[b] .. q_start[b+1]-1
  const int32_t* block_tables;   // [batch][bt_stride]
  const int32_t* context_lens;   // [batch], the chunk included
  uint16_t* out;                 // bf16 [total_q][num_q_heads][128]
  int32_t num_blocks;
  int32_t num_kv_heads;
  int32_t num_q_heads;
  int32_t batch;
  int32_t bt_stride;
  int32_t max_ctx;               // bound of context_lens (at most kExtendMaxTokens)
  int32_t max_chunk;             // bound of the chunk lengths
  int32_t total_q;               // rows of q and out
  int32_t groups;                // row groups per sequence in the grid
  float scale_log2;
};
hipError_t launch_extend(const ExtendParams& p, int group, hipStream_t stream);
constexpr int kExtendMaxTokens = 8192;   // context bound of one extend launch
constexpr int kExtendRowsPerWg = 128;    // query rows (chunk token x head) per extend workgroup

// Append of one token's K and V rows per sequence.
struct AppendParams {
  uint16_t* k_pool;              // bf16 [num_blocks][num_kv_heads][16][head_dim]
  uint16_t* v_pool;
  const uint16_t* k_new;         // bf16 [batch][num_kv_heads][head_dim]
  const uint16_t* v_new;
  const int32_t* block_tables;   // [batch][bt_stride]
  const int32_t* context_lens;   // [batch], the new token included
  int32_t num_blocks;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t bt_stride;
  int32_t batch;
};
hipError_t launch_append(const AppendParams& p, hipStream_t stream);
// Streaming device copy (measurement helper).
hipError_t launch_stream_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);

// Reads the K and V tiles of token spans ([num_spans][3] int32: sequence,
// first token, end token) for every KV head, with no arithmetic, keeping
// tiles_in_flight (2 or 4) tiles in flight per wavefront.
hipError_t launch_gather_tiles(const void* k_pool, const void* v_pool, int num_blocks,
                               int num_kv_heads, int head_dim, const int32_t* block_tables,
                               int bt_stride, int batch, const int32_t* spans, int num_spans,
                               int tiles_in_flight, uint32_t* sink, hipStream_t stream);

}  // namespace pa
