// Device-side helpers for the gfx950 (CDNA4) paged decode-attention kernels.
//
// Lane conventions used throughout: a wavefront has 64 lanes in four DPP
// "rows" of 16.  Lane `l` belongs to row group `l >> 4` and row position
// `l & 15`.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

constexpr int kBlockTokens = 16;  // tokens per KV block
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ---- bf16 ------------------------------------------------------------------

// Low / high bf16 of a packed pair, widened exactly to fp32.
__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

// fp32 -> bf16 bits with round-to-nearest-even; NaN stays a (quiet) NaN.
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Dot product of two bf16 pairs accumulated into fp32 (v_dot2c_f32_bf16).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// 2^x on the hardware transcendental unit (v_exp_f32); exp2(-inf) = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Split-KV partial rows are written once by the decode and read once by the
// reduce kernel.  They are stored with device scope (relaxed atomic stores at
// agent scope: plain vector stores with the sc1 bit), which writes them
// through L2 instead of leaving dirty lines among the KV tiles that the
// decode is still reading.  On the 8K-32K-token batch, where partials are 2%
// of the bytes moved, the decode measured 1.6% faster than with non-temporal
// stores and 8% faster than with default (write-back) stores.
__device__ __forceinline__ void store_partial(float* dst, float a) {
  __hip_atomic_store(dst, a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_partial2(float* dst, float a, float b) {
  const uint64_t v = ((uint64_t)__float_as_uint(b) << 32) | __float_as_uint(a);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(dst), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Cache-policy operand of a buffer load: bit 1 is the non-temporal hint of
// the gfx940 family.  Tiles that one step reads exactly once (a sequence's
// tokens after what the batch shares, in the cascade; every tile when the
// pool holds no shared block) are loaded with it, so they do not push lines
// that are still in use out of L2 and the infinity cache: 8-11% of the
// decode time on the long-context and shared-pool batches.  A line must be
// read whole by one instruction: one read in parts by several instructions
// can be evicted between them and fetched again.  Where blocks are shared
// between sequences the plain decode keeps the default (the hint cost 5%
// there on the long-context batch).
constexpr int kLoadDefault = 0;
constexpr int kLoadStreaming = 2;

// Fourth word of a raw buffer descriptor on gfx9-family GPUs (32-bit data
// format, no swizzle); the first three hold the base and the byte size.
constexpr int kBufferDescWord3 = 0x00020000;

// LDS (address space 3) pointer types.
typedef __attribute__((address_space(3))) uint8_t lds_u8_t;
typedef __attribute__((address_space(3))) float lds_f32_t;
typedef __attribute__((address_space(3))) int32_t lds_i32_t;

// ---- cross-lane movement ---------------------------------------------------

// DPP controls (gfx9 encoding).
constexpr int kDppQuadXor1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kDppRowRor4 = 0x124;   // row_ror:4
constexpr int kDppRowRor8 = 0x128;   // row_ror:8
constexpr int kDppRowNewBcast = 0x150;  // row_newbcast:n = 0x150 + n

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, true));
}

// Every lane of a 16-lane row gets the value of row position T.
template <int T>
__device__ __forceinline__ float row_bcast(float x) {
  return dpp<kDppRowNewBcast + T>(x);
}

constexpr int kDppRowHalfMirror = 0x141;  // lane i <-> 7 - i within each half-row of 8

// Max / sum over the 4 lanes of each quad; every lane receives the result.
__device__ __forceinline__ float quad_max4(float x) {
  x = fmaxf(x, dpp<kDppQuadXor1>(x));
  return fmaxf(x, dpp<kDppQuadXor2>(x));
}
__device__ __forceinline__ float quad_sum4(float x) {
  x += dpp<kDppQuadXor1>(x);
  return x + dpp<kDppQuadXor2>(x);
}

// Reduce-scatter over the 16 lanes of each DPP row without lane-dependent
// selects.  Every lane holds N partial values (N a multiple of 16) in slot
// order s; slot s of lane c must hold index s XOR M(c), where M is the
// GF(2)-linear map M(c) = b3 e3 + b2 (e2 + e1 + e0) + b1 e1 + b0 e0 on the
// top four bits of the index (b_i = bit i of c, e_j = bit j of s * 16 / N).
// Each level keeps the lower half of the slots and adds the partner's upper
// half; the partners (c^8 by row_ror 8, c^7 by row_half_mirror, c^2, c^1)
// hold the same indices there because M(partner flip) is exactly the bit the
// level consumes.  Afterwards lane c holds in x[0 .. N/16) the row-wide sums
// of indices M(c) * N/16 ...
template <int CTRL, int H, int N>
__device__ __forceinline__ void fold_level(float (&x)[N]) {
#pragma unroll
  for (int i = 0; i < H; ++i) x[i] = x[i] + dpp<CTRL>(x[i + H]);
}
template <int N>
__device__ __forceinline__ void row_reduce_scatter16(float (&x)[N]) {
  static_assert(N % 16 == 0, "N must be a multiple of 16");
  fold_level<kDppRowRor8, N / 2>(x);        // partner c ^ 8
  fold_level<kDppRowHalfMirror, N / 4>(x);  // partner c ^ 7
  fold_level<kDppQuadXor2, N / 8>(x);       // partner c ^ 2
  fold_level<kDppQuadXor1, N / 16>(x);      // partner c ^ 1
}

// Max / sum over the 16 lanes of each row; every lane receives the result.
__device__ __forceinline__ float row_max16(float x) {
  x = fmaxf(x, dpp<kDppQuadXor1>(x));
  x = fmaxf(x, dpp<kDppQuadXor2>(x));
  x = fmaxf(x, dpp<kDppRowRor4>(x));
  x = fmaxf(x, dpp<kDppRowRor8>(x));
  return x;
}
__device__ __forceinline__ float row_sum16(float x) {
  x += dpp<kDppQuadXor1>(x);
  x += dpp<kDppQuadXor2>(x);
  x += dpp<kDppRowRor4>(x);
  x += dpp<kDppRowRor8>(x);
  return x;
}

// v_permlane32_swap: a' = [a(0..31), b(0..31)], b' = [a(32..63), b(32..63)].
__device__ __forceinline__ void swap32(float& a, float& b) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(a), __float_as_int(b), false, false);
  a = __int_as_float(r[0]);
  b = __int_as_float(r[1]);
}
// v_permlane16_swap: a' rows = [a0, b0, a2, b2], b' rows = [a1, b1, a3, b3].
__device__ __forceinline__ void swap16(float& a, float& b) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(a), __float_as_int(b), false, false);
  a = __int_as_float(r[0]);
  b = __int_as_float(r[1]);
}

// Reduce-scatter over the four row groups: every lane holds partials
// x0..x3 (one per query row); afterwards the lanes of row group j hold the
// sum over the four groups of x_j, at the same row position.
__device__ __forceinline__ float reduce_scatter4(float x0, float x1, float x2, float x3) {
  swap32(x0, x2);
  swap32(x1, x3);
  float y0 = x0 + x2;  // groups 0,1: row 0 | groups 2,3: row 2
  float y1 = x1 + x3;  // groups 0,1: row 1 | groups 2,3: row 3
  swap16(y0, y1);
  return y0 + y1;      // group j: row j
}

// All-gather over the four row groups: lane (j, t) holds x_j(t); afterwards
// every lane (*, t) holds x_0(t) .. x_3(t).
__device__ __forceinline__ void allgather4(float x, float& r0, float& r1, float& r2, float& r3) {
  float a = x, b = x;
  swap32(a, b);        // a: rows of group j%2, b: rows of group j%2+2
  float c = a, d = b;
  swap16(a, c);        // a: x_0, c: x_1
  swap16(b, d);        // b: x_2, d: x_3
  r0 = a; r1 = c; r2 = b; r3 = d;
}

// All-reduce over the four 16-lane groups (lanes i, i+16, i+32, i+48).
__device__ __forceinline__ float group_max4(float x) {
  float a = x, b = x;
  swap32(a, b);
  const float y = fmaxf(a, b);
  float c = y, d = y;
  swap16(c, d);
  return fmaxf(c, d);
}
__device__ __forceinline__ float group_sum4(float x) {
  float a = x, b = x;
  swap32(a, b);
  const float y = a + b;
  float c = y, d = y;
  swap16(c, d);
  return c + d;
}

__device__ __forceinline__ int wave_uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

}  // namespace pa
