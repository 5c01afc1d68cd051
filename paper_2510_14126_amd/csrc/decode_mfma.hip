// Split-KV paged decode attention on MFMA tiles for GQA groups of 8 (gfx950).
//
// With eight query heads per KV head, QK^T and PV of a 16-token block are
// dense enough for the matrix cores:
//
//  * S^T = K Q^T with v_mfma_f32_16x16x32_bf16: A = the K tile (16 tokens x 32
//    dims per instruction, 4 instructions for D = 128), loaded straight from
//    the pool in the same "token lane" order as the VALU kernel; B = Q^T with
//    the eight query rows in columns 0..7 (columns 8..15 repeat them).  Lane
//    (q, n) = (lane >> 4, lane & 15) receives scores of tokens 4q..4q+3 for
//    query row n, which is exactly the A-operand layout of the PV product, so
//    the probabilities never move between lanes.
//  * O += P V with v_mfma_f32_16x16x16bf16_1k (one per 16 output dims): the
//    B operand needs 4 consecutive tokens of one dim per lane, so the V tile is
//    staged in LDS (row pitch 288 bytes) and read back with the transposing
//    ds_read_b64_tr_b16, which hands lane (q, n) V[4q..4q+3][dim n].
//
// The online softmax keeps one running max per query row, replicated over the
// four lane groups, and rescales the accumulator only when a block raises the
// max by more than kLazyRescale (log2 units): probabilities stay <= 2^8, the
// rescale branch is wave-uniform and rare.  P is rounded to bf16 for the
// matrix core and the row sum adds the same rounded values, so the result is
// an exact convex combination of the V rows up to fp32 accumulation.
// Tail rows are removed by select: score -inf and V row zero.
#include "kernels.h"
#include "pa_device.h"

namespace pa {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t lds_short4_t;
typedef __attribute__((address_space(3))) uint8_t lds_u8_t;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;

constexpr int kD = 128;
constexpr int kG = 8;
constexpr int kWaves = 4;
constexpr int kPitch = kD * 2 + 32;           // LDS bytes per staged V token row
constexpr int kVTileBytes = 16 * kPitch;      // one staged V tile
constexpr float kLazyRescale = 8.0f;

struct MfmaTile {
  uint4 k[4];  // token n, K chunks 4s+q (16 bytes each)
  uint4 v[4];  // token n, V chunks 4s+q
};

__device__ __forceinline__ void load_tile(MfmaTile& T, const uint16_t* __restrict__ kt,
                                          const uint16_t* __restrict__ vt, int q, int n) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    T.k[s] = *reinterpret_cast<const uint4*>(kt + n * kD + (4 * s + q) * 8);
    T.v[s] = *reinterpret_cast<const uint4*>(vt + n * kD + (4 * s + q) * 8);
  }
}

// All-reduce over the four 16-lane groups (lanes n, n+16, n+32, n+48).
__device__ __forceinline__ float group_max4(float x) {
  float a = x, b = x;
  swap32(a, b);
  float y = fmaxf(a, b);
  float c = y, d = y;
  swap16(c, d);
  return fmaxf(c, d);
}
__device__ __forceinline__ float group_sum4(float x) {
  float a = x, b = x;
  swap32(a, b);
  float y = a + b;
  float c = y, d = y;
  swap16(c, d);
  return c + d;
}

struct MfmaState {
  float m;            // running max of query row n (log2 units), same in all groups
  float l;            // this lane's share of the row sum (tokens 4q..4q+3 of each block)
  floatx4_t o[8];     // O[rows 4q+r][dims 16*blk + n]
};

template <bool TAIL>
__device__ __forceinline__ void process_tile(MfmaState& S, const MfmaTile& T, const uint4 (&qb)[4],
                                             lds_u8_t* vbuf, int valid, int q, int n,
                                             float scale_log2) {
  // Stage V (token n, chunks 4s+q) into LDS; tail rows become zero.
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    u32x4_t v = {T.v[s].x, T.v[s].y, T.v[s].z, T.v[s].w};
    if (TAIL && n >= valid) v = u32x4_t{0u, 0u, 0u, 0u};
    *reinterpret_cast<lds_u32x4_t*>(vbuf + n * kPitch + (4 * s + q) * 16) = v;
  }

  floatx4_t st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s)
    st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, T.k[s]),
                                                 __builtin_bit_cast(bf16x8_t, qb[s]), st, 0, 0, 0);

  float sc[4];
  float bm = -__builtin_inff();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float x = st[r] * scale_log2;
    if (TAIL && 4 * q + r >= valid) x = -__builtin_inff();
    sc[r] = x;
    bm = fmaxf(bm, x);
  }
  bm = group_max4(bm);
  const bool raise = bm > S.m + kLazyRescale;
  if (__builtin_amdgcn_ballot_w64(raise) != 0) {
    const float mn = raise ? bm : S.m;
    const float alpha = fast_exp2(S.m - mn);   // 1 for rows that keep their max
    S.l *= alpha;
    S.m = mn;
    // Accumulator rows are indexed by lane group: row 4q+r takes alpha of lane 4q+r.
    float ar[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float a_lo = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), r));
      const float a_hi = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), 4 + r));
      ar[r] = q == 0 ? a_lo : (q == 1 ? a_hi : 0.f);
    }
#pragma unroll
    for (int blk = 0; blk < 8; ++blk)
#pragma unroll
      for (int r = 0; r < 4; ++r) S.o[blk][r] *= ar[r];
  }

  // Probabilities, rounded to bf16 for the matrix core; the row sum uses the
  // same rounded values.
  __bf16 pb[4];
  float lsum = 0.f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    pb[r] = (__bf16)fast_exp2(sc[r] - S.m);
    lsum += (float)pb[r];
  }
  S.l += lsum;
  short4_t pa;
#pragma unroll
  for (int r = 0; r < 4; ++r) pa[r] = __builtin_bit_cast(short, pb[r]);

  // PV: B operand = V[4q..4q+3][16*blk + n] through the transposing LDS read.
  // Source lane (q, n) points at token 4q + n/4, dims 16*blk + 4*(n%4).
  lds_u8_t* src = vbuf + (4 * q + (n >> 2)) * kPitch + (n & 3) * 8;
#pragma unroll
  for (int blk = 0; blk < 8; ++blk) {
    const short4_t vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<lds_short4_t*>(src + blk * 32));
    S.o[blk] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, vb, S.o[blk], 0, 0, 0);
  }
}

template <bool TRACE>
__global__ void __launch_bounds__(64 * kWaves) decode_mfma_g8_kernel(const DecodeParams p) {
  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int q = lane >> 4;
  const int n = lane & 15;

  int wg = blockIdx.x;
  const int g = wg % p.num_kv_heads;
  wg /= p.num_kv_heads;
  const int b = wg % p.batch;
  const int part = wg / p.batch;

  int ctx = p.context_lens[b];
  ctx = ctx < 0 ? 0 : (ctx > p.max_ctx ? p.max_ctx : ctx);
  const int start = part * p.part_tokens;
  const bool split = p.num_parts > 1;
  if (split && start >= ctx) return;
  const int end = min(ctx, start + p.part_tokens);
  const int nblk = end > start ? (end - start + 15) >> 4 : 0;
  const int j0 = start >> 4;
  const int h0 = g * kG;

  __shared__ __attribute__((aligned(16))) uint8_t smem[kWaves * 2 * kVTileBytes];
  lds_u8_t* lds = (lds_u8_t*)smem;  // C-style cast: generic to LDS address space
  lds_u8_t* vbufs[2] = {lds + (wave * 2) * kVTileBytes, lds + (wave * 2 + 1) * kVTileBytes};

  // Q^T operand: column n holds query row n % 8; dims 32s + 8q .. +8.
  uint4 qb[4];
  {
    const uint16_t* qrow = p.q + ((size_t)b * p.num_q_heads + h0 + (n & 7)) * kD;
#pragma unroll
    for (int s = 0; s < 4; ++s) qb[s] = *reinterpret_cast<const uint4*>(qrow + (4 * s + q) * 8);
  }

  MfmaState S;
  S.m = -__builtin_inff();
  S.l = 0.f;
#pragma unroll
  for (int blk = 0; blk < 8; ++blk) S.o[blk] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  const int32_t* bt = p.block_tables + (size_t)b * p.bt_stride + j0;
  constexpr size_t kTileElems = 16 * kD;
  const size_t blk_stride = (size_t)p.num_kv_heads * kTileElems;
  const uint16_t* kbase = p.k_pool + (size_t)g * kTileElems;
  const uint16_t* vbase = p.v_pool + (size_t)g * kTileElems;
  const size_t item = ((size_t)part * p.batch + b) * p.num_kv_heads + g;
  int flip = 0;

  for (int c0 = 0; c0 < nblk; c0 += 64) {
    const int cn = min(64, nblk - c0);
    const int raw = lane < cn ? bt[c0 + lane] : 0;
    const int idc = min(max(raw, 0), p.num_blocks - 1);
    auto tile_of = [&](int i, const uint16_t*& kt, const uint16_t*& vt) {
      const size_t id = (size_t)__builtin_amdgcn_readlane(idc, i);
      kt = kbase + id * blk_stride;
      vt = vbase + id * blk_stride;
    };
    auto run = [&](const MfmaTile& T, int i) {
      const int valid = min(16, end - (start + (c0 + i) * 16));
      lds_u8_t* vb = vbufs[flip];
      flip ^= 1;
      if (valid == 16)
        process_tile<false>(S, T, qb, vb, 16, q, n, p.scale_log2);
      else
        process_tile<true>(S, T, qb, vb, valid, q, n, p.scale_log2);
      if constexpr (TRACE) {
        if (lane == 0) {
          int32_t* tr = p.trace + (item * p.trace_tiles + (c0 + i)) * 3;
          tr[0] = j0 + c0 + i;
          tr[1] = __builtin_amdgcn_readlane(raw, i);
          tr[2] = valid;
        }
      }
    };

    int i = wave;
    if (i >= cn) continue;
    MfmaTile TA, TB;
    const uint16_t *kt, *vt;
    tile_of(i, kt, vt);
    load_tile(TA, kt, vt, q, n);
    while (true) {
      int nx = i + kWaves;
      if (nx < cn) { tile_of(nx, kt, vt); load_tile(TB, kt, vt, q, n); }
      run(TA, i);
      if (nx >= cn) break;
      i = nx;
      nx = i + kWaves;
      if (nx < cn) { tile_of(nx, kt, vt); load_tile(TA, kt, vt, q, n); }
      run(TB, i);
      if (nx >= cn) break;
      i = nx;
    }
  }

  // Merge the waves through LDS (the V staging area is free now).
  const float lrow = group_sum4(S.l);
  __syncthreads();
  float* sm = reinterpret_cast<float*>(smem);               // [W][8]
  float* sl = sm + kWaves * kG;                              // [W][8]
  float* sacc = sl + kWaves * kG;                            // [W][8][128]
  if (q == 0 && n < kG) { sm[wave * kG + n] = S.m; sl[wave * kG + n] = lrow; }
  if (q < 2) {
#pragma unroll
    for (int blk = 0; blk < 8; ++blk)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        sacc[(wave * kG + 4 * q + r) * kD + 16 * blk + n] = S.o[blk][r];
  }
  __syncthreads();
  if (wave != 0) return;

#pragma unroll
  for (int r = 0; r < kG; ++r) {
    float mx = sm[r];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) mx = fmaxf(mx, sm[w * kG + r]);
    const float mref = (mx == -__builtin_inff()) ? 0.f : mx;
    float lt = 0.f, o0 = 0.f, o1 = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = fast_exp2(sm[w * kG + r] - mref);
      lt = fmaf(sl[w * kG + r], f, lt);
      const float2 a = *reinterpret_cast<const float2*>(sacc + (w * kG + r) * kD + 2 * lane);
      o0 = fmaf(a.x, f, o0);
      o1 = fmaf(a.y, f, o1);
    }
    const float inv = lt > 0.f ? 1.0f / lt : 0.f;
    if (!split) {
      uint16_t* orow = p.out + ((size_t)b * p.num_q_heads + h0 + r) * kD;
      *reinterpret_cast<uint32_t*>(orow + 2 * lane) = bf16_rne(o0 * inv) | (bf16_rne(o1 * inv) << 16);
    } else {
      const size_t row = ((size_t)b * p.num_q_heads + h0 + r) * p.num_parts + part;
      *reinterpret_cast<float2*>(p.part_o + row * kD + 2 * lane) = make_float2(o0 * inv, o1 * inv);
      if (lane == 0)
        p.part_lse[row] = lt > 0.f ? (mx + log2f(lt)) * kLn2 : -__builtin_inff();
    }
  }
}

}  // namespace

hipError_t launch_decode_mfma(const DecodeParams& p, bool trace, hipStream_t stream) {
  const int64_t grid = (int64_t)p.num_parts * p.batch * p.num_kv_heads;
  if (trace)
    hipLaunchKernelGGL(decode_mfma_g8_kernel<true>, dim3((unsigned)grid), dim3(64 * kWaves), 0,
                       stream, p);
  else
    hipLaunchKernelGGL(decode_mfma_g8_kernel<false>, dim3((unsigned)grid), dim3(64 * kWaves), 0,
                       stream, p);
  return hipGetLastError();
}

}  // namespace pa
