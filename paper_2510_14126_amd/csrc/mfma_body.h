// Split-KV paged decode attention on MFMA tiles for GQA groups of 8 (gfx950).
//
// With eight query heads per KV head, QK^T and PV of a 16-token block are
// dense enough for the matrix cores:
//
//  * Both tiles of a block are read from the pool in row order: each 16-lane
//    group takes one whole 256-byte token row, so a load instruction reads
//    1 KiB of contiguous memory and the vector L1 sees one access per 64
//    bytes.  (Reading the MFMA operand layout straight from the pool would
//    put 16 different rows in every 16-lane group, about one L1 access per
//    lane, and the L1 becomes the limit when the tiles come from L2.)  Lane
//    (q, n) = (lane >> 4, lane & 15) then holds tokens 4u+q (u = 0..3),
//    dims 8n .. 8n+7, of both tiles.
//  * S^T = K Q^T with v_mfma_f32_16x16x32_bf16: A = K rows (16 tokens x 32
//    dims per instruction, 4 instructions for D = 128) read back from an LDS
//    copy of the K tile (k_stage: XOR-swizzled 256-byte rows, so writes and
//    reads spread over the banks); B = Q^T with the query rows in its 16
//    columns.  A row i
//    is token 4(i%4) + i/4, so lane (q, n) receives the scores of tokens
//    4r+q (r = 0..3) for query column n.
//  * O += P V with v_mfma_f32_16x16x16bf16_1k, one per 8 output dims: the
//    contraction index k = 4q+e stands for token 4e+q, which makes the
//    scores above exactly the A operand (P never moves between lanes), and
//    output column n of instruction j is dim 8n + j, which makes the B
//    operand V[token 4e+q][dim 8n+j] element j of the lane's own V registers
//    (two v_perm_b32 per instruction; V never goes through LDS).
//
// The online softmax keeps one running max per query row, replicated over the
// four lane groups, and rescales the accumulator only when a block raises the
// max by more than kLazyRescale (log2 units): probabilities stay <= 2^8, the
// rescale branch is wave-uniform and rare.  Each probability reaches the
// matrix core as a bf16 pair (high part and the rounded remainder, two MFMAs
// per PV step), which carries it to about 2^-17 relative; the row sum adds the
// fp32 values.
// Tail rows are removed by select: score -inf and V row zero.
#pragma once

#include "kernels.h"
#include "pa_device.h"

namespace pa {
namespace mfma {


typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t lds_short4_t;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;

constexpr int kD = 128;
constexpr int kG = 8;
constexpr int kWaves = 4;
constexpr int kKPitch = kD * 2;               // LDS bytes per staged K token row (swizzled, k_stage)
constexpr int kStageBytes = 16 * kKPitch;     // one staged K tile
constexpr float kLazyRescale = 8.0f;
#ifndef PA_MFMA_NBUF
#define PA_MFMA_NBUF 3
#endif
constexpr int kNbuf = PA_MFMA_NBUF;  // tiles kept in flight per wavefront

struct MfmaTile {
  uint4 k[4];  // [u]: row 4u+q, 16-byte chunk n of the K tile
  uint4 v[4];  // [u]: row 4u+q, chunk n of the V tile
};


// Rows 4u+q, chunk n of one K or V tile (lane_off = the byte offset of row q,
// chunk n) through a buffer descriptor built from the wave-uniform tile
// address; `bytes` = 0 makes the loads no-ops that return zeros but still
// count as issued.  AUX: the loads' cache policy (kLoadDefault or
// kLoadStreaming).
template <int AUX>
__device__ __forceinline__ void load_chunks(uint4 (&dst)[4], const uint16_t* tile, uint32_t lane_off,
                                            int bytes) {
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(tile), 0, bytes, kBufferDescWord3);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const auto x =
        __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)lane_off + u * 4 * kD * 2, 0, AUX);
    dst[u] = make_uint4(x[0], x[1], x[2], x[3]);
  }
}

// Value of query column 4q+r (held by lane 4q+r) for the accumulator rows
// of lane group q.
__device__ __forceinline__ float column_value(float x, int q, int r) {
  const int xi = __builtin_bit_cast(int, x);
  const float c0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(xi, r));
  const float c1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(xi, 4 + r));
  const float c2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(xi, 8 + r));
  const float c3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(xi, 12 + r));
  return q == 0 ? c0 : (q == 1 ? c1 : (q == 2 ? c2 : c3));
}

// Online-softmax state of NT column tiles (16 query columns each).
template <int NT>
struct MfmaState {
  float m[NT];        // running max of query column n (log2 units), same in all groups
  float l[NT];        // this lane's share of the column sum (tokens 4q..4q+3 of each block)
  floatx4_t o[NT][8]; // [j]: O[rows 4q+r][dim 8n + j] (tile_core) or [dim 16j + n] (tile_core_nb)
};

// One 16-token block against NT column tiles that share the K and V
// operands (their MFMA chains are independent and interleave).
// ka[s]: A operand of k-step s (token 4(n%4) + n/4, chunk 4s+q of the K
// tile); vrow[u]: the lane's V registers (token 4u+q, chunk n); `valid`:
// tokens of this tile that exist (V rows past it are zeroed); `limit[t]`:
// tokens this lane's column of tile t may attend to (<= valid).
template <bool TAIL, int NT>
__device__ __forceinline__ void tile_core(MfmaState<NT>& S, const u32x4_t (&ka)[4],
                                          const uint4 (&vrow)[4], const uint4 (&qb)[NT][4],
                                          int valid, const int (&limit)[NT], int q,
                                          float scale_log2) {

  // Two independent accumulation chains per tile, summed at the end.
  floatx4_t st[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const floatx4_t z = {0.f, 0.f, 0.f, 0.f};
    floatx4_t a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        __builtin_bit_cast(bf16x8_t, ka[0]), __builtin_bit_cast(bf16x8_t, qb[t][0]), z, 0, 0, 0);
    floatx4_t b = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        __builtin_bit_cast(bf16x8_t, ka[1]), __builtin_bit_cast(bf16x8_t, qb[t][1]), z, 0, 0, 0);
    a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ka[2]),
                                                __builtin_bit_cast(bf16x8_t, qb[t][2]), a, 0, 0, 0);
    b = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ka[3]),
                                                __builtin_bit_cast(bf16x8_t, qb[t][3]), b, 0, 0, 0);
    st[t] = a + b;
  }

  // Scores of tokens 4r+q; the rescale test needs no cross-lane reduction:
  // any lane above its column's max + kLazyRescale triggers it.
  float sc[NT][4];
  bool raise = false;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float x = st[t][r] * scale_log2;
      if (TAIL && 4 * r + q >= limit[t]) x = -__builtin_inff();
      sc[t][r] = x;
      raise |= x > S.m[t] + kLazyRescale;
    }
  }
  if (__builtin_amdgcn_ballot_w64(raise) != 0) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float bm = group_max4(fmaxf(fmaxf(sc[t][0], sc[t][1]), fmaxf(sc[t][2], sc[t][3])));
      const float mn = bm > S.m[t] + kLazyRescale ? bm : S.m[t];
      // 1 for columns that keep their max (or have attended to nothing yet)
      const float alpha = mn == -__builtin_inff() ? 1.f : fast_exp2(S.m[t] - mn);
      S.l[t] *= alpha;
      S.m[t] = mn;
      // Accumulator rows are indexed by lane group: row 4q+r takes alpha of
      // column 4q+r, held by lane 4q+r.
      float ar[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) ar[r] = column_value(alpha, q, r);
#pragma unroll
      for (int blk = 0; blk < 8; ++blk)
#pragma unroll
        for (int r = 0; r < 4; ++r) S.o[t][blk][r] *= ar[r];
    }
  }

  // Probabilities as bf16 pairs for the matrix core: p = hi + lo, hi = bf16(p)
  // and lo = bf16(p - hi) (the difference is exact in fp32), so the PV
  // product sees each weight to about 2^-17 relative; the column sum adds the
  // fp32 values.
  short4_t pa[NT], pl[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const float mref = S.m[t] == -__builtin_inff() ? 0.f : S.m[t];  // fully masked: p = 0
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float pf = fast_exp2(sc[t][r] - mref);
      const __bf16 hi = (__bf16)pf;
      pa[t][r] = __builtin_bit_cast(short, hi);
      pl[t][r] = __builtin_bit_cast(short, (__bf16)(pf - (float)hi));
      ps += pf;
    }
    S.l[t] += ps;
  }

  // PV: instruction j takes B = V[token 4e+q][dim 8n+j], e = 0..3: bf16 j of
  // the lane's chunk in each of its four rows.  Tail rows become zero.
  uint32_t vw[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const bool keep = !(TAIL && 4 * u + q >= valid);
    vw[u][0] = keep ? vrow[u].x : 0u;
    vw[u][1] = keep ? vrow[u].y : 0u;
    vw[u][2] = keep ? vrow[u].z : 0u;
    vw[u][3] = keep ? vrow[u].w : 0u;
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
    const uint32_t lo = __builtin_amdgcn_perm(vw[1][j >> 1], vw[0][j >> 1], sel);
    const uint32_t hi = __builtin_amdgcn_perm(vw[3][j >> 1], vw[2][j >> 1], sel);
    const short4_t vb = __builtin_bit_cast(short4_t, make_uint2(lo, hi));
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      S.o[t][j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa[t], vb, S.o[t][j], 0, 0, 0);
      S.o[t][j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pl[t], vb, S.o[t][j], 0, 0, 0);
    }
  }
}

// Row of the K tile that lane (q, n) supplies as A row n: token 4(n%4) + n/4.
__device__ __forceinline__ int k_arow(int n) { return 4 * (n & 3) + (n >> 2); }

// LDS byte offset of 16-byte chunk c of token row r in a staged K tile:
// rows of 256 bytes, chunk c at position c ^ k_arow(r).  Writers (16 lanes
// per row, chunks 0..15) and A-operand readers (lane (q, n): row k_arow(n),
// chunk 4s+q, i.e. position (4s+q) ^ n since k_arow is its own inverse) then
// touch 16 distinct positions per instruction, with no padding.
__device__ __forceinline__ int k_stage(int r, int c) { return r * kKPitch + ((c ^ k_arow(r)) << 4); }

// Window position of row r in a staged V tile: v_swz(r) = (r ^ r/4) & 7.
// A transposing read of one window serves each group of 16 lanes from rows
// q, q+4, q+8, q+12, and v_swz puts those four rows at window positions
// that differ modulo 4, i.e. on four different sets of eight banks (a 32-byte
// window covers 8 of the 32 four-byte banks, and windows w and w+4 share
// them): each group's read is free of bank conflicts.
__device__ __forceinline__ int v_swz(int r) { return (r ^ (r >> 2)) & 7; }

// LDS byte offset of 16-byte chunk c (dims 8c .. 8c+7) of token row r in a
// staged V tile: rows of 256 bytes, each of eight 32-byte windows (dims
// 16w .. 16w+15) at window position w ^ v_swz(r).  Writers (16 lanes per
// row) fill whole rows.
__device__ __forceinline__ int v_stage(int r, int c) {
  return r * 256 + ((((c >> 1) ^ v_swz(r)) << 5) | ((c & 1) << 4));
}

// Lane (q, n)'s address in a staged V tile for the transposing read of
// window 0 (XOR j << 5 for window j): row q + 4(n/4), dims 4(n%4) .. +3.  The
// read hands lane n of group q element n%4 of the rows addressed by lanes
// 4k + n/4 of its group, i.e. V[token q + 4k][dim 16j + n] for k = 0..3.
__device__ __forceinline__ int v_tr(int q, int n) {
  const int r = q + 4 * (n >> 2);
  return r * 256 + (v_swz(r) << 5) + ((n & 3) << 3);
}

// One staged block in the shared-span pass and extend: its K tile (k_stage
// layout) then its V tile (v_stage layout).
constexpr int kPrefixKBytes = 16 * kKPitch;
constexpr int kPrefixStageBytes = kPrefixKBytes + 16 * kD * 2;
// The shared-prefix pass streams its blocks in pairs (one LDS stage and one
// barrier per pair) through a ring of kPrefixRing quarter-blocks: the first
// pair is loaded before the loop and each pair's successor while it is
// published.  Extend streams kExtendStageBlocks blocks per stage through
// kExtendRingSets sets of slots, each stage loaded kExtendLoadAhead stages
// before it is published (1 <= AHEAD <= SETS; stage j in set j % SETS).
// Measured fastest: the prefix pass as described (the generic loop at the
// same depth was 4% slower on the generator batch), extend at (2, 2, 2)
// (with one tile per wavefront that form needed 162 VGPRs and ran three
// wavefronts per SIMD; two tiles per wavefront need 218 and run two, and
// are faster).
constexpr int kPrefixStageBlocks = 2;
constexpr int kPrefixRing = 4;
constexpr int kExtendStageBlocks = 2;
constexpr int kExtendRingSets = 2;
constexpr int kExtendLoadAhead = 2;
static_assert(kPrefixRing == 2 * kPrefixStageBlocks, "two pairs of slots");
static_assert(kExtendStageBlocks % 2 == 0, "blocks go in pairs");
static_assert(1 <= kExtendLoadAhead && kExtendLoadAhead <= kExtendRingSets, "loads stay in the ring");

// NB 16-token blocks (NB even) staged at st + b * kPrefixStageBytes (K in the
// k_stage layout, V in the v_stage layout) against NT column tiles, which
// share every K and V operand read from LDS.  The
// QK^T of every block comes first (independent MFMA chains); lane (q, n)
// then holds the scores of tokens 4r+q of each block for column n, and one
// online-softmax step covers all NB*16 tokens.  For PV, blocks 2p and 2p+1
// form the contraction index k = 8q + e (token 4e+q of block 2p for e < 4,
// token 4(e-4)+q of block 2p+1 for e >= 4), so the lane's eight
// probabilities are exactly the A operand of one v_mfma_f32_16x16x32_bf16
// per 16 output dims (output column n = dim 16j + n), whose B operand two
// transposing LDS reads deliver straight from the staged V tiles (vtr is
// the lane's v_tr offset).  valid[b]: rows of block b that hold tokens of the
// span (0: an empty block); lim[t][b]: rows of block b that column n of
// tile t may see.  Rows past valid[b] are zeroed in the B operand (their V may be
// anything, NaN included).  With FOLD (scale_log2 >= 0 required) the scale
// is applied inside the exponent's FMA, and the running-max test uses the
// lane's largest unmasked raw score times the scale (the same value as the
// largest scaled score, since multiplying by a non-negative number keeps
// the order).
template <bool TAIL, int NB, int NT, bool FOLD = false>
__device__ __forceinline__ void tile_core_nb(MfmaState<NT>& S, const lds_u8_t* st, int vtr,
                                             const uint4 (&qb)[NT][4], const int (&valid)[NB],
                                             const int (&lim)[NT][NB], int q, int n, float scale_log2) {
  static_assert(NB % 2 == 0, "blocks go in pairs through the PV contraction");
  const floatx4_t z = {0.f, 0.f, 0.f, 0.f};
  // K operands of every block first (shared by the NT tiles), then the score
  // MFMAs interleaved over tiles and blocks so that consecutive MFMAs do not
  // depend on each other.
  u32x4_t ka[NB][4];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int c = 0; c < 4; ++c)
      ka[b][c] = *reinterpret_cast<const lds_u32x4_t*>(st + b * kPrefixStageBytes + k_stage(k_arow(n), 4 * c + q));
  floatx4_t a[NT][NB];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int b = 0; b < NB; ++b)
      a[t][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ka[b][0]),
                                                        __builtin_bit_cast(bf16x8_t, qb[t][0]), z, 0, 0, 0);
#pragma unroll
  for (int c = 1; c < 4; ++c)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int b = 0; b < NB; ++b)
        a[t][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ka[b][c]),
                                                          __builtin_bit_cast(bf16x8_t, qb[t][c]), a[t][b], 0, 0, 0);

  // Probabilities of tile t as bf16 pairs (the A operands: element e of
  // pa[t][p] and pl[t][p] is the high and low part of the weight of score
  // 8p + e, p = hi + lo to about 2^-17 relative); the column sum adds the fp32
  // values.
  bf16x8_t pa[NT][NB / 2], pl[NT][NB / 2];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    float sc[4 * NB];   // scaled scores, or raw ones with FOLD
    bool raise = false;
    float mx = -__builtin_inff();   // FOLD: the lane's largest unmasked raw score
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if constexpr (FOLD) {
          const float raw = a[t][b][r];
          sc[4 * b + r] = raw;
          if (!TAIL || 4 * r + q < lim[t][b]) mx = fmaxf(mx, raw);
        } else {
          float x = a[t][b][r] * scale_log2;
          if (TAIL && 4 * r + q >= lim[t][b]) x = -__builtin_inff();
          sc[4 * b + r] = x;
          raise |= x > S.m[t] + kLazyRescale;
        }
      }
    const float xmax = mx * scale_log2;   // FOLD only (NaN when all are masked and the scale is 0)
    if constexpr (FOLD) raise = xmax > S.m[t] + kLazyRescale;
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
      float bmax = sc[0];
      if constexpr (FOLD) {
        bmax = xmax;
      } else {
#pragma unroll
        for (int e = 1; e < 4 * NB; ++e) bmax = fmaxf(bmax, sc[e]);
      }
      const float bm = group_max4(bmax);
      const float mn = bm > S.m[t] + kLazyRescale ? bm : S.m[t];
      const float alpha = mn == -__builtin_inff() ? 1.f : fast_exp2(S.m[t] - mn);
      S.l[t] *= alpha;
      S.m[t] = mn;
      float ar[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) ar[r] = column_value(alpha, q, r);
#pragma unroll
      for (int blk = 0; blk < 8; ++blk)
#pragma unroll
        for (int r = 0; r < 4; ++r) S.o[t][blk][r] *= ar[r];
    }

    const float mref = S.m[t] == -__builtin_inff() ? 0.f : S.m[t];
    float lsum = 0.f;
#pragma unroll
    for (int pp = 0; pp < NB / 2; ++pp) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float ex;
        if constexpr (FOLD) {
          ex = fmaf(sc[8 * pp + e], scale_log2, -mref);
          // element e is token 4(e % 4) + q of block 2pp + e / 4
          if (TAIL && 4 * (e & 3) + q >= lim[t][2 * pp + (e >> 2)]) ex = -__builtin_inff();
        } else {
          ex = sc[8 * pp + e] - mref;
        }
        const float pf = fast_exp2(ex);
        const __bf16 hi = (__bf16)pf;
        pa[t][pp][e] = hi;
        pl[t][pp][e] = (__bf16)(pf - (float)hi);
        lsum += pf;
      }
    }
    S.l[t] += lsum;
  }

  // Element e of a block's B words is its token 4e + q.
  uint32_t mlo[NB], mhi[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    mlo[b] = 0xffffffffu;
    mhi[b] = 0xffffffffu;
    if constexpr (TAIL) {
      mlo[b] = (q < valid[b] ? 0xffffu : 0u) | (q + 4 < valid[b] ? 0xffff0000u : 0u);
      mhi[b] = (q + 8 < valid[b] ? 0xffffu : 0u) | (q + 12 < valid[b] ? 0xffff0000u : 0u);
    }
  }
  // Each B operand (two transposing reads) serves the NT tiles.
#pragma unroll
  for (int pp = 0; pp < NB / 2; ++pp) {
    const lds_u8_t* v0 = st + (2 * pp) * kPrefixStageBytes + kPrefixKBytes;
    const lds_u8_t* v1 = v0 + kPrefixStageBytes;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int off = vtr ^ (j << 5);
      const uint2 b0 = __builtin_bit_cast(
          uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4_t*)(v0 + off)));
      const uint2 b1 = __builtin_bit_cast(
          uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4_t*)(v1 + off)));
      const u32x4_t vb = {b0.x & mlo[2 * pp], b0.y & mhi[2 * pp], b1.x & mlo[2 * pp + 1],
                          b1.y & mhi[2 * pp + 1]};
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        S.o[t][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa[t][pp], __builtin_bit_cast(bf16x8_t, vb),
                                                            S.o[t][j], 0, 0, 0);
        S.o[t][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl[t][pp], __builtin_bit_cast(bf16x8_t, vb),
                                                            S.o[t][j], 0, 0, 0);
      }
    }
  }
}


// One block of a per-sequence work item: the wavefront's own K tile goes
// through `stage` (kStageBytes of its LDS) to reach the A-operand layout;
// V is used from the registers it was loaded into.
template <bool TAIL, int NT>
__device__ __forceinline__ void process_tile(MfmaState<NT>& S, const MfmaTile& T,
                                             const uint4 (&qb)[NT][4], lds_u8_t* stage, int valid,
                                             const int (&limit)[NT], int q, int n,
                                             float scale_log2) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const u32x4_t k = {T.k[u].x, T.k[u].y, T.k[u].z, T.k[u].w};
    *reinterpret_cast<lds_u32x4_t*>(stage + k_stage(4 * u + q, n)) = k;
  }
  u32x4_t ka[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    ka[s] = *reinterpret_cast<const lds_u32x4_t*>(stage + k_stage(k_arow(n), 4 * s + q));
  tile_core<TAIL, NT>(S, ka, T.v, qb, valid, limit, q, scale_log2);
}

// LDS bytes either body needs (two staged K tiles per wavefront, then the
// end-of-item merge).
constexpr int kMergeLdsBytes = (2 * kWaves * 16 + kWaves * 16 * kD) * 4;  // up to 16 rows per wave
constexpr int kLdsBytes = kWaves * 2 * kStageBytes > kMergeLdsBytes ? kWaves * 2 * kStageBytes
                                                                    : kMergeLdsBytes;

// One decode work item (partition, sequence, KV head) = workgroup `wg_index`.
// STREAM: load the tiles as streaming data (the cascade's per-sequence half,
// whose tokens come after everything the sequences share and are normally
// read by this item only).  The hint changes caching, never the results.
// APPEND: the fused KV append (DecodeParams::k_new): the item that holds
// token ctx - 1 takes its K and V rows from k_new / v_new in registers
// (whatever the pool slot holds) and stores them into the slot.
template <bool TRACE, bool STREAM, bool APPEND = false>
__device__ __forceinline__ void decode_mfma_body(const DecodeParams& p, int wg_index, lds_u8_t* smem) {
  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int q = lane >> 4;
  const int n = lane & 15;

  int g, b, part;
  decode_item(p, wg_index, g, b, part);

  const int start = p.token_offset + part * p.part_tokens;
  const int j0 = start >> 4;
  const int h0 = g * kG;
  const int32_t* bt = p.block_tables + (size_t)b * p.bt_stride + j0;
  // The first 64 block ids and the query rows are loaded before the context
  // length arrives (j0 < bt_stride for every launched partition).
  const int raw_first = lane < min(64, p.bt_stride - j0) ? bt[lane] : 0;

  // Q^T operand: column n holds query row n % 8; dims 32s + 8q .. +8.
  uint4 qb[1][4];
  {
    const uint16_t* qrow = p.q + ((size_t)b * p.num_q_heads + h0 + (n & 7)) * kD;
#pragma unroll
    for (int s = 0; s < 4; ++s) qb[0][s] = *reinterpret_cast<const uint4*>(qrow + (4 * s + q) * 8);
  }

  int ctx = p.context_lens[b];
  ctx = ctx < 0 ? 0 : (ctx > p.max_ctx ? p.max_ctx : ctx);
  const bool split = p.write_partials != 0;
  if (split && start >= ctx) return;
  const int end = min(ctx, start + p.part_tokens);
  const int nblk = end > start ? (end - start + 15) >> 4 : 0;

  // Fused append: block jnew of this item (-1: none) holds the new token in
  // row rnew; knew / vnew are chunk n (dims 8n .. 8n+7) of its K and V rows.
  // The lanes of row group rnew % 4 store the rows.
  int jnew = -1, rnew = 0;
  uint4 knew = make_uint4(0, 0, 0, 0), vnew = make_uint4(0, 0, 0, 0);
  if constexpr (APPEND) {
    if (ctx > 0 && ctx - 1 >= start && ctx - 1 < end) {
      jnew = ((ctx - 1) >> 4) - j0;
      rnew = (ctx - 1) & 15;
      const size_t src = ((size_t)b * p.num_kv_heads + g) * kD + 8 * n;
      knew = *reinterpret_cast<const uint4*>(p.k_new + src);
      vnew = *reinterpret_cast<const uint4*>(p.v_new + src);
      if (wave == 0 && q == (rnew & 3)) {
        int phys = p.block_tables[(size_t)b * p.bt_stride + ((ctx - 1) >> 4)];
        phys = min(max(phys, 0), p.num_blocks - 1);
        const size_t dst = (((size_t)phys * p.num_kv_heads + g) * 16 + rnew) * kD + 8 * n;
        *reinterpret_cast<uint4*>(p.k_pool_w + dst) = knew;
        *reinterpret_cast<uint4*>(p.v_pool_w + dst) = vnew;
      }
    }
  }

  lds_u8_t* lds = smem;
  lds_u8_t* stages[2] = {lds + (wave * 2) * kStageBytes, lds + (wave * 2 + 1) * kStageBytes};

  MfmaState<1> S;
  S.m[0] = -__builtin_inff();
  S.l[0] = 0.f;
#pragma unroll
  for (int blk = 0; blk < 8; ++blk) S.o[0][blk] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  constexpr size_t kTileElems = 16 * kD;
  const size_t blk_stride = (size_t)p.num_kv_heads * kTileElems;
  const uint16_t* kbase = p.k_pool + (size_t)g * kTileElems;
  const uint16_t* vbase = p.v_pool + (size_t)g * kTileElems;
  const size_t item = ((size_t)part * p.batch + b) * p.num_kv_heads + g;
  const uint32_t lane_off = (uint32_t)(q * kD + n * 8) * 2u;  // row q, chunk n (+ 4 rows per u)
  int flip = 0;

  for (int c0 = 0; c0 < nblk; c0 += 64) {
    const int cn = min(64, nblk - c0);
    const int raw = c0 == 0 ? (lane < cn ? raw_first : 0) : (lane < cn ? bt[c0 + lane] : 0);
    const int idc = min(max(raw, 0), p.num_blocks - 1);
    auto load = [&](MfmaTile& T, int i) {
      const bool ok = i < cn;
      const size_t id = (size_t)__builtin_amdgcn_readlane(idc, ok ? i : 0);
      const int bytes = ok ? (int)(kTileElems * 2) : 0;
      constexpr int kAux = STREAM ? kLoadStreaming : kLoadDefault;
      load_chunks<kAux>(T.k, kbase + id * blk_stride, lane_off, bytes);
      load_chunks<kAux>(T.v, vbase + id * blk_stride, lane_off, bytes);
    };
    auto run = [&](MfmaTile& T, int i) {
      const int valid = min(16, end - (start + (c0 + i) * 16));
      if constexpr (APPEND) {
        // the new token's rows replace whatever the slot held (the ring slot
        // is loaded again before its next use)
        if (c0 + i == jnew) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (4 * u + q == rnew) { T.k[u] = knew; T.v[u] = vnew; }
        }
      }
      lds_u8_t* vb = stages[flip];
      flip ^= 1;
      const int lim[1] = {valid};
      if (valid == 16)
        process_tile<false, 1>(S, T, qb, vb, 16, lim, q, n, p.scale_log2);
      else
        process_tile<true, 1>(S, T, qb, vb, valid, lim, q, n, p.scale_log2);
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
    MfmaTile T[kNbuf];
    int ld = i;
#pragma unroll
    for (int s = 0; s < kNbuf - 1; ++s) {
      load(T[s], ld);
      ld += kWaves;
    }
    bool done = false;
    while (!done) {
#pragma unroll
      for (int s = 0; s < kNbuf; ++s) {
        if (!done) {
          load(T[(s + kNbuf - 1) % kNbuf], ld);
          ld += kWaves;
          run(T[s], i);
          i += kWaves;
          done = i >= cn;
        }
      }
    }
  }

  // Merge the waves through LDS (the staging area is free now).
  const float lrow = group_sum4(S.l[0]);
  __syncthreads();
  lds_f32_t* sm = reinterpret_cast<lds_f32_t*>(smem);       // [W][8]
  lds_f32_t* sl = sm + kWaves * kG;                          // [W][8]
  lds_f32_t* sacc = sl + kWaves * kG;                        // [W][8][128]
  if (q == 0 && n < kG) { sm[wave * kG + n] = S.m[0]; sl[wave * kG + n] = lrow; }
  if (q < 2) {
#pragma unroll
    for (int blk = 0; blk < 8; ++blk)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        sacc[(wave * kG + 4 * q + r) * kD + 8 * n + blk] = S.o[0][blk][r];
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
      const float2 a = {sacc[(w * kG + r) * kD + 2 * lane], sacc[(w * kG + r) * kD + 2 * lane + 1]};
      o0 = fmaf(a.x, f, o0);
      o1 = fmaf(a.y, f, o1);
    }
    const float inv = lt > 0.f ? 1.0f / lt : 0.f;
    if (!split) {
      uint16_t* orow = p.out + ((size_t)b * p.num_q_heads + h0 + r) * kD;
      *reinterpret_cast<uint32_t*>(orow + 2 * lane) = bf16_rne(o0 * inv) | (bf16_rne(o1 * inv) << 16);
    } else {
      const size_t row = ((size_t)b * p.num_q_heads + h0 + r) * p.part_stride + p.part_offset + part;
      store_partial2(p.part_o + row * kD + 2 * lane, o0 * inv, o1 * inv);
      if (lane == 0)
        p.part_lse[row] = lt > 0.f ? (mx + log2f(lt)) * kLn2 : -__builtin_inff();
    }
  }
}

// Attention over the prefix that every sequence of the batch shares: for KV
// head g the B*G query rows form the columns of dense 16-row tiles (four
// sequences of four heads, or two of eight, per tile).  One workgroup owns
// kWaves adjacent tiles (wavefront w: tile w) and one prefix partition, and
// its wavefronts share every block: each loads one quarter (four token rows
// of K and of V, 2 KiB) into a double-buffered LDS stage, and after a
// barrier every wavefront runs its own tile against the staged blocks, two
// blocks per barrier through tile_core_nb.  A block
// thus crosses from L2 to the CU once per four tiles, and each wavefront owns
// whole query rows, so no cross-wavefront merge is needed.  All workgroups of
// a KV head read the same blocks, so each comes from HBM once and from L2
// afterwards.  Every row writes its (o, lse) partial for the partition,
// lse = -inf when it attended to nothing.
constexpr int kPrefixRowsPerWg = 16 * kWaves;
static_assert(kPrefixRowsPerWg == kSharedRowsPerWg, "the host sizes traces from kSharedRowsPerWg");
constexpr int kPrefixLdsBytes = 2 * kPrefixStageBlocks * kPrefixStageBytes;   // two stages

// Rows and tokens of one shared-span workgroup: rows R = row0 .. (16 per
// wavefront) of span rows 0 .. total_rows-1, row R being sequence seq0 + R / G
// and head g*G + R % G; tokens start .. end-1, whose block ids begin at bt;
// the result goes to partial slot `part`; the walk over the blocks starts at
// block `rot`.
struct SharedSpan {
  int seq0, total_rows, row0;
  int start, end;
  const int32_t* bt;
  int part;
  int rot;
};

template <int G, bool TRACE>
__device__ __forceinline__ void shared_span_body(const PrefixParams& p, int g, const SharedSpan& sp,
                                                 lds_u8_t* smem, int32_t* trace) {
  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int q = lane >> 4;
  const int n = lane & 15;

  const int total_rows = sp.total_rows;
  const int row0 = sp.row0 + 16 * wave;   // this wavefront's tile
  const int start = sp.start;
  const int end = sp.end;
  const int part = sp.part;
  const int nblk = (end - start + 15) >> 4;     // 1 .. 64 for every launched span
  const int raw = lane < nblk ? sp.bt[lane] : 0;
  const int idc = min(max(raw, 0), p.num_blocks - 1);

  // Column n is query row R = row0 + n: sequence seq0 + R / G, head g*G + R % G.
  uint4 qb[1][4];
  int ctx;
  int min_ctx;
  {
    const int R = row0 + n;
    const bool ok = R < total_rows;
    const int bR = ok ? sp.seq0 + R / G : 0;
    const uint16_t* qrow = p.q + ((size_t)bR * p.num_q_heads + g * G + R % G) * kD;
#pragma unroll
    for (int s = 0; s < 4; ++s)
      qb[0][s] = ok ? *reinterpret_cast<const uint4*>(qrow + (4 * s + q) * 8) : make_uint4(0, 0, 0, 0);
    int c = ok ? p.context_lens[bR] : 0;
    c = c < 0 ? 0 : (c > p.max_ctx ? p.max_ctx : c);
    ctx = c;
    // shortest context among the tile's columns (decides when to mask)
    min_ctx = __builtin_amdgcn_readfirstlane(-(int)group_max4(row_max16(-(float)c)));
  }

  MfmaState<1> S;
  S.m[0] = -__builtin_inff();
  S.l[0] = 0.f;
#pragma unroll
  for (int blk = 0; blk < 8; ++blk) S.o[0][blk] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  constexpr size_t kTileElems = 16 * kD;
  const size_t blk_stride = (size_t)p.num_kv_heads * kTileElems;
  // This wavefront's quarter of a tile: token row 4*wave + q, chunk n.
  const int share_off = ((4 * wave + q) * kD + n * 8) * 2;
  const int vtr = v_tr(q, n);
  const uint16_t* kbase = p.k_pool + (size_t)g * kTileElems;
  const uint16_t* vbase = p.v_pool + (size_t)g * kTileElems;

  const int rot = sp.rot;
  auto block_of = [&](int i) { const int j = i + rot; return j >= nblk ? j - nblk : j; };
  auto load = [&](uint4 (&dst)[2], int i) {
    const bool ok = i < nblk;
    const size_t id = (size_t)__builtin_amdgcn_readlane(idc, ok ? block_of(i) : 0);
    const int bytes = ok ? (int)(kTileElems * 2) : 0;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(kbase + id * blk_stride), 0, bytes, kBufferDescWord3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(vbase + id * blk_stride), 0, bytes, kBufferDescWord3);
    const auto k = __builtin_amdgcn_raw_buffer_load_b128(rk, share_off, 0, 0);
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(rv, share_off, 0, 0);
    dst[0] = make_uint4(k[0], k[1], k[2], k[3]);
    dst[1] = make_uint4(v[0], v[1], v[2], v[3]);
  };

  // The blocks go in pairs: every wavefront publishes its quarter of both
  // blocks of pair j to one LDS stage (double-buffered), loads the quarters
  // of pair j+1 into the other two ring slots, one barrier, then every
  // wavefront runs its tile against the pair.  The two blocks of a pair need
  // not be adjacent; an odd last block pairs with an empty one (valid = 0).
  constexpr int NB = 2;
  constexpr int kRing = kPrefixRing;
  uint4 ring[kRing][2];
#pragma unroll
  for (int s = 0; s < kRing - 2; ++s) load(ring[s], s);
  const int npair = (nblk + 1) >> 1;
  for (int j0 = 0; j0 < npair; j0 += kRing / 2) {
#pragma unroll
    for (int h = 0; h < kRing / 2; ++h) {
      const int j = j0 + h;
      if (j < npair) {                         // uniform over the workgroup
        lds_u8_t* st = smem + (j & 1) * 2 * kPrefixStageBytes;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          lds_u8_t* sb = st + e * kPrefixStageBytes;
          const int s = 2 * h + e;
          *reinterpret_cast<lds_u32x4_t*>(sb + k_stage(4 * wave + q, n)) =
              u32x4_t{ring[s][0].x, ring[s][0].y, ring[s][0].z, ring[s][0].w};
          *reinterpret_cast<lds_u32x4_t*>(sb + kPrefixKBytes + v_stage(4 * wave + q, n)) =
              u32x4_t{ring[s][1].x, ring[s][1].y, ring[s][1].z, ring[s][1].w};
        }
        load(ring[(2 * h + kRing - 2) % kRing], 2 * j + kRing - 2);
        load(ring[(2 * h + kRing - 1) % kRing], 2 * j + kRing - 1);
        __syncthreads();
        int valid[NB], lim[1][NB];
        bool fast = true;
#pragma unroll
        for (int s = 0; s < NB; ++s) {
          const int i = NB * j + s;
          const bool has = i < nblk;
          const int tb = has ? start + block_of(i) * 16 : end;
          valid[s] = has ? min(16, end - tb) : 0;
          lim[0][s] = min(valid[s], max(ctx - tb, 0));
          fast = fast && valid[s] == 16 && min_ctx - tb >= 16;
          if constexpr (TRACE) {
            // slot = the block's position in the span (not in the walk)
            const int bi = has ? block_of(i) : 0;
            const int id = __builtin_amdgcn_readlane(raw, bi);
            if (has && wave == 0 && lane == 0) {
              int32_t* tr = trace + 3 * bi;
              tr[0] = (start >> 4) + bi;
              tr[1] = id;
              tr[2] = valid[s];
            }
          }
        }
        if (fast)
          tile_core_nb<false, NB>(S, st, vtr, qb, valid, lim, q, n, p.scale_log2);
        else
          tile_core_nb<true, NB>(S, st, vtr, qb, valid, lim, q, n, p.scale_log2);
      }
    }
  }

  // Normalise per row and write this partition's partials: lane (q, n)
  // holds O[rows 4q+r][dims 16j + n], j = 0..7.
  const float lcol = group_sum4(S.l[0]);
  const float inv = lcol > 0.f ? 1.0f / lcol : 0.f;
  if (q == 0 && row0 + n < total_rows) {
    const int R = row0 + n;
    const size_t row = ((size_t)(sp.seq0 + R / G) * p.num_q_heads + g * G + R % G) * p.part_stride + part;
    p.part_lse[row] = lcol > 0.f ? (S.m[0] + log2f(lcol)) * kLn2 : -__builtin_inff();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int R = row0 + 4 * q + r;
    const float f = column_value(inv, q, r);
    if (R < total_rows) {
      const size_t row =
          ((size_t)(sp.seq0 + R / G) * p.num_q_heads + g * G + R % G) * p.part_stride + part;
      float* po = p.part_o + row * kD + n;
#pragma unroll
      for (int j = 0; j < 8; ++j) store_partial(po + 16 * j, S.o[0][j][r] * f);
    }
  }
}

// The batch-wide prefix: partition `part` of the prefix against row group
// `grp` (64 rows) of all B*G query rows of KV head g.
template <int G, bool TRACE>
__device__ __forceinline__ void prefix_mfma_body(const PrefixParams& p, int wg_index, lds_u8_t* smem) {
  const int total_rows = p.batch * G;
  const int groups = (total_rows + kPrefixRowsPerWg - 1) / kPrefixRowsPerWg;
  int wg = wg_index;
  const int g = wg % p.num_kv_heads;
  wg /= p.num_kv_heads;
  const int grp = wg % groups;
  const int part = wg / groups;
  SharedSpan sp;
  sp.seq0 = 0;
  sp.total_rows = total_rows;
  sp.row0 = grp * kPrefixRowsPerWg;
  sp.start = part * p.part_tokens;
  sp.end = min(p.prefix_len, sp.start + p.part_tokens);
  sp.bt = p.block_tables + (sp.start >> 4);
  sp.part = part;
  // The workgroups of a KV head walk the partition from evenly spread
  // starting blocks, so at any moment they read different blocks instead of
  // all queueing on the L2 lines of the same one.
  const int nblk = (sp.end - sp.start + 15) >> 4;
  sp.rot = (int)(((int64_t)grp * nblk) / groups) % nblk;
  int32_t* tr = nullptr;
  if constexpr (TRACE)
    tr = p.trace_prefix + (((size_t)part * groups + grp) * p.num_kv_heads + g) * p.prefix_trace_tiles * 3;
  shared_span_body<G, TRACE>(p, g, sp, smem, tr);
}

// The second level: group k's rows (its sequences x G heads of KV head g,
// at most 64) against the group_len tokens the group shares after the
// prefix, one partition written to slot prefix_parts.
template <int G, bool TRACE>
__device__ __forceinline__ void group_mfma_body(const PrefixParams& p, int wg_index, lds_u8_t* smem) {
  const int g = wg_index % p.num_kv_heads;
  const int k = wg_index / p.num_kv_heads;
  // device data: clamped into the batch and the stated bound
  int s0 = p.group_start[k];
  s0 = s0 < 0 ? 0 : (s0 > p.batch ? p.batch : s0);
  int s1 = p.group_start[k + 1];
  s1 = s1 < s0 ? s0 : (s1 > p.batch ? p.batch : s1);
  s1 = min(s1, s0 + p.max_group_size);
  if (s1 == s0) return;                        // whole workgroup: an empty group
  SharedSpan sp;
  sp.seq0 = s0;
  sp.total_rows = (s1 - s0) * G;
  sp.row0 = 0;
  sp.start = p.prefix_len;
  sp.end = p.prefix_len + p.group_len;
  sp.bt = p.block_tables + (size_t)s0 * p.bt_stride + (sp.start >> 4);
  sp.part = p.prefix_parts;
  sp.rot = 0;
  int32_t* tr = nullptr;
  if constexpr (TRACE)
    tr = p.trace_group + ((size_t)k * p.num_kv_heads + g) * p.group_trace_tiles * 3;
  shared_span_body<G, TRACE>(p, g, sp, smem, tr);
}

// Causal attention of a chunk of new tokens over its sequence's paged
// context (extend / chunked prefill).  For KV head g, the (chunk token i,
// head j) pairs of sequence b form rows R = i*G + j of dense 16-row tiles;
// row R sees the tokens 0 .. n - L + i (n: context with the chunk, L: chunk
// length), which is the per-column limit the MFMA core already applies.
// One workgroup owns kExtendRowsPerWg rows, kExtendTilesPerWave adjacent
// tiles per wavefront, and streams the sequence's blocks once through LDS
// for all of them, as the shared-prefix pass does, two blocks per barrier
// through tile_core_nb, whose K and V operand reads serve all of a
// wavefront's tiles; the stream stops at the workgroup's last visible token.
// Each wavefront normalises its rows and writes them as bf16.
constexpr int kExtendTilesPerWave = kExtendRowsPerWg / (16 * kWaves);
template <bool B> struct BoolTag { static constexpr bool value = B; };
static_assert(kExtendTilesPerWave * 16 * kWaves == kExtendRowsPerWg, "whole tiles per wavefront");
constexpr int kExtendIdOffset = 2 * kExtendStageBlocks * kPrefixStageBytes;   // after two stages
constexpr int kExtendLdsBytes = kExtendIdOffset + kExtendMaxTokens / 16 * 4;   // + the block ids

template <int G>
__device__ __forceinline__ void extend_mfma_body(const ExtendParams& p, int wg_index, lds_u8_t* smem) {
  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int q = lane >> 4;
  const int n = lane & 15;

  int wg = wg_index;
  const int g = wg % p.num_kv_heads;
  wg /= p.num_kv_heads;
  const int grp = wg % p.groups;
  const int b = wg / p.groups;

  int ctx = p.context_lens[b];
  ctx = ctx < 0 ? 0 : (ctx > p.max_ctx ? p.max_ctx : ctx);
  int qs = p.q_start[b];
  int L = p.q_start[b + 1] - qs;
  qs = qs < 0 ? 0 : qs;
  L = L < 0 ? 0 : (L > ctx ? ctx : (L > p.max_chunk ? p.max_chunk : L));
  L = qs + L > p.total_q ? (p.total_q > qs ? p.total_q - qs : 0) : L;
  const int rows = L * G;
  if (grp * kExtendRowsPerWg >= rows) return;          // whole workgroup: no rows here
  constexpr int NT = kExtendTilesPerWave;
  const int row0 = grp * kExtendRowsPerWg + 16 * NT * wave;   // this wavefront's first tile
  const int first = ctx - L;                           // position of chunk token 0

  // Tokens the workgroup needs: up to its last row's position.
  const int last_row = min(rows, (grp + 1) * kExtendRowsPerWg) - 1;
  const int vis_max = first + last_row / G + 1;
  const int nblk = (vis_max + 15) >> 4;

  // Block ids of the stream, clamped into the pool, staged once in LDS
  // (at most kExtendMaxTokens / 16 of them); each is read back as a
  // broadcast when its block is loaded.
  lds_i32_t* ids = reinterpret_cast<lds_i32_t*>(smem + kExtendIdOffset);
  {
    const int32_t* bt = p.block_tables + (size_t)b * p.bt_stride;
    for (int j = threadIdx.x; j < nblk; j += 64 * kWaves)
      ids[j] = min(max(bt[j], 0), p.num_blocks - 1);
    __syncthreads();
  }
  auto block_id = [&](int i) { return __builtin_amdgcn_readfirstlane(ids[i]); };

  // Column n of tile t is row R = row0 + 16t + n: chunk token R / G, query
  // head g*G + R % G.  A negative scale goes into the sign of Q (bf16
  // negation is exact, and so is the negation of every score), so the core
  // folds a non-negative scale into its exponent.
  const uint32_t qflip = p.scale_log2 < 0.f ? 0x80008000u : 0u;
  const float scale_abs = fabsf(p.scale_log2);
  uint4 qb[NT][4];
  int lim_col[NT];   // tokens column n of tile t sees
  {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int R = row0 + 16 * t + n;
      const bool ok = R < rows;
      const int i = ok ? R / G : 0;
      const uint16_t* qrow = p.q + ((size_t)(qs + i) * p.num_q_heads + g * G + R % G) * kD;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        uint4 w = ok ? *reinterpret_cast<const uint4*>(qrow + (4 * s + q) * 8) : make_uint4(0, 0, 0, 0);
        w.x ^= qflip; w.y ^= qflip; w.z ^= qflip; w.w ^= qflip;
        qb[t][s] = w;
      }
      lim_col[t] = ok ? first + i + 1 : 0;
    }
  }

  MfmaState<NT> S;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    S.m[t] = -__builtin_inff();
    S.l[t] = 0.f;
#pragma unroll
    for (int blk = 0; blk < 8; ++blk) S.o[t][blk] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  }

  constexpr size_t kTileElems = 16 * kD;
  const size_t blk_stride = (size_t)p.num_kv_heads * kTileElems;
  const int share_off = ((4 * wave + q) * kD + n * 8) * 2;   // token row 4*wave + q, chunk n
  const int vtr = v_tr(q, n);
  const uint16_t* kbase = p.k_pool + (size_t)g * kTileElems;
  const uint16_t* vbase = p.v_pool + (size_t)g * kTileElems;
  auto load = [&](uint4 (&dst)[2], int i) {
    const bool ok = i < nblk;
    const size_t id = (size_t)block_id(ok ? i : 0);
    const int bytes = ok ? (int)(kTileElems * 2) : 0;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(kbase + id * blk_stride), 0, bytes, kBufferDescWord3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(vbase + id * blk_stride), 0, bytes, kBufferDescWord3);
    const auto k = __builtin_amdgcn_raw_buffer_load_b128(rk, share_off, 0, 0);
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(rv, share_off, 0, 0);
    dst[0] = make_uint4(k[0], k[1], k[2], k[3]);
    dst[1] = make_uint4(v[0], v[1], v[2], v[3]);
  };

  // The blocks go NB at a time: every wavefront publishes its quarter of
  // each block of stage j to one LDS stage (double-buffered), loads the
  // quarters of stage j + AHEAD, one barrier, then every wavefront runs its
  // tiles against the stage.  Blocks past the stream are empty (valid = 0).
  constexpr int NB = kExtendStageBlocks;
  constexpr int SETS = kExtendRingSets;
  constexpr int AHEAD = kExtendLoadAhead;
  uint4 ring[SETS * NB][2];                     // stage j's blocks in slot set j % SETS
#pragma unroll
  for (int s = 0; s < AHEAD * NB; ++s) load(ring[s], s);
  const int nit = (nblk + NB - 1) / NB;
  // Stages 0 .. nfast-1 are wholly visible to every row of the workgroup
  // (its first row sees the fewest tokens) and run unmasked in a loop of
  // their own; the rest, up to the causal diagonal, run masked in a second
  // loop.  One core per loop keeps the compiler from copying the output
  // accumulators where the two cores' paths would otherwise merge.  nfast
  // is a multiple of SETS so that both loops find stage j in slot set
  // j % SETS.
  const int wg_min_lim = first + grp * kExtendRowsPerWg / G + 1;
  int nfast = min(wg_min_lim, vis_max) / (16 * NB);
  nfast = min(nfast - nfast % SETS, nit);
  auto stream = [&](auto tail, int jb, int je) {
  constexpr bool TAIL = decltype(tail)::value;
  for (int j0 = jb; j0 < je; j0 += SETS) {
#pragma unroll
  for (int h = 0; h < SETS; ++h) {
    const int j = j0 + h;
    if (j < je) {                               // uniform over the workgroup
      lds_u8_t* st = smem + (j & 1) * NB * kPrefixStageBytes;
#pragma unroll
      for (int s = 0; s < NB; ++s) {
        lds_u8_t* sb = st + s * kPrefixStageBytes;
        const uint4 (&rs)[2] = ring[h * NB + s];
        *reinterpret_cast<lds_u32x4_t*>(sb + k_stage(4 * wave + q, n)) =
            u32x4_t{rs[0].x, rs[0].y, rs[0].z, rs[0].w};
        *reinterpret_cast<lds_u32x4_t*>(sb + kPrefixKBytes + v_stage(4 * wave + q, n)) =
            u32x4_t{rs[1].x, rs[1].y, rs[1].z, rs[1].w};
      }
#pragma unroll
      for (int s = 0; s < NB; ++s) load(ring[((h + AHEAD) % SETS) * NB + s], NB * (j + AHEAD) + s);
      __syncthreads();

      int valid[NB], lim[NT][NB];
      const int t0 = NB * j * 16;
#pragma unroll
      for (int s = 0; s < NB; ++s) {
        const int tb = t0 + 16 * s;
        valid[s] = max(0, min(16, vis_max - tb));
#pragma unroll
        for (int t = 0; t < NT; ++t) lim[t][s] = min(valid[s], max(lim_col[t] - tb, 0));
      }
      tile_core_nb<TAIL, NB, NT, true>(S, st, vtr, qb, valid, lim, q, n, scale_abs);
    }
  }
  }
  };
  stream(BoolTag<false>{}, 0, nfast);
  stream(BoolTag<true>{}, nfast, nit);

  // Normalise and write bf16: lane (q, n) holds O[rows 4q+r of tile t][dims 16j + n].
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const float lcol = group_sum4(S.l[t]);
    const float inv = lcol > 0.f ? 1.0f / lcol : 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int R = row0 + 16 * t + 4 * q + r;
      const float f = column_value(inv, q, r);
      if (R < rows) {
        uint16_t* orow = p.out + ((size_t)(qs + R / G) * p.num_q_heads + g * G + R % G) * kD + n;
#pragma unroll
        for (int j = 0; j < 8; ++j) orow[16 * j] = (uint16_t)bf16_rne(S.o[t][j][r] * f);
      }
    }
  }
}

}  // namespace mfma
}  // namespace pa
