// Split-KV paged decode attention on VALU dot products (gfx950).
//
// One workgroup handles one work item (partition p, sequence b, KV head g):
// the G query heads g*G .. g*G+G-1 that share KV head g attend to the
// tokens [p*S, min((p+1)*S, ctx_b)) of sequence b.  Its W wavefronts take
// the partition's 16-token KV blocks round-robin, each keeping its own
// online-softmax state, and merge through LDS at the end.  Each wavefront
// keeps NBUF tiles in a register ring, so the next NBUF-1 blocks stream in
// while one is being computed.
//
// A 16-token block of one KV head is a K tile and a V tile (16 x D bf16,
// contiguous in the pool).  Both are read in "quad lanes": lane (J, c) =
// (lane >> 4, lane & 15) holds dims (D/16)*c .. of tokens 4u+J, u = 0..3,
// so one 16-byte (8-byte at D = 64) load instruction reads four whole token
// rows, contiguous in memory, and a lane needs only its (D/16)-dim slice of
// the G query rows.
//
//  * QK^T: each lane forms 4G partial dot products (v_dot2c_f32_bf16) over
//    its dims; a DPP reduce-scatter across the 16 lanes of the row (ror 8,
//    half-mirror, quad xor 2, quad xor 1) leaves in lane (J, c) the score of
//    query row c/4 (+4k) for token 4 tg(c) + J, tg(c) = (c%4) ^ 3*bit2(c).
//    The reduce-scatter needs no lane-dependent selects: each lane holds its
//    query rows and its K row quads in a lane-dependent order (row r ^ c/4,
//    quad u ^ tg(c)), so every level keeps the same slots on both partners.
//    The query rows are loaded in that order; K is loaded in row order, so
//    that every load instruction reads whole token rows, and its quads are
//    put in order by selects in registers (two conditional swaps).
//  * PV: lane (J, c) accumulates its dims over tokens = J mod 4, two tokens
//    per v_dot2c_f32_bf16: each probability is split into a bf16 high part
//    and the bf16-rounded remainder (about 2^-17 relative together; the row
//    sum adds the fp32 values), the parts are packed in pairs (tokens
//    4(2h)+J, 4(2h+1)+J) by the even lane of each lane pair and each pair
//    takes one dot2; one v_perm_b32 pairs the V values of those tokens for
//    one dim.
//    The packed probabilities of row r sit in the same row group at a fixed
//    position, so one DPP row broadcast delivers them.  The four row groups
//    are summed once, at the end.
//
// The online softmax runs in log2 units (scores times scale*log2 e, hardware
// exp2) and rescales the accumulator only when a block raises a row max by
// more than kLazyRescale, so probabilities stay <= 2^8 and the rescale branch
// is wave-uniform and rare.  Tail rows are removed by select (score -inf, V
// zero), so stale or NaN data past the context never reaches the result.
#pragma once

#include "kernels.h"
#include "pa_device.h"

#include <type_traits>

// Wavefronts per workgroup and tiles kept in flight per wavefront.
#ifndef PA_VALU_WAVES
#define PA_VALU_WAVES 4
#endif
#ifndef PA_VALU_NBUF
#define PA_VALU_NBUF 3
#endif
#ifndef PA_VALU_MIN_WAVES
#define PA_VALU_MIN_WAVES 2
#endif

namespace pa {
namespace valu {

constexpr float kLazyRescale = 8.0f;

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

template <int D>
struct KvTile {
  static constexpr int VW = D / 32;   // dwords per lane per token (4: 16 B, 2: 8 B)
  uint32_t k[4][VW];                  // token 4u + J, dims (D/16)*c ..
  uint32_t v[4][VW];                  // token 4u + J, dims (D/16)*c ..
};

// Token quad whose scores lane (J, c) holds after the reduce-scatter.
__device__ __forceinline__ int token_quad(int c) { return (c & 3) ^ (3 * ((c >> 2) & 1)); }

// Row-group position holding the packed probabilities of row r (mod 4) for
// token quads 2h and 2h+1: the even lane of the two that own those quads.
template <int R4, int H>
constexpr int pair_pos() { return 4 * R4 + ((R4 & 1) ? 2 - 2 * H : 2 * H); }

// Dims (D/16)*c .. of one token row per row quad u, through a buffer
// descriptor built from the wave-uniform tile address (scalar registers) and
// the lane's fixed byte offset lane_off[u] into the tile: no per-tile vector
// address math, and the descriptor bounds every access to the tile.
// `bytes` = 0 turns the loads into no-ops that return zeros but still count
// as issued, so every path through the prefetch ring issues the same loads.
// AUX: the loads' cache policy (kLoadDefault or kLoadStreaming).
template <int D, int AUX>
__device__ __forceinline__ void load_rows(uint32_t (&dst)[4][D / 32], const uint16_t* tile,
                                          const uint32_t (&lane_off)[4], int bytes) {
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(tile), 0, bytes, kBufferDescWord3);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int off = (int)lane_off[u];
    if constexpr (D == 128) {
      const auto x = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, AUX);
      dst[u][0] = x[0]; dst[u][1] = x[1]; dst[u][2] = x[2]; dst[u][3] = x[3];
    } else {
      const auto x = __builtin_amdgcn_raw_buffer_load_b64(rsrc, off, 0, AUX);
      dst[u][0] = x[0]; dst[u][1] = x[1];
    }
  }
}

template <int D, int G>
struct WaveState {
  static constexpr int R = G / 4;     // score slots per lane: rows c/4 + 4k
  static constexpr int DPL = D / 16;  // PV dims per lane
  float m[R];                         // running row max, log2 units
  float l[R];                         // this lane's share of the row sum
  float acc[G][DPL];                  // unnormalised output over tokens = J mod 4
};

template <int D, int G, bool TAIL>
__device__ __forceinline__ void process_tile(WaveState<D, G>& S, const KvTile<D>& T,
                                             const uint32_t (&qv)[G][D / 32], int valid,
                                             int grp, int c, float scale_log2) {
  // (slot order of qv and T.k is lane-dependent; see row_reduce_scatter16)
  constexpr int R = G / 4;
  constexpr int VW = D / 32;
  constexpr int DPL = D / 16;

  // K quads in reduce-scatter order: slot u takes row quad u ^ tg(c), by a
  // conditional swap on each bit of tg(c).
  uint32_t kq[4][VW];
  {
    const int t = token_quad(c);
    const bool s1 = (t & 1) != 0, s2 = (t & 2) != 0;
#pragma unroll
    for (int w = 0; w < VW; ++w) {
      const uint32_t a0 = s1 ? T.k[1][w] : T.k[0][w], a1 = s1 ? T.k[0][w] : T.k[1][w];
      const uint32_t a2 = s1 ? T.k[3][w] : T.k[2][w], a3 = s1 ? T.k[2][w] : T.k[3][w];
      kq[0][w] = s2 ? a2 : a0;
      kq[1][w] = s2 ? a3 : a1;
      kq[2][w] = s2 ? a0 : a2;
      kq[3][w] = s2 ? a1 : a3;
    }
  }

  // Partial scores over this lane's dims, ordered so the reduce-scatter hands
  // lane c the values (row c/4 + 4k, token quad c%4) in slot k.
  float y[4 * G];
#pragma unroll
  for (int r = 0; r < G; ++r)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      float a = 0.f;
#pragma unroll
      for (int w = 0; w < VW; ++w) a = dot2_bf16(qv[r][w], kq[u][w], a);
      y[R * (4 * (r % 4) + u) + r / 4] = a;
    }
  row_reduce_scatter16(y);

  const int token = 4 * token_quad(c) + grp;
  float sc[R];
  bool raise = false;
  // The rescale test needs no cross-lane reduction: any lane above its row's
  // max + kLazyRescale triggers it; only then is the block's row max formed.
#pragma unroll
  for (int k = 0; k < R; ++k) {
    float s = y[k] * scale_log2;
    if (TAIL && token >= valid) s = -__builtin_inff();
    sc[k] = s;
    raise |= s > S.m[k] + kLazyRescale;
  }
  if (__builtin_amdgcn_ballot_w64(raise) != 0) {
    float alpha[R];
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const float bm = group_max4(quad_max4(sc[k]));
      const float mn = bm > S.m[k] + kLazyRescale ? bm : S.m[k];
      alpha[k] = mn == -__builtin_inff() ? 1.f : fast_exp2(S.m[k] - mn);
      S.l[k] *= alpha[k];
      S.m[k] = mn;
    }
    static_for<0, G>([&](auto rc) {
      constexpr int r = decltype(rc)::value;
      const float a = row_bcast<4 * (r % 4)>(alpha[r / 4]);
#pragma unroll
      for (int d = 0; d < DPL; ++d) S.acc[r][d] *= a;
    });
  }

  // Probabilities as bf16 pairs: p = hi + lo with hi = bf16(p) and lo =
  // bf16(p - hi) (the difference is exact in fp32), about 2^-17 relative; the
  // row sum adds the fp32 values.  Even lanes then hold the packed high parts
  // (even token quad, odd token quad) of their row, and likewise the low
  // parts: the lane's own quad is even unless bit 2 of c is set.
  const uint32_t pack_sel = ((c >> 2) & 1) ? 0x03020706u : 0x07060302u;
  float pk[R], pkl[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const float mref = S.m[k] == -__builtin_inff() ? 0.f : S.m[k];
    const float pf = fast_exp2(sc[k] - mref);
    const uint32_t pb = bf16_rne(pf) << 16;
    const uint32_t lb = bf16_rne(pf - __uint_as_float(pb)) << 16;
    S.l[k] += pf;
    const uint32_t nb = __float_as_uint(dpp<kDppQuadXor1>(__uint_as_float(pb)));
    const uint32_t nl = __float_as_uint(dpp<kDppQuadXor1>(__uint_as_float(lb)));
    pk[k] = __uint_as_float(__builtin_amdgcn_perm(nb, pb, pack_sel));
    pkl[k] = __uint_as_float(__builtin_amdgcn_perm(nl, lb, pack_sel));
  }

  // PV: step h covers tokens 4(2h)+J and 4(2h+1)+J; row r's packed pair is at
  // position pair_pos<r % 4, h> of slot r/4 in the same row group.
  static_for<0, 2>([&](auto hc) {
    constexpr int h = decltype(hc)::value;
    uint32_t vp[DPL];  // (token 2h, token 2h+1) bf16 pairs, one per dim
#pragma unroll
    for (int w = 0; w < VW; ++w) {
      uint32_t a = T.v[2 * h][w], b = T.v[2 * h + 1][w];
      if (TAIL && 4 * (2 * h) + grp >= valid) a = 0u;
      if (TAIL && 4 * (2 * h + 1) + grp >= valid) b = 0u;
      vp[2 * w] = __builtin_amdgcn_perm(b, a, 0x05040100u);      // dim 2w of both tokens
      vp[2 * w + 1] = __builtin_amdgcn_perm(b, a, 0x07060302u);  // dim 2w+1
    }
    static_for<0, G>([&](auto rc) {
      constexpr int r = decltype(rc)::value;
      const uint32_t pp = __float_as_uint(row_bcast<pair_pos<r % 4, h>()>(pk[r / 4]));
      const uint32_t pl = __float_as_uint(row_bcast<pair_pos<r % 4, h>()>(pkl[r / 4]));
#pragma unroll
      for (int d = 0; d < DPL; ++d) S.acc[r][d] = dot2_bf16(pl, vp[d], dot2_bf16(pp, vp[d], S.acc[r][d]));
    });
  });
}

// LDS bytes the body needs for the end-of-item merge.
template <int D, int G, int W>
constexpr int valu_lds_bytes() { return (2 * W * G + W * 4 * G * D) * 4; }

// One work item (partition, sequence, KV head) = workgroup `wg_index`;
// `smem` points at valu_lds_bytes<D, G, W>() bytes of LDS.  STREAM: load the
// tiles as streaming data (kLoadStreaming); it changes caching, never the
// results.  APPEND: the fused KV append (DecodeParams::k_new): the item that
// holds token ctx - 1 takes its K and V rows from k_new / v_new in registers
// (whatever the pool slot holds) and stores them into the slot.
template <int D, int G, int W, int NBUF, bool TRACE, bool STREAM, bool APPEND = false>
__device__ __forceinline__ void decode_valu_body(const DecodeParams& p, int wg_index, lds_u8_t* smem) {
  constexpr int R = G / 4;
  constexpr int DPL = D / 16;
  static_assert(G == 4 || G == 8, "group size");
  static_assert(D == 64 || D == 128, "head dim");

  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int grp = lane >> 4;
  const int tok = lane & 15;

  int g, b, part;
  decode_item(p, wg_index, g, b, part);

  const int start = p.token_offset + part * p.part_tokens;
  const int j0 = start >> 4;
  const int h0 = g * G;
  const int32_t* bt = p.block_tables + (size_t)b * p.bt_stride + j0;
  // The first 64 block ids and the query rows are loaded before the context
  // length arrives (j0 < bt_stride for every launched partition).
  const int raw_first = lane < min(64, p.bt_stride - j0) ? bt[lane] : 0;

  // Query slices: lane (J, c) keeps dims (D/16)*c .. of every query row, row
  // r in slot r ^ c/4 (mod 4), the order the reduce-scatter needs.
  uint32_t qv[G][D / 32];
  {
    const uint16_t* qb = p.q + ((size_t)b * p.num_q_heads + h0) * D + (D / 16) * tok;
#pragma unroll
    for (int r = 0; r < G; ++r) {
      const int qr = (r & ~3) | ((r & 3) ^ (tok >> 2));
      if constexpr (D == 128) {
        const uint4 v = *reinterpret_cast<const uint4*>(qb + qr * D);
        qv[r][0] = v.x; qv[r][1] = v.y; qv[r][2] = v.z; qv[r][3] = v.w;
      } else {
        const uint2 v = *reinterpret_cast<const uint2*>(qb + qr * D);
        qv[r][0] = v.x; qv[r][1] = v.y;
      }
    }
  }

  int n = p.context_lens[b];
  n = n < 0 ? 0 : (n > p.max_ctx ? p.max_ctx : n);
  const bool split = p.write_partials != 0;
  if (split && start >= n) return;  // whole workgroup; the reduce skips this partition
  const int end = min(n, start + p.part_tokens);
  const int nblk = end > start ? (end - start + 15) >> 4 : 0;

  // Fused append: block jnew of this item (-1: none) holds the new token in
  // row rnew; knew / vnew are the lane's slice of its K and V rows (dims
  // (D/16)*tok ..).  The lanes of row group rnew % 4 store the rows.
  constexpr int VW = D / 32;
  int jnew = -1, rnew = 0;
  uint32_t knew[VW], vnew[VW];
  if constexpr (APPEND) {
    if (n > 0 && n - 1 >= start && n - 1 < end) {
      jnew = ((n - 1) >> 4) - j0;
      rnew = (n - 1) & 15;
      const size_t src = ((size_t)b * p.num_kv_heads + g) * D + (D / 16) * tok;
#pragma unroll
      for (int w = 0; w < VW; ++w) {
        knew[w] = reinterpret_cast<const uint32_t*>(p.k_new + src)[w];
        vnew[w] = reinterpret_cast<const uint32_t*>(p.v_new + src)[w];
      }
      if (wave == 0 && grp == (rnew & 3)) {
        int phys = p.block_tables[(size_t)b * p.bt_stride + ((n - 1) >> 4)];
        phys = min(max(phys, 0), p.num_blocks - 1);
        const size_t dst = (((size_t)phys * p.num_kv_heads + g) * 16 + rnew) * D + (D / 16) * tok;
#pragma unroll
        for (int w = 0; w < VW; ++w) {
          reinterpret_cast<uint32_t*>(p.k_pool_w + dst)[w] = knew[w];
          reinterpret_cast<uint32_t*>(p.v_pool_w + dst)[w] = vnew[w];
        }
      }
    }
  }

  WaveState<D, G> S;
#pragma unroll
  for (int k = 0; k < R; ++k) { S.m[k] = -__builtin_inff(); S.l[k] = 0.f; }
#pragma unroll
  for (int r = 0; r < G; ++r)
#pragma unroll
    for (int d = 0; d < DPL; ++d) S.acc[r][d] = 0.f;

  constexpr size_t kTileElems = 16 * D;
  const size_t blk_stride = (size_t)p.num_kv_heads * kTileElems;
  const uint16_t* kbase = p.k_pool + (size_t)g * kTileElems;
  const uint16_t* vbase = p.v_pool + (size_t)g * kTileElems;
  const size_t item = ((size_t)part * p.batch + b) * p.num_kv_heads + g;
  // Byte offsets of the lane's slice in row quad u (K and V alike).
  uint32_t roff[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) roff[u] = (uint32_t)((4 * u + grp) * D + (D / 16) * tok) * 2u;

  for (int c0 = 0; c0 < nblk; c0 += 64) {
    const int cn = min(64, nblk - c0);
    const int raw = c0 == 0 ? (lane < cn ? raw_first : 0) : (lane < cn ? bt[c0 + lane] : 0);
    const int idc = min(max(raw, 0), p.num_blocks - 1);

    // Loads for blocks past the chunk are issued with an empty descriptor.
    auto load = [&](KvTile<D>& T, int i) {
      const bool ok = i < cn;
      const size_t id = (size_t)__builtin_amdgcn_readlane(idc, ok ? i : 0);
      const int bytes = ok ? 16 * D * 2 : 0;
      constexpr int kAux = STREAM ? kLoadStreaming : kLoadDefault;
      load_rows<D, kAux>(T.k, kbase + id * blk_stride, roff, bytes);
      load_rows<D, kAux>(T.v, vbase + id * blk_stride, roff, bytes);
    };
    auto run = [&](KvTile<D>& T, int i) {
      const int valid = min(16, end - (start + (c0 + i) * 16));
      if constexpr (APPEND) {
        // the new token's rows replace whatever the slot held (the ring slot
        // is loaded again before its next use)
        if (c0 + i == jnew) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (4 * u + grp == rnew) {
#pragma unroll
              for (int w = 0; w < VW; ++w) { T.k[u][w] = knew[w]; T.v[u][w] = vnew[w]; }
            }
        }
      }
      if (valid == 16)
        process_tile<D, G, false>(S, T, qv, 16, grp, tok, p.scale_log2);
      else
        process_tile<D, G, true>(S, T, qv, valid, grp, tok, p.scale_log2);
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
    KvTile<D> T[NBUF];
    int ld = i;
#pragma unroll
    for (int s = 0; s < NBUF - 1; ++s) {
      load(T[s], ld);
      ld += W;
    }
    bool done = false;
    while (!done) {
#pragma unroll
      for (int s = 0; s < NBUF; ++s) {
        if (!done) {
          load(T[(s + NBUF - 1) % NBUF], ld);
          ld += W;
          run(T[s], i);
          i += W;
          done = i >= cn;
        }
      }
    }
  }

  // Row statistics of this wave: slot k of lane (J, c) belongs to row
  // c/4 + 4k; every lane gathers all rows by row broadcast.
  float Mw[G], Lw[G];
  {
    float lsum[R];
#pragma unroll
    for (int k = 0; k < R; ++k) lsum[k] = group_sum4(quad_sum4(S.l[k]));
    static_for<0, G>([&](auto rc) {
      constexpr int r = decltype(rc)::value;
      Mw[r] = row_bcast<4 * (r % 4)>(S.m[r / 4]);
      Lw[r] = row_bcast<4 * (r % 4)>(lsum[r / 4]);
    });
  }

  // Merge waves and row groups through LDS; lane l then owns output dims
  // (D/64)*l .. of every row.
  constexpr int OPL = D / 64;
  lds_f32_t (*sm)[G] = reinterpret_cast<lds_f32_t (*)[G]>(smem);
  lds_f32_t (*sl)[G] = sm + W;
  lds_f32_t (*sacc)[4][G][D] = reinterpret_cast<lds_f32_t (*)[4][G][D]>(smem + 2 * W * G * 4);
  if (lane == 0) {
#pragma unroll
    for (int r = 0; r < G; ++r) { sm[wave][r] = Mw[r]; sl[wave][r] = Lw[r]; }
  }
#pragma unroll
  for (int r = 0; r < G; ++r)
#pragma unroll
    for (int d = 0; d < DPL; ++d) sacc[wave][grp][r][DPL * tok + d] = S.acc[r][d];
  __syncthreads();
  if (wave != 0) return;

#pragma unroll
  for (int r = 0; r < G; ++r) {
    float mx = sm[0][r];
#pragma unroll
    for (int w = 1; w < W; ++w) mx = fmaxf(mx, sm[w][r]);
    const float mref = (mx == -__builtin_inff()) ? 0.f : mx;
    float lt = 0.f, o[OPL];
#pragma unroll
    for (int d = 0; d < OPL; ++d) o[d] = 0.f;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const float f = fast_exp2(sm[w][r] - mref);
      lt = fmaf(sl[w][r], f, lt);
#pragma unroll
      for (int d = 0; d < OPL; ++d) {
        const float part_sum = (sacc[w][0][r][OPL * lane + d] + sacc[w][1][r][OPL * lane + d]) +
                               (sacc[w][2][r][OPL * lane + d] + sacc[w][3][r][OPL * lane + d]);
        o[d] = fmaf(part_sum, f, o[d]);
      }
    }
    const float inv = lt > 0.f ? 1.0f / lt : 0.f;
    if (!split) {
      uint16_t* orow = p.out + ((size_t)b * p.num_q_heads + h0 + r) * D;
      if constexpr (OPL == 2)
        *reinterpret_cast<uint32_t*>(orow + 2 * lane) =
            bf16_rne(o[0] * inv) | (bf16_rne(o[1] * inv) << 16);
      else
        orow[lane] = (uint16_t)bf16_rne(o[0] * inv);
    } else {
      const size_t row = ((size_t)b * p.num_q_heads + h0 + r) * p.part_stride + p.part_offset + part;
      float* po = p.part_o + row * D;
      if constexpr (OPL == 2)
        store_partial2(po + 2 * lane, o[0] * inv, o[1] * inv);
      else
        store_partial(po + lane, o[0] * inv);
      if (lane == 0)
        p.part_lse[row] = lt > 0.f ? (mx + log2f(lt)) * kLn2 : -__builtin_inff();
    }
  }
}

}  // namespace valu
}  // namespace pa
