// Split-KV paged decode attention on VALU dot products (gfx950).
//
// One workgroup handles one work item (partition p, sequence b, KV head g):
// the G query heads g*G .. g*G+G-1 that share KV head g attend to the
// tokens [p*S, min((p+1)*S, ctx_b)) of sequence b.  Its W wavefronts take
// the partition's 16-token KV blocks round-robin, each keeping its own
// online-softmax state, and merge through LDS at the end.
//
// Per block a wavefront loads one K tile and one V tile (16 tokens x D
// bf16, contiguous in the pool) and uses two lane layouts:
//
//  * QK^T in "token lanes": lane (j, t) = (lane >> 4, lane & 15) holds token
//    t's K chunks 4i+j (16 bytes each), so each load instruction reads a
//    64-byte segment of every token row.  Partial dot products over those
//    dims (v_dot2c_f32_bf16) are reduce-scattered over the four row groups
//    with two permlane swaps, leaving score s[row j][token t] in lane (j, t).
//  * PV in "dim lanes": lane l holds dims (D/64)*l .. of all 16 tokens, so
//    every V load instruction reads one whole 256-byte token row and the
//    accumulator acc[row][dims of l] never needs a cross-lane reduction.
//    The probabilities reach the dim lanes through a permlane all-gather and
//    a DPP row broadcast per token.
//
// The online softmax runs in log2 units (scores pre-multiplied by
// scale*log2 e, hardware exp2); masked tail rows are removed by select, and
// their V values are replaced by zero, so stale or NaN data past the context
// never reaches the result.
#include "kernels.h"
#include "pa_device.h"

#include <type_traits>

namespace pa {
namespace {

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

template <int D>
struct KvTile {
  static constexpr int KC = D / 32;  // 16-byte K chunks per lane
  uint4 k[KC];
  uint32_t v[16];  // D=128: dims (2l, 2l+1) of token t; D=64: dim l in the low half
};

template <int D>
__device__ __forceinline__ void load_tile(KvTile<D>& T, const uint16_t* __restrict__ kt,
                                          const uint16_t* __restrict__ vt, int grp, int tok,
                                          int lane) {
#pragma unroll
  for (int i = 0; i < KvTile<D>::KC; ++i)
    T.k[i] = *reinterpret_cast<const uint4*>(kt + tok * D + (4 * i + grp) * 8);
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    if constexpr (D == 128)
      T.v[t] = *reinterpret_cast<const uint32_t*>(vt + t * D + 2 * lane);
    else
      T.v[t] = vt[t * D + lane];
  }
}

template <int D, int G>
struct WaveState {
  static constexpr int R = G / 4;    // query rows owned per lane (row j + 4k)
  static constexpr int DPL = D / 64; // output dims per lane
  float m[R];                        // running row max, log2 units (row-uniform)
  float l[R];                        // this lane's token column share of the row sum
  float acc[G][DPL];                 // unnormalised output, dims DPL*lane ..
};

__device__ __forceinline__ uint32_t chunk_word(const uint4& c, int w) {
  return w == 0 ? c.x : (w == 1 ? c.y : (w == 2 ? c.z : c.w));
}

template <int D, int G, bool TAIL>
__device__ __forceinline__ void process_tile(WaveState<D, G>& S, const KvTile<D>& T,
                                             const uint32_t (&qv)[G][D / 32][4], int valid,
                                             int tok, float scale_log2) {
  constexpr int R = G / 4;
  constexpr int KC = D / 32;
  constexpr int DPL = D / 64;

  // QK^T partials over this lane's dims, then reduce-scatter over row groups.
  float x[G];
#pragma unroll
  for (int r = 0; r < G; ++r) {
    float a = 0.f;
#pragma unroll
    for (int i = 0; i < KC; ++i)
#pragma unroll
      for (int w = 0; w < 4; ++w) a = dot2_bf16(qv[r][i][w], chunk_word(T.k[i], w), a);
    x[r] = a;
  }

  float A[G], P[G];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    float s = reduce_scatter4(x[4 * k], x[4 * k + 1], x[4 * k + 2], x[4 * k + 3]) * scale_log2;
    if (TAIL && tok >= valid) s = -__builtin_inff();
    const float mn = fmaxf(S.m[k], row_max16(s));
    const float mref = (mn == -__builtin_inff()) ? 0.f : mn;
    const float alpha = fast_exp2(S.m[k] - mref);
    const float pk = fast_exp2(s - mref);
    S.l[k] = fmaf(S.l[k], alpha, pk);
    S.m[k] = mn;
    allgather4(alpha, A[4 * k], A[4 * k + 1], A[4 * k + 2], A[4 * k + 3]);
    allgather4(pk, P[4 * k], P[4 * k + 1], P[4 * k + 2], P[4 * k + 3]);
  }
#pragma unroll
  for (int r = 0; r < G; ++r)
#pragma unroll
    for (int d = 0; d < DPL; ++d) S.acc[r][d] *= A[r];

  // PV: token t's probabilities broadcast from row position t.
  static_for<0, 16>([&](auto tc) {
    constexpr int t = decltype(tc)::value;
    float v0 = bf16_lo(T.v[t]);
    float v1 = (DPL == 2) ? bf16_hi(T.v[t]) : 0.f;
    if (TAIL && t >= valid) { v0 = 0.f; v1 = 0.f; }
#pragma unroll
    for (int r = 0; r < G; ++r) {
      const float pb = row_bcast<t>(P[r]);
      S.acc[r][0] = fmaf(pb, v0, S.acc[r][0]);
      if constexpr (DPL == 2) S.acc[r][1] = fmaf(pb, v1, S.acc[r][1]);
    }
  });
}

template <int D, int G, int W, bool TRACE>
__global__ void __launch_bounds__(64 * W) decode_valu_kernel(const DecodeParams p) {
  constexpr int R = G / 4;
  constexpr int KC = D / 32;
  constexpr int DPL = D / 64;
  static_assert(G == 4 || G == 8, "group size");
  static_assert(D == 64 || D == 128, "head dim");

  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int grp = lane >> 4;
  const int tok = lane & 15;

  // Work item; the KV head varies fastest so consecutive workgroups, which
  // the dispatcher spreads over the XCDs round-robin, keep one KV head per XCD.
  int wg = blockIdx.x;
  const int g = wg % p.num_kv_heads;
  wg /= p.num_kv_heads;
  const int b = wg % p.batch;
  const int part = wg / p.batch;

  int n = p.context_lens[b];
  n = n < 0 ? 0 : (n > p.max_ctx ? p.max_ctx : n);
  const int start = part * p.part_tokens;
  const bool split = p.num_parts > 1;
  if (split && start >= n) return;  // whole workgroup; the reduce skips this partition
  const int end = min(n, start + p.part_tokens);
  const int nblk = end > start ? (end - start + 15) >> 4 : 0;
  const int j0 = start >> 4;
  const int h0 = g * G;

  uint32_t qv[G][KC][4];
  {
    const uint16_t* qb = p.q + ((size_t)b * p.num_q_heads + h0) * D;
#pragma unroll
    for (int r = 0; r < G; ++r)
#pragma unroll
      for (int i = 0; i < KC; ++i) {
        const uint4 v = *reinterpret_cast<const uint4*>(qb + r * D + (4 * i + grp) * 8);
        qv[r][i][0] = v.x; qv[r][i][1] = v.y; qv[r][i][2] = v.z; qv[r][i][3] = v.w;
      }
  }

  WaveState<D, G> S;
#pragma unroll
  for (int k = 0; k < R; ++k) { S.m[k] = -__builtin_inff(); S.l[k] = 0.f; }
#pragma unroll
  for (int r = 0; r < G; ++r)
#pragma unroll
    for (int d = 0; d < DPL; ++d) S.acc[r][d] = 0.f;

  const int32_t* bt = p.block_tables + (size_t)b * p.bt_stride + j0;
  constexpr size_t kTileElems = 16 * D;
  const size_t blk_stride = (size_t)p.num_kv_heads * kTileElems;
  const uint16_t* kbase = p.k_pool + (size_t)g * kTileElems;
  const uint16_t* vbase = p.v_pool + (size_t)g * kTileElems;
  const size_t item = ((size_t)part * p.batch + b) * p.num_kv_heads + g;

  for (int c0 = 0; c0 < nblk; c0 += 64) {
    const int cn = min(64, nblk - c0);
    const int raw = lane < cn ? bt[c0 + lane] : 0;
    const int idc = min(max(raw, 0), p.num_blocks - 1);

    auto tile_of = [&](int i, const uint16_t*& kt, const uint16_t*& vt) {
      const size_t id = (size_t)__builtin_amdgcn_readlane(idc, i);
      kt = kbase + id * blk_stride;
      vt = vbase + id * blk_stride;
    };
    auto run = [&](const KvTile<D>& T, int i) {
      const int valid = min(16, end - (start + (c0 + i) * 16));
      if (valid == 16)
        process_tile<D, G, false>(S, T, qv, 16, tok, p.scale_log2);
      else
        process_tile<D, G, true>(S, T, qv, valid, tok, p.scale_log2);
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
    KvTile<D> TA, TB;
    const uint16_t *kt, *vt;
    tile_of(i, kt, vt);
    load_tile<D>(TA, kt, vt, grp, tok, lane);
    while (true) {
      int nx = i + W;
      if (nx < cn) { tile_of(nx, kt, vt); load_tile<D>(TB, kt, vt, grp, tok, lane); }
      run(TA, i);
      if (nx >= cn) break;
      i = nx;
      nx = i + W;
      if (nx < cn) { tile_of(nx, kt, vt); load_tile<D>(TA, kt, vt, grp, tok, lane); }
      run(TB, i);
      if (nx >= cn) break;
      i = nx;
    }
  }

  // Row statistics of this wave for every row r, in every lane.
  float Mw[G], Lw[G];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const float lsum = row_sum16(S.l[k]);
    allgather4(S.m[k], Mw[4 * k], Mw[4 * k + 1], Mw[4 * k + 2], Mw[4 * k + 3]);
    allgather4(lsum, Lw[4 * k], Lw[4 * k + 1], Lw[4 * k + 2], Lw[4 * k + 3]);
  }

  float M[G], L[G], O[G][DPL];
  if constexpr (W == 1) {
#pragma unroll
    for (int r = 0; r < G; ++r) {
      M[r] = Mw[r]; L[r] = Lw[r];
#pragma unroll
      for (int d = 0; d < DPL; ++d) O[r][d] = S.acc[r][d];
    }
  } else {
    __shared__ float sm[W][G], sl[W][G];
    __shared__ float sacc[W][G][D];
    if (lane == 0) {
#pragma unroll
      for (int r = 0; r < G; ++r) { sm[wave][r] = Mw[r]; sl[wave][r] = Lw[r]; }
    }
#pragma unroll
    for (int r = 0; r < G; ++r)
#pragma unroll
      for (int d = 0; d < DPL; ++d) sacc[wave][r][DPL * lane + d] = S.acc[r][d];
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int r = 0; r < G; ++r) {
      float mx = sm[0][r];
#pragma unroll
      for (int w = 1; w < W; ++w) mx = fmaxf(mx, sm[w][r]);
      const float mref = (mx == -__builtin_inff()) ? 0.f : mx;
      float lt = 0.f, o[DPL];
#pragma unroll
      for (int d = 0; d < DPL; ++d) o[d] = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        const float f = fast_exp2(sm[w][r] - mref);
        lt = fmaf(sl[w][r], f, lt);
#pragma unroll
        for (int d = 0; d < DPL; ++d) o[d] = fmaf(sacc[w][r][DPL * lane + d], f, o[d]);
      }
      M[r] = mx; L[r] = lt;
#pragma unroll
      for (int d = 0; d < DPL; ++d) O[r][d] = o[d];
    }
  }

#pragma unroll
  for (int r = 0; r < G; ++r) {
    const float inv = L[r] > 0.f ? 1.0f / L[r] : 0.f;
    if (!split) {
      uint16_t* orow = p.out + ((size_t)b * p.num_q_heads + h0 + r) * D;
      if constexpr (DPL == 2)
        *reinterpret_cast<uint32_t*>(orow + 2 * lane) =
            bf16_rne(O[r][0] * inv) | (bf16_rne(O[r][1] * inv) << 16);
      else
        orow[lane] = (uint16_t)bf16_rne(O[r][0] * inv);
    } else {
      const size_t row = ((size_t)b * p.num_q_heads + h0 + r) * p.num_parts + part;
      float* po = p.part_o + row * D;
      if constexpr (DPL == 2)
        *reinterpret_cast<float2*>(po + 2 * lane) = make_float2(O[r][0] * inv, O[r][1] * inv);
      else
        po[lane] = O[r][0] * inv;
      if (lane == 0)
        p.part_lse[row] = L[r] > 0.f ? (M[r] + log2f(L[r])) * kLn2 : -__builtin_inff();
    }
  }
}

constexpr int kWaves = 4;

template <int D, int G, bool TRACE>
hipError_t launch_t(const DecodeParams& p, hipStream_t stream) {
  const int64_t grid = (int64_t)p.num_parts * p.batch * p.num_kv_heads;
  hipLaunchKernelGGL((decode_valu_kernel<D, G, kWaves, TRACE>), dim3((unsigned)grid),
                     dim3(64 * kWaves), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_valu(const DecodeParams& p, int head_dim, int group, bool trace,
                              hipStream_t stream) {
  if (head_dim == 128 && group == 4)
    return trace ? launch_t<128, 4, true>(p, stream) : launch_t<128, 4, false>(p, stream);
  if (head_dim == 64 && group == 4)
    return trace ? launch_t<64, 4, true>(p, stream) : launch_t<64, 4, false>(p, stream);
  if (head_dim == 128 && group == 8)
    return trace ? launch_t<128, 8, true>(p, stream) : launch_t<128, 8, false>(p, stream);
  if (head_dim == 64 && group == 8)
    return trace ? launch_t<64, 8, true>(p, stream) : launch_t<64, 8, false>(p, stream);
  return hipErrorInvalidValue;
}

}  // namespace pa
