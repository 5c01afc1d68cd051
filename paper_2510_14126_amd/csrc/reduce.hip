// Cross-split reduce: merge split-KV partials into the bf16 output.
//
// For sequence b and query head h the decode kernels left, per partition p,
// the partition-normalised output o_p and its log-sum-exp lse_p (natural
// log): first the partitions of a prefix shared by the whole batch (if any),
// then ceil((ctx_b - prefix) / S) partitions of the rest.  With M = max lse_p:
//     w_p = exp(lse_p - M),   out = sum_p w_p o_p / sum_p w_p,
// which is exactly softmax attention over the whole context (zeros when
// every w_p is 0).  One wavefront per (b, h).  Lane q loads lse_q (64
// partitions per round) together with the o rows of the first kGroup
// partitions, so up to kGroup partitions cost one memory round trip; lane l
// owns output dims (D/64)*l .. and adds the partitions in order p = 0, 1, ..
// (weights broadcast from the lane that computed them), so the result is
// deterministic and P_b = 1 reproduces o_0 bit for bit.
#include "kernels.h"
#include "pa_device.h"

namespace pa {
namespace {

constexpr int kGroup = 8;   // partitions whose o rows are loaded together

template <int D>
__global__ void __launch_bounds__(64) reduce_kernel(const ReduceParams p) {
  constexpr int DPL = D / 64;
  const int lane = threadIdx.x;
  const int bh = blockIdx.x;
  const int b = bh / p.num_q_heads;
  int n = p.context_lens[b] - p.prefix_len;
  n = n < 0 ? 0 : n;
  int pb = p.prefix_parts + n / p.part_tokens + (n % p.part_tokens != 0);
  pb = pb > p.part_stride ? p.part_stride : pb;
  const float* lse = p.part_lse + (size_t)bh * p.part_stride;
  const float* po = p.part_o + (size_t)bh * p.part_stride * D + DPL * lane;

  // o rows of partitions first .. first+kGroup-1 (clamped into the row's
  // slots; entries past pb are never used)
  float v[kGroup][DPL];
  auto load_group = [&](int first) {
    const int lastq = pb > 0 ? pb - 1 : 0;
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      const int q = min(first + k, lastq);
#pragma unroll
      for (int d = 0; d < DPL; ++d) v[k][d] = po[(size_t)q * D + d];
    }
  };
  const float l0 = lane < pb ? lse[lane] : -__builtin_inff();
  load_group(0);

  float mx = l0;
  for (int c0 = 64; c0 < pb; c0 += 64)
    mx = fmaxf(mx, c0 + lane < pb ? lse[c0 + lane] : -__builtin_inff());
  mx = group_max4(row_max16(mx));
  const float mref = (mx == -__builtin_inff()) ? 0.f : mx;

  float wsum = 0.f, o[DPL];
#pragma unroll
  for (int d = 0; d < DPL; ++d) o[d] = 0.f;
  for (int c0 = 0; c0 < pb; c0 += 64) {
    const float x = c0 == 0 ? l0 : (c0 + lane < pb ? lse[c0 + lane] : 0.f);
    const int wl = __float_as_int(fast_exp2((x - mref) * kLog2e));   // w of partition c0 + lane
    const int cnt = min(64, pb - c0);
    for (int j0 = 0; j0 < cnt; j0 += kGroup) {
      if (c0 + j0 > 0) load_group(c0 + j0);
#pragma unroll
      for (int k = 0; k < kGroup; ++k) {
        if (j0 + k < cnt) {
          const float w = __int_as_float(__builtin_amdgcn_readlane(wl, j0 + k));
          wsum += w;
#pragma unroll
          for (int d = 0; d < DPL; ++d) o[d] = fmaf(w, v[k][d], o[d]);
        }
      }
    }
  }
  const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
  uint16_t* orow = p.out + (size_t)bh * D;
  if constexpr (DPL == 2)
    *reinterpret_cast<uint32_t*>(orow + 2 * lane) = bf16_rne(o[0] * inv) | (bf16_rne(o[1] * inv) << 16);
  else
    orow[lane] = (uint16_t)bf16_rne(o[0] * inv);
}

}  // namespace

hipError_t launch_reduce(const ReduceParams& p, int head_dim, hipStream_t stream) {
  const int64_t grid = (int64_t)p.batch * p.num_q_heads;
  if (head_dim == 128)
    hipLaunchKernelGGL(reduce_kernel<128>, dim3((unsigned)grid), dim3(64), 0, stream, p);
  else if (head_dim == 64)
    hipLaunchKernelGGL(reduce_kernel<64>, dim3((unsigned)grid), dim3(64), 0, stream, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa
