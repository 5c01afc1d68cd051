"""A decode input on which rounding the softmax weights to bf16 before the
PV product fails the parity gate (shared by the CPU pin and the GPU test).

Every 16-token block holds two tokens of score 0 (the maximum, V = 0), seven
"A" tokens whose weight 2^(s - max) is 0.5 + 0.75 * 2^-8 (V = +1 in every
dimension) and seven "B" tokens whose weight is just above 0.5 (V = -1).  In
[0.5, 1) bf16 values are 2^-8 apart, so A weights round up to 0.5 + 2^-8 and
B weights down to 0.5: the rounding errors are correlated with the sign of V.
The exact output is 7 (p_A - p_B) / (2 + 7 (p_A + p_B)) in every dimension;
with bf16 weights it comes out 1.45 times as large.  All weights are near
0.5 -- many near-equal scores -- over contexts up to 32k tokens.

Only dimension 0 of q and K is non-zero (q = e0), so every score is the exact
product scale * K[t][0]; the scale puts the A tokens (K = -8) at
log2(p_A) = log2(0.5 + 0.75 * 2^-8) and the B tokens (K = -8.0625) at a
weight inside (0.5, 0.5 + 2^-9).
"""
from __future__ import annotations

import math

import numpy as np

from workloads import LogicalCase, f32_to_bf16_bits, page_case

BF16_ULP_HALF = 2.0 ** -8                     # bf16 spacing in [0.5, 1)
P_A = 0.5 + 0.75 * BF16_ULP_HALF
K_A, K_B = -8.0, -8.0625                      # exact bf16 values
SCALE = math.log2(P_A) / (K_A * math.log2(math.e))
P_B = 2.0 ** (K_B * SCALE * math.log2(math.e))
ROLE = np.array([0] + [1, 2] * 7 + [0])        # per row of a block: 0 max, 1 A, 2 B


def exact_output(n: int) -> float:
    """The exact attention output (every dimension) over n tokens."""
    roles = ROLE[np.arange(n) % 16]
    w = np.where(roles == 0, 1.0, np.where(roles == 1, P_A, P_B))
    v = np.where(roles == 0, 0.0, np.where(roles == 1, 1.0, -1.0))
    return float((w * v).sum() / w.sum())


def near_tie_case(ctx_lens, hq: int, hkv: int, d: int = 128, seed: int = 0, prefix_len: int = 0):
    """The paged workload (shared prefix blocks when prefix_len > 0)."""
    ctx_lens = [int(n) for n in ctx_lens]
    B = len(ctx_lens)
    q = np.zeros((B, hq, d), np.float32)
    q[:, :, 0] = 1.0
    ks, vs = [], []
    for n in ctx_lens:
        roles = ROLE[np.arange(n) % 16]
        k = np.zeros((hkv, n, d), np.float32)
        k[:, :, 0] = np.where(roles == 0, 0.0, np.where(roles == 1, K_A, K_B))
        v = np.repeat(np.where(roles == 0, 0.0, np.where(roles == 1, 1.0, -1.0)
                               ).astype(np.float32)[None, :, None], hkv, 0).repeat(d, 2)
        ks.append(f32_to_bf16_bits(k))
        vs.append(f32_to_bf16_bits(v))
    case = LogicalCase(q=f32_to_bf16_bits(q), k=ks, v=vs, scale=SCALE, num_kv_heads=hkv,
                       prefix_len=prefix_len)
    return page_case(case, seed, share_prefix=prefix_len > 0, name="near_tie")
