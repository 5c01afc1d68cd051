"""Write hand_cases.json: small worked examples whose answers are closed forms.

The paper prints no worked example, table or formula for the attention step,
so every expected value here is derived by hand from the definition of scaled
dot-product softmax attention and evaluated with the ``math`` module only (no
oracle and no GPU code is involved).  Inputs are chosen exactly representable
in bf16.  Run: ``python tests/golden/make_hand_cases.py``.
"""
import json
import math
import os
import struct


def bf16_bits(x: float) -> int:
    """Bits of a value that is exactly representable in bf16."""
    b = struct.unpack("<I", struct.pack("<f", x))[0]
    assert b & 0xFFFF == 0, f"{x} is not exact in bf16"
    return b >> 16


cases = []

# 1. Two tokens: w0 = 1 / (1 + e^(s1 - s0)), out = w0 V0 + (1 - w0) V1,
#    lse = s0 + ln(1 + e^(s1 - s0)).
q = [1.0, 2.0, 0.0, -1.0]
K = [[0.5, 0.25, 1.0, 0.0], [1.0, -1.0, 0.0, 2.0]]
V = [[1.0, 0.0, -2.0, 3.0], [0.0, 4.0, 1.0, -1.0]]
scale = 0.5
s0 = scale * (0.5 + 0.5 + 0.0 + 0.0)      # 0.5
s1 = scale * (1.0 - 2.0 + 0.0 - 2.0)      # -1.5
w0 = 1.0 / (1.0 + math.exp(s1 - s0))
cases.append(dict(
    name="two_tokens", derivation="s0=0.5, s1=-1.5; w0=1/(1+e^-2); out=w0*V0+(1-w0)*V1",
    q=[q], K=K, V=V, scale=scale,
    out=[[w0 * V[0][i] + (1 - w0) * V[1][i] for i in range(4)]],
    lse=[s0 + math.log1p(math.exp(s1 - s0))]))

# 2. Zero query: every weight is 1/n and out is the arithmetic mean of V.
V = [[1.0, -3.0], [2.0, 5.0], [4.0, 0.5], [-8.0, 1.0], [16.0, 2.0]]
cases.append(dict(
    name="zero_query_mean", derivation="q=0 -> w_t=1/5; out = column means; lse = ln 5",
    q=[[0.0, 0.0]], K=[[3.0, 1.0], [-2.0, 7.0], [0.25, 0.5], [9.0, -1.0], [1.0, 1.0]], V=V,
    scale=1.0, out=[[sum(r[0] for r in V) / 5, sum(r[1] for r in V) / 5]], lse=[math.log(5.0)]))

# 3. One token: out = V0 exactly, lse = s0.
cases.append(dict(
    name="single_token", derivation="n=1 -> w0=1; out=V0; lse=s0=scale*<q,K0>",
    q=[[0.5, -1.0, 2.0]], K=[[2.0, 1.0, 0.25]], V=[[-0.375, 3.5, 1024.0]], scale=0.25,
    out=[[-0.375, 3.5, 1024.0]], lse=[0.25 * (1.0 - 1.0 + 0.5)]))

# 4. Round-to-nearest-even ties on the bf16 output (q = 0, two tokens, so the
#    exact result is the midpoint of two adjacent bf16 values in [128, 256),
#    where bf16 spacing is 1).  RNE keeps the even mantissa.
for a, b, rne in [(128.0, 129.0, 128.0), (129.0, 130.0, 130.0), (-129.0, -130.0, -130.0)]:
    cases.append(dict(
        name=f"rne_tie_{a:g}_{b:g}", derivation=f"out=({a:g}+{b:g})/2 exactly; RNE -> {rne:g}",
        q=[[0.0, 0.0]], K=[[1.0, 2.0], [3.0, -4.0]], V=[[a, a], [b, b]], scale=1.0,
        out=[[(a + b) / 2, (a + b) / 2]], lse=[math.log(2.0)],
        out_bf16_bits=[[bf16_bits(rne), bf16_bits(rne)]]))

# 5. Two query rows sharing one KV head (G = 2) with a dominant token: the
#    score gap is 0.5 * 4096 = 2048 natural-log units, so every other weight
#    is e^-2048, below the smallest positive double, and out = V of that
#    token exactly.
cases.append(dict(
    name="argmax_group2", derivation="row0 picks token 1 (gap 2048), row1 picks token 0",
    q=[[1.0, 0.0], [0.0, 1.0]],
    K=[[0.0, 4096.0], [4096.0, 0.0], [0.0, 0.0]],
    V=[[7.0, -1.0], [0.5, 96.0], [3.0, 3.0]], scale=0.5,
    out=[[0.5, 96.0], [7.0, -1.0]], lse=[2048.0, 2048.0]))

for c in cases:
    for key in ("q", "K", "V"):
        c[key + "_bits"] = [[bf16_bits(x) for x in row] for row in c[key]]

path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "hand_cases.json")
with open(path, "w") as f:
    json.dump({"source": "closed forms of scaled dot-product softmax attention, derived by hand "
                         "(the paper prints no worked example)", "cases": cases}, f, indent=1)
print(f"wrote {len(cases)} cases to {path}")
