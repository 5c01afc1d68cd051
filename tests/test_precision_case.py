"""Pins of the near-tie decode input (tests/precision_case.py): the oracle
reproduces its closed form, and the input tells apart exact weights from
weights rounded to bf16 before the PV product (the GPU test then requires
the exact behaviour)."""
import numpy as np

from oracle import compare, decode_workload
from precision_case import P_A, P_B, exact_output, near_tie_case


def bf16_round(x):
    """Round to bf16 (nearest even), as float64."""
    f = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = ((f + 0x7FFF + ((f >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def test_weights_straddle_bf16_rounding_points():
    assert bf16_round(P_A) == 0.5 + 2.0 ** -8 and bf16_round(P_B) == 0.5
    assert 0.5 < P_B < 0.5 + 2.0 ** -9 < P_A


def test_oracle_matches_the_closed_form():
    w = near_tie_case([16, 100, 4099], hq=8, hkv=2, seed=1)
    out, _ = decode_workload(w)
    for b, n in enumerate(w.context_lens):
        assert np.allclose(out[b], exact_output(int(n)), rtol=1e-12, atol=0)


def test_bf16_weights_fail_the_gate_and_hi_lo_weights_pass():
    n = 4096
    roles = np.arange(n) % 16
    role = np.where((roles == 0) | (roles == 15), 0, np.where(roles % 2 == 1, 1, 2))
    p = np.where(role == 0, 1.0, np.where(role == 1, P_A, P_B)).astype(np.float32)
    v = np.where(role == 0, 0.0, np.where(role == 1, 1.0, -1.0))
    exact = exact_output(n)
    # weights rounded to bf16 in both the PV product and the row sum
    pr = bf16_round(p)
    rounded = (pr * v).sum() / pr.sum()
    # weights split into a bf16 high part and a bf16 low part, row sum in fp32
    lo = bf16_round(p.astype(np.float64) - pr)
    split = ((pr + lo) * v).sum() / p.astype(np.float64).sum()
    ref = np.full((1, 1, 128), exact)
    assert not compare(np.full((1, 1, 128), rounded), ref, gpu_is_bf16_bits=False).passed
    assert rounded / exact > 1.4            # 45% too large
    assert compare(np.full((1, 1, 128), split), ref, gpu_is_bf16_bits=False).passed
    assert abs(split / exact - 1.0) < 1e-3
