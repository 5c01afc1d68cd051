"""Parity gate between a bf16 GPU output and the float64 oracle.

TEST INFRASTRUCTURE ONLY (see ``oracle.attention``).

The tolerance is the one the hot path is held to: bf16 outputs accumulated in
fp32 must match the fp64 reference within max absolute error 2e-2 and max
relative error 1e-2.  Read element-wise in the ``assert_close`` form

    |g - r| <= 2e-2 + 1e-2 |r|                      for every element,

plus a discriminating per-row check, because long-context outputs are about
1e-2 in magnitude and an absolute bound alone would accept an all-zero row:

    ||g_row - r_row||_2 <= 1e-2 ||r_row||_2          for every (sequence, head).

A reference row that is exactly zero (an empty context) must be matched by an
exactly zero row.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .attention import bf16_to_f64

ATOL = 2e-2
RTOL = 1e-2
ROW_REL_L2 = 1e-2


@dataclass
class GateReport:
    passed: bool
    max_abs: float
    max_rel: float          # over |r| >= 1e-3
    worst_row_rel_l2: float
    n_bad_elements: int
    n_bad_rows: int
    n_elements: int

    def __str__(self):
        return (f"gate {'PASS' if self.passed else 'FAIL'}: max_abs={self.max_abs:.3e} "
                f"max_rel={self.max_rel:.3e} worst_row_rel_l2={self.worst_row_rel_l2:.3e} "
                f"bad_elems={self.n_bad_elements}/{self.n_elements} bad_rows={self.n_bad_rows}")


def compare(gpu, ref, atol: float = ATOL, rtol: float = RTOL, row_rel_l2: float = ROW_REL_L2,
            gpu_is_bf16_bits: bool = True) -> GateReport:
    """Gate a GPU result [..., D] (bf16 bits, or floats) against ref [..., D]."""
    g = bf16_to_f64(gpu) if gpu_is_bf16_bits else np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if g.shape != r.shape:
        raise ValueError(f"shape mismatch {g.shape} vs {r.shape}")
    if g.size == 0:
        return GateReport(True, 0.0, 0.0, 0.0, 0, 0, 0)
    err = np.abs(g - r)
    err = np.where(np.isnan(err), np.inf, err)
    bad_el = ~(err <= atol + rtol * np.abs(r))
    big = np.abs(r) >= 1e-3
    max_rel = float(np.max(err[big] / np.abs(r[big]))) if big.any() else 0.0
    rn = np.sqrt((r * r).sum(axis=-1))
    finite_rows = np.isfinite(err).all(axis=-1)
    en = np.where(finite_rows,
                  np.sqrt((np.where(np.isfinite(err), err, 0.0) ** 2).sum(axis=-1)), np.inf)
    zero_rows = rn == 0
    rel = np.where(zero_rows, np.where(en == 0, 0.0, np.inf), en / np.where(zero_rows, 1.0, rn))
    bad_rows = ~(rel <= row_rel_l2)
    return GateReport(passed=bool(not bad_el.any() and not bad_rows.any()),
                      max_abs=float(err.max()), max_rel=max_rel,
                      worst_row_rel_l2=float(rel.max()), n_bad_elements=int(bad_el.sum()),
                      n_bad_rows=int(bad_rows.sum()), n_elements=int(g.size))
