"""Pins of the CPU oracle against things other than itself.

Closed forms (hand-derived golden cases), brute force on tiny inputs,
invariants of paging and softmax, and planted mistakes that must fail.
"""
import json
import math
import os
import struct

import numpy as np
import pytest

import oracle.attention as oa
from oracle import brute, compare
from workloads import (build_config, duplicate_shared_blocks, f32_to_bf16_bits, logical_case,
                       page_case, permute_blocks)

HERE = os.path.dirname(os.path.abspath(__file__))
with open(os.path.join(HERE, "golden", "hand_cases.json")) as f:
    HAND = json.load(f)["cases"]


def _pool_from_logical(k_bits, v_bits, perm_seed=0):
    """One sequence, one KV head: place tokens in a shuffled pool by hand."""
    k_bits = np.asarray(k_bits, np.uint16); v_bits = np.asarray(v_bits, np.uint16)
    n, d = k_bits.shape
    nb = (n + 15) // 16
    rng = np.random.default_rng(perm_seed)
    ids = rng.permutation(nb + 2)[:nb].astype(np.int32)
    kp = np.zeros((nb + 2, 1, 16, d), np.uint16); vp = np.zeros_like(kp)
    for t in range(n):
        kp[ids[t // 16], 0, t % 16] = k_bits[t]; vp[ids[t // 16], 0, t % 16] = v_bits[t]
    return kp, vp, ids[None, :], np.array([n], np.int32)


# ---------------------------------------------------------------- bf16 decode

def test_bf16_decode_known_values():
    bits = np.array([0x3F80, 0xC000, 0x4300, 0x4302, 0x0001, 0x7F80, 0xFF80, 0x8000], np.uint16)
    want = [1.0, -2.0, 128.0, 130.0, 2.0 ** -133, math.inf, -math.inf, -0.0]
    got = oa.bf16_to_f64(bits)
    for g, w in zip(got, want):
        assert g == w and math.copysign(1, g) == math.copysign(1, w)
    assert np.isnan(oa.bf16_to_f64(np.array([0x7FC0], np.uint16)))[0]


# ---------------------------------------------------------- hand golden cases

@pytest.mark.parametrize("case", HAND, ids=[c["name"] for c in HAND])
def test_hand_cases(case):
    q = np.array(case["q_bits"], np.uint16)[None]          # [1][R][D]
    kp, vp, bt, ctx = _pool_from_logical(case["K_bits"], case["V_bits"], perm_seed=len(case["K"]))
    out, lse = oa.paged_decode(q, kp, vp, bt, ctx, case["scale"])
    np.testing.assert_allclose(out[0], np.array(case["out"]), rtol=1e-15, atol=1e-15)
    np.testing.assert_allclose(lse[0], np.array(case["lse"]), rtol=1e-15, atol=1e-15)


def test_rne_tie_cases_distinguish_rounding_modes():
    """The tie cases separate RNE from truncation and from round-half-away."""
    def f32_bits(x):
        return struct.unpack("<I", struct.pack("<f", x))[0]
    ties = [c for c in HAND if c["name"].startswith("rne_tie")]
    assert len(ties) >= 2
    trunc_ok = away_ok = True
    for c in ties:
        exact = c["out"][0][0]
        want = c["out_bf16_bits"][0][0]
        trunc = f32_bits(exact) >> 16
        away = (f32_bits(exact) + 0x8000) >> 16
        trunc_ok &= trunc == want
        away_ok &= away == want
        assert int(f32_to_bf16_bits(np.float32([exact]))[0]) == want
    assert not trunc_ok and not away_ok


# ------------------------------------------------------------- brute force

TINY_SHAPES = [
    # seed, B, Hq, Hkv, D, ctx list, prefix
    (1, 1, 1, 1, 4, [1], 0),
    (2, 2, 4, 2, 8, [5, 17], 0),
    (3, 3, 4, 1, 16, [16, 33, 40], 16),
    (4, 4, 8, 2, 8, [32, 17, 39, 16], 16),
    (5, 2, 2, 2, 16, [40, 3], 0),
    (6, 4, 8, 2, 16, [35, 40, 38, 33], 32),
]


@pytest.mark.parametrize("shape", TINY_SHAPES)
def test_oracle_matches_bruteforce_tiny(shape):
    seed, B, hq, hkv, d, ctx, pre = shape
    case = logical_case(seed, B, hq, hkv, d, ctx, prefix_len=pre)
    w = page_case(case, seed + 100, share_prefix=True)
    out, lse = oa.decode_workload(w)
    bo, bl = brute.decode_logical(case.q.tolist(), [k.tolist() for k in case.k],
                                  [v.tolist() for v in case.v], case.scale)
    bo = np.array(bo); bl = np.array(bl)
    np.testing.assert_allclose(out, bo, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, bl, rtol=1e-12, atol=1e-13)


def test_oracle_matches_bruteforce_tiny_config():
    """The whole 4-sequence tiny configuration, brute-forced through its own gather."""
    w = build_config(1)
    out, lse = oa.decode_workload(w)
    bo, bl = brute.decode_paged(w.q.tolist(), w.k_pool.tolist(), w.v_pool.tolist(),
                                w.block_tables.tolist(), w.context_lens.tolist(), w.scale)
    np.testing.assert_allclose(out, np.array(bo), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, np.array(bl), rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------- paging invariants

def _shared_case(seed=11):
    case = logical_case(seed, 4, 8, 2, 16, [70, 48, 90, 33], prefix_len=32)
    return page_case(case, seed, share_prefix=True, extra_blocks=5)


@pytest.mark.parametrize("builder", ["tiny_config", "shared"])
def test_block_permutation_bit_identical(builder):
    w = build_config(1) if builder == "tiny_config" else _shared_case()
    o1, l1 = oa.decode_workload(w)
    for s in range(3):
        o2, l2 = oa.decode_workload(permute_blocks(w, 50 + s))
        assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_shared_prefix_equals_duplicated_copies():
    w = _shared_case()
    assert w.meta["shared_blocks"] == 2
    d = duplicate_shared_blocks(w)
    assert d.meta["duplicated"] == 2 * 3
    o1, l1 = oa.decode_workload(w)
    o2, l2 = oa.decode_workload(d)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_unread_slots_never_matter():
    """Poisoned rows past ctx and unused blocks (K huge, V NaN) give the same bits."""
    case = logical_case(21, 3, 4, 2, 16, [17, 31, 5], prefix_len=0)
    clean = page_case(case, 7, poison=False)
    dirty = page_case(case, 7, poison=True)
    assert np.isnan(oa.bf16_to_f64(dirty.v_pool)).any()
    o1, l1 = oa.decode_workload(clean)
    o2, l2 = oa.decode_workload(dirty)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    assert np.isfinite(o2).all()


# ------------------------------------------------------------ softmax closed forms

def test_weights_sum_to_one():
    w = build_config(1)
    _, _, ws = oa.decode_workload(w, return_weights=True)
    for wb in ws:
        np.testing.assert_allclose(wb.sum(axis=1), 1.0, rtol=0, atol=1e-12)
        assert (wb >= 0).all()


def test_single_token_returns_v_exactly():
    case = logical_case(31, 3, 8, 2, 32, [1, 1, 1])
    w = page_case(case, 3)
    out, lse = oa.decode_workload(w)
    for b in range(3):
        for h in range(8):
            g = h // 4
            assert np.array_equal(out[b, h], oa.bf16_to_f64(case.v[b][g, 0]))
            k = oa.bf16_to_f64(case.k[b][g, 0]); qv = oa.bf16_to_f64(case.q[b, h])
            assert lse[b, h] == pytest.approx(case.scale * float(k @ qv), rel=1e-14, abs=1e-14)


def test_zero_query_gives_mean_of_v():
    case = logical_case(32, 2, 4, 1, 8, [37, 20])
    case.q[:] = 0
    w = page_case(case, 4)
    out, lse = oa.decode_workload(w)
    for b in range(2):
        mean = oa.bf16_to_f64(case.v[b][0]).mean(axis=0)
        np.testing.assert_allclose(out[b], np.broadcast_to(mean, out[b].shape), rtol=1e-13,
                                   atol=1e-14)
        np.testing.assert_allclose(lse[b], math.log(case.context_lens[b]), rtol=1e-14)


def test_constant_v_rows():
    case = logical_case(33, 2, 4, 2, 8, [29, 45])
    for b in range(2):
        case.v[b][:] = f32_to_bf16_bits(np.float32([[[-2.75]]]))[0, 0, 0]
    out, _ = oa.decode_workload(page_case(case, 5))
    np.testing.assert_allclose(out, -2.75, rtol=1e-14, atol=0)


def test_two_token_weight_closed_form():
    case = logical_case(34, 1, 2, 1, 16, [2])
    out, lse, ws = oa.decode_workload(page_case(case, 6), return_weights=True)
    k = oa.bf16_to_f64(case.k[0][0]); q = oa.bf16_to_f64(case.q[0])
    for h in range(2):
        s0, s1 = case.scale * float(q[h] @ k[0]), case.scale * float(q[h] @ k[1])
        assert ws[0][h, 0] == pytest.approx(1.0 / (1.0 + math.exp(s1 - s0)), rel=1e-14)


def test_query_scale_tradeoff_invariance():
    """q * 2 with scale / 2 (both exact) leaves the result unchanged."""
    case = logical_case(35, 2, 4, 2, 16, [40, 23])
    w = page_case(case, 7)
    o1, l1 = oa.decode_workload(w)
    q2 = f32_to_bf16_bits(oa.bf16_to_f64(case.q).astype(np.float32) * 2)
    o2, l2 = oa.paged_decode(q2, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale / 2)
    np.testing.assert_allclose(o1, o2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-13, atol=1e-14)


def test_empty_context():
    case = logical_case(36, 2, 4, 2, 8, [0, 5])
    out, lse = oa.decode_workload(page_case(case, 8))
    assert np.array_equal(out[0], np.zeros_like(out[0])) and np.all(lse[0] == -np.inf)
    assert np.isfinite(out[1]).all()


# ----------------------------------------------------------------- split merge

@pytest.mark.parametrize("S", [16, 64, 512, 4096])
def test_split_merge_equals_unsplit(S):
    case = logical_case(41, 3, 8, 2, 16, [700, 16, 513], prefix_len=0)
    w = page_case(case, 9)
    full, lfull = oa.decode_workload(w)
    o, l = oa.split_partials(w.q, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale, S)
    merged, lm = oa.merge_partials(o, l)
    np.testing.assert_allclose(merged, full, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lm, lfull, rtol=1e-12, atol=1e-13)
    # the last partition of each sequence ends at its context length
    for b, n in enumerate(w.context_lens):
        pb = -(-int(n) // S)
        assert np.all(np.isfinite(l[b, :, :pb])) and np.all(l[b, :, pb:] == -np.inf)


def test_merge_of_single_partition_is_identity():
    o = np.random.default_rng(0).standard_normal((3, 4, 1, 8))
    lse = np.random.default_rng(1).standard_normal((3, 4, 1))
    m, l = oa.merge_partials(o, lse)
    assert np.array_equal(m, o[:, :, 0]) and np.array_equal(l, lse[..., 0])


def test_merge_of_empty_rows():
    o = np.zeros((2, 3, 8)); lse = np.full((2, 3), -np.inf)
    m, l = oa.merge_partials(o, lse)
    assert np.array_equal(m, np.zeros((2, 8))) and np.all(l == -np.inf)


# ----------------------------------------------------------- argmax selection

def argmax_case(d=16, ctx=(40, 23), target=(39, 16), hq=4, hkv=1, seed=3):
    """K of one target token = 4096 e0, q = e0: out = V of that token exactly.

    V encodes (physical block mod 256, physical block div 256, row) as exact
    bf16 integers so the output names the slot that was read.
    """
    case = logical_case(seed, len(ctx), hq, hkv, d, list(ctx))
    w = page_case(case, seed + 1, extra_blocks=4)
    e0 = np.zeros(d, np.float32); e0[0] = 1.0
    w.q[:] = f32_to_bf16_bits(e0)
    w.k_pool[..., :] = 0
    want = []
    for b, t in enumerate(target):
        pid = int(w.block_tables[b, t // 16]); row = t % 16
        w.k_pool[pid, :, row, 0] = 0x4580  # 4096.0
        want.append((pid, row))
    for pid in range(w.num_blocks):
        for row in range(16):
            w.v_pool[pid, :, row, :] = 0
            w.v_pool[pid, :, row, 0:3] = f32_to_bf16_bits(np.float32([pid % 256, pid // 256, row]))
    return w, want


def test_argmax_selects_exact_slot():
    w, want = argmax_case()
    out, _ = oa.decode_workload(w)
    for b, (pid, row) in enumerate(want):
        for h in range(w.num_q_heads):
            assert out[b, h, 0] == pid % 256 and out[b, h, 1] == pid // 256 and out[b, h, 2] == row


# ------------------------------------------------- planted mistakes must fail

def _brute_vs_oracle_ok():
    case = logical_case(4, 4, 8, 2, 8, [32, 17, 39, 16], prefix_len=16)
    w = page_case(case, 104)
    out, _ = oa.decode_workload(w)
    bo, _ = brute.decode_logical(case.q.tolist(), [k.tolist() for k in case.k],
                                 [v.tolist() for v in case.v], case.scale)
    return np.allclose(out, np.array(bo), rtol=1e-12, atol=1e-13)


def test_planted_head_map_fails(monkeypatch):
    assert _brute_vs_oracle_ok()
    monkeypatch.setattr(oa, "kv_head_for", lambda h, hq, hkv: h % hkv)
    assert not _brute_vs_oracle_ok()


def test_planted_dropped_last_token_fails(monkeypatch):
    real = oa.softmax_attention

    def drop_last(q_rows, k, v, scale):
        o, l, w = real(q_rows, k[:-1], v[:-1], scale)
        return o, l, np.concatenate([w, np.zeros((w.shape[0], 1))], axis=1)
    monkeypatch.setattr(oa, "softmax_attention", drop_last)
    assert not _brute_vs_oracle_ok()


def test_planted_swapped_table_entries_fail():
    """Swapping a full block with the partial last block moves the target out
    of the context (a swap of two full blocks is invisible: attention does not
    depend on token order)."""
    w, want = argmax_case(ctx=(40,), target=(12,))   # last block keeps rows 0..7
    w.block_tables[0, [0, 2]] = w.block_tables[0, [2, 0]]
    out, _ = oa.decode_workload(w)
    pid, row = want[0]
    assert not (out[0, 0, 0] == pid % 256 and out[0, 0, 1] == pid // 256)


def test_gate_rejects_zero_and_accepts_rounded_truth():
    w = build_config(1)
    out, _ = oa.decode_workload(w)
    rounded = f32_to_bf16_bits(out.astype(np.float32))
    ok = compare(rounded, out)
    assert ok.passed, str(ok)
    assert ok.worst_row_rel_l2 < 5e-3
    assert not compare(np.zeros_like(rounded), out).passed
    bad = rounded.copy(); bad[0, 0, 5] = 0x7FC0
    assert not compare(bad, out).passed


def test_gate_rejects_planted_kernel_style_mistakes():
    """Outputs of planted mistakes in the oracle fail the gate against the truth."""
    case = logical_case(51, 4, 8, 2, 64, [300, 150, 257, 100])
    w = page_case(case, 52)
    truth, _ = oa.decode_workload(w)
    # dropped last token
    ctx2 = w.context_lens - 1
    o_drop, _ = oa.paged_decode(w.q, w.k_pool, w.v_pool, w.block_tables, ctx2, w.scale)
    # first table entry swapped with the partial last one
    bt = w.block_tables.copy()
    for b, n in enumerate(w.context_lens):
        last = (int(n) - 1) // 16
        bt[b, [0, last]] = bt[b, [last, 0]]
    o_swap, _ = oa.paged_decode(w.q, w.k_pool, w.v_pool, bt, w.context_lens, w.scale)
    for bad in (o_drop, o_swap):
        assert not compare(f32_to_bf16_bits(bad.astype(np.float32)), truth).passed
