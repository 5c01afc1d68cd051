"""Pins of the KV-append oracle (CPU only).

The oracle's append is checked against things it does not compute itself: the
logical per-sequence K/V that the generator builds before paging, the brute
force gather and attention of ``oracle.brute``, and an element-wise diff of
the pools.  A planted off-by-one (writing slot ctx instead of ctx - 1) must
fail.
"""
import numpy as np
import pytest

from oracle import append_kv, paged_decode
from oracle import brute
from workloads import logical_case, page_case
from workloads.generate import f32_to_bf16_bits

BS = 16


def _random_pool(seed, nb=12, hkv=2, d=8):
    rng = np.random.default_rng(seed)
    kp = f32_to_bf16_bits(rng.standard_normal((nb, hkv, BS, d), dtype=np.float32))
    vp = f32_to_bf16_bits(rng.standard_normal((nb, hkv, BS, d), dtype=np.float32))
    return rng, kp, vp


def test_append_writes_exactly_the_new_slot():
    rng, kp, vp = _random_pool(1)
    bt = np.array([[3, 7, -1], [5, -1, -1], [9, 2, 11], [0, -1, -1]], np.int32)
    ctx = np.array([17, 16, 40, 0], np.int32)        # mid block, block end, third block, empty
    kn = f32_to_bf16_bits(rng.standard_normal((4, 2, 8), dtype=np.float32))
    vn = f32_to_bf16_bits(rng.standard_normal((4, 2, 8), dtype=np.float32))
    k2, v2 = append_kv(kp, vp, bt, ctx, kn, vn)
    expect = {(7, 0): 0, (5, 15): 1, (11, 7): 2}     # (physical block, row) -> sequence
    changed_k = {tuple(ix[[0, 2]]) for ix in np.argwhere(k2 != kp)}
    changed_v = {tuple(ix[[0, 2]]) for ix in np.argwhere(v2 != vp)}
    assert changed_k <= set(expect) and changed_v <= set(expect)
    for (pid, row), b in expect.items():
        assert np.array_equal(k2[pid, :, row, :], kn[b])
        assert np.array_equal(v2[pid, :, row, :], vn[b])
    # untouched pools are not modified in place
    assert not np.shares_memory(k2, kp)


def _append_off_by_one(k_pool, v_pool, block_tables, context_lens, k_new, v_new):
    """A planted mistake: writes slot ctx instead of ctx - 1."""
    k, v = k_pool.copy(), v_pool.copy()
    for b, n in enumerate(context_lens):
        n = int(n)
        if n <= 0:
            continue
        phys = int(block_tables[b, n // BS])
        k[phys, :, n % BS, :] = k_new[b]
        v[phys, :, n % BS, :] = v_new[b]
    return k, v


def _grow(case_full, n0, seed, append=append_kv):
    """Page the first n0[b] tokens of each sequence, then append the rest one
    decode step at a time, taking a fresh block from a free list whenever a
    new token starts a block (one spare block per sequence past its end so a
    planted off-by-one stays in bounds).  Returns (k_pool, v_pool, tables, ctx)."""
    B, hq, d = case_full.q.shape
    pre = logical_case(0, B, hq, case_full.num_kv_heads, d, n0)
    pre.k = [k[:, :n, :].copy() for k, n in zip(case_full.k, n0)]
    pre.v = [v[:, :n, :].copy() for v, n in zip(case_full.v, n0)]
    pre.q = case_full.q
    extra = sum((k.shape[1] + BS - 1) // BS + 1 for k in case_full.k) + 2
    w = page_case(pre, seed, share_prefix=False, extra_blocks=extra, table_pad=64)
    used = set(int(x) for x in w.block_tables[w.block_tables >= 0])
    free = [i for i in range(w.num_blocks) if i not in used]
    kp, vp, bt = w.k_pool, w.v_pool, w.block_tables.copy()
    for b in range(B):                       # spare block after the last one
        bt[b, (case_full.k[b].shape[1] + BS - 1) // BS] = free.pop()
    ctx = np.array(n0, np.int32)
    final = np.array([k.shape[1] for k in case_full.k])
    while np.any(ctx < final):
        grow = ctx < final
        new_ctx = ctx + grow
        for b in np.nonzero(grow)[0]:
            t = int(new_ctx[b]) - 1
            if t % BS == 0 and t // BS < (final[b] + BS - 1) // BS:
                bt[b, t // BS] = free.pop()
        kn = np.stack([case_full.k[b][:, int(new_ctx[b]) - 1, :] for b in range(B)])
        vn = np.stack([case_full.v[b][:, int(new_ctx[b]) - 1, :] for b in range(B)])
        step_ctx = np.where(grow, new_ctx, 0)          # finished sequences append nothing
        kp, vp = append(kp, vp, bt, step_ctx, kn, vn)
        ctx = new_ctx
    return kp, vp, bt, ctx


def _logical_equal(kp, vp, bt, ctx, case):
    for b in range(len(ctx)):
        got_k = brute.gather_paged(kp, bt[b], int(ctx[b]))
        got_v = brute.gather_paged(vp, bt[b], int(ctx[b]))
        for g in range(case.num_kv_heads):
            if [list(r) for r in got_k[g]] != [list(r) for r in case.k[b][g]]:
                return False
            if [list(r) for r in got_v[g]] != [list(r) for r in case.v[b][g]]:
                return False
    return True


@pytest.mark.parametrize("n0,final", [([1, 16, 5], [40, 33, 5]), ([15, 17], [48, 18])])
def test_appends_rebuild_the_logical_sequences(n0, final):
    case = logical_case(21, len(final), 4, 2, 8, final)
    kp, vp, bt, ctx = _grow(case, n0, seed=22)
    assert list(ctx) == final
    assert _logical_equal(kp, vp, bt, ctx, case)


def test_decode_after_appends_matches_brute_force():
    final = [37, 20]
    case = logical_case(31, 2, 4, 2, 8, final)
    kp, vp, bt, ctx = _grow(case, [3, 16], seed=32)
    out, _ = paged_decode(case.q, kp, vp, bt, ctx, case.scale)
    ref, _ = brute.decode_logical(case.q, case.k, case.v, case.scale)
    np.testing.assert_allclose(out, np.array(ref), rtol=1e-12, atol=1e-12)


def test_planted_off_by_one_fails():
    final = [21, 34]
    case = logical_case(41, 2, 4, 2, 8, final)
    kp, vp, bt, ctx = _grow(case, [3, 16], seed=42, append=_append_off_by_one)
    assert not _logical_equal(kp, vp, bt, ctx, case)
