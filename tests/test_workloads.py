"""Structure of the seeded stage-shaped workloads (no attention arithmetic)."""
import math

import numpy as np
import pytest

from workloads import build_config, f32_to_bf16_bits, normal_bf16, touched_slots


def _used(w):
    nb = w.blocks_per_seq()
    return [list(w.block_tables[b, : nb[b]]) for b in range(w.batch)]


def _check_tables(w):
    nb = w.blocks_per_seq()
    for b in range(w.batch):
        row = w.block_tables[b]
        assert (row[: nb[b]] >= 0).all() and (row[: nb[b]] < w.num_blocks).all()
        assert (row[nb[b]:] == -1).all()


def test_tiny():
    w = build_config(1, values=False)
    assert (w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.num_blocks) == (4, 8, 2, 64, 128)
    assert w.context_lens.min() >= 100 and w.context_lens.max() <= 300
    ids = sum(_used(w), [])
    assert len(ids) == len(set(ids)) <= 128
    assert w.scale == 1 / 8
    _check_tables(w)


def test_sql_generator_shares_one_schema_prefix():
    w = build_config(2, values=False)
    assert (w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim) == (64, 32, 8, 128)
    suf = w.context_lens - 2048
    assert suf.min() >= 64 and suf.max() <= 512
    used = _used(w)
    pre = used[0][:128]
    assert all(u[:128] == pre for u in used)
    rest = sum((u[128:] for u in used), [])
    assert len(rest) == len(set(rest)) and not set(rest) & set(pre)
    assert w.num_blocks == math.ceil(1.2 * w.meta["needed_blocks"])
    _check_tables(w)


def test_sql_error_fixer_retries_share_prefix_and_first_attempt():
    w = build_config(3, values=False)
    retries = w.meta["retries"]
    assert len(retries) == 32 and retries.min() >= 1 and retries.max() <= 5
    assert w.batch == retries.sum()
    assert w.context_lens.min() >= 2432 and w.context_lens.max() <= 3328
    used = _used(w)
    groups = w.meta["groups"]
    pre = used[0][:128]
    for b in range(w.batch):
        assert used[b][:128] == pre
        same = [c for c in range(w.batch) if groups[c] == groups[b]]
        assert all(used[c][128:144] == used[b][128:144] for c in same)
        other = [c for c in range(w.batch) if groups[c] != groups[b]]
        assert all(not set(used[c][128:144]) & set(used[b][128:144]) for c in other)
    _check_tables(w)


def test_shared_pool_is_half_holes_and_unshared():
    w = build_config(4, values=False)
    assert w.batch == 256 and w.num_kv_heads == 8 and w.num_q_heads == 32
    assert w.context_lens.min() >= 64 and w.context_lens.max() <= 8192
    tags = list(w.meta["tags"])
    assert tags.count("generator") == 128 and tags.count("fixer") == 128
    ids = sum(_used(w), [])
    assert len(ids) == len(set(ids)) == w.meta["needed_blocks"]
    assert w.num_blocks == 2 * len(ids)
    assert 1300 < w.context_lens.mean() < 1700
    _check_tables(w)


def test_long_context_prefix():
    w = build_config(5, values=False)
    assert (w.batch, w.num_q_heads, w.num_kv_heads) == (128, 64, 8)
    assert w.context_lens.min() >= 8192 and w.context_lens.max() <= 32768
    used = _used(w)
    assert all(u[:256] == used[0][:256] for u in used)
    _check_tables(w)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_structure_is_deterministic(k):
    a, b = build_config(k, values=False), build_config(k, values=False)
    assert np.array_equal(a.block_tables, b.block_tables)
    assert np.array_equal(a.context_lens, b.context_lens)


def test_touched_slots_counts_shared_blocks_once():
    w = build_config(2, values=False)
    uniq = 2048 + int((w.context_lens - 2048).sum())
    assert touched_slots(w) == uniq


def test_values_independent_of_threads():
    a = normal_bf16((3, 1 << 21), 9, 1, threads=1)
    b = normal_bf16((3, 1 << 21), 9, 1, threads=4)
    assert np.array_equal(a, b)
    x = a.astype(np.uint32) << 16
    f = x.view(np.float32)
    assert abs(f.mean()) < 5e-3 and abs(f.std() - 1) < 5e-3


def test_bf16_encoding_rounds_to_nearest_even():
    vals = np.float32([1.0, 128.5, 129.5, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, np.nan, -0.0])
    want = [0x3F80, 0x4300, 0x4302, 0x3F80, 0x3F82, 0x7FC0, 0x8000]
    assert list(f32_to_bf16_bits(vals)) == want
