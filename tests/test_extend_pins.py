"""Pins of the extend (chunked prefill) oracle (CPU only).

Checked against pure-Python brute force over each token's visible prefix, the
closed form of a chunk that starts the sequence (its first token sees only
itself, so its output is exactly V[0]), the decode oracle (a one-token chunk
is a decode step), invariance to physical block placement, and a planted
non-causal variant that must fail.
"""
import numpy as np
import pytest

from oracle import extend_attention, paged_decode
from oracle import brute
from oracle.attention import bf16_to_f64
from workloads import logical_case, page_case, permute_blocks
from workloads.generate import f32_to_bf16_bits


def _case(seed, ctx, chunk, hq=4, hkv=2, d=8):
    case = logical_case(seed, len(ctx), hq, hkv, d, ctx)
    w = page_case(case, seed + 1, share_prefix=False)
    rng = np.random.default_rng(seed + 2)
    q_start = np.concatenate([[0], np.cumsum(chunk)]).astype(np.int32)
    q = f32_to_bf16_bits(rng.standard_normal((int(q_start[-1]), hq, d), dtype=np.float32))
    return case, w, q, q_start


def _brute(case, q, q_start, chunk):
    outs = []
    hq = q.shape[1]
    hkv = case.num_kv_heads
    G = hq // hkv
    for b, L in enumerate(chunk):
        n = case.k[b].shape[1]
        keys = [[[brute.bf16_bits_to_float(x) for x in row] for row in case.k[b][g]] for g in range(hkv)]
        vals = [[[brute.bf16_bits_to_float(x) for x in row] for row in case.v[b][g]] for g in range(hkv)]
        for i in range(L):
            p = n - L + i
            row = []
            for h in range(hq):
                qr = [brute.bf16_bits_to_float(x) for x in q[q_start[b] + i][h]]
                o, _ = brute.attend(qr, keys[h // G][: p + 1], vals[h // G][: p + 1], case.scale)
                row.append(o)
            outs.append(row)
    return np.array(outs)


@pytest.mark.parametrize("ctx,chunk", [([5, 20], [5, 3]), ([33, 16, 47], [1, 16, 20])])
def test_extend_matches_brute_force(ctx, chunk):
    case, w, q, q_start = _case(3, ctx, chunk)
    out, _ = extend_attention(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale)
    np.testing.assert_allclose(out, _brute(case, q, q_start, chunk), rtol=1e-12, atol=1e-12)


def test_chunk_starting_the_sequence_first_token_returns_v0():
    case, w, q, q_start = _case(5, [12, 7], [12, 7])
    out, lse = extend_attention(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale)
    for b in range(2):
        first = out[q_start[b]]
        for h in range(4):
            assert np.array_equal(first[h], bf16_to_f64(case.v[b][h // 2][0]))


def test_one_token_chunks_equal_decode():
    case, w, q, q_start = _case(7, [30, 17, 64], [1, 1, 1])
    out, lse = extend_attention(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale)
    ref, ref_lse = paged_decode(q, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale)
    assert np.array_equal(out, ref) and np.array_equal(lse, ref_lse)


def test_block_placement_does_not_matter():
    case, w, q, q_start = _case(9, [40, 25], [10, 25])
    a, _ = extend_attention(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale)
    w2 = permute_blocks(w, 10)
    b, _ = extend_attention(q, q_start, w2.k_pool, w2.v_pool, w2.block_tables, w2.context_lens, w2.scale)
    assert np.array_equal(a, b)


def test_planted_non_causal_variant_fails():
    ctx, chunk = [20, 9], [6, 9]
    case, w, q, q_start = _case(11, ctx, chunk)
    # planted mistake: every chunk token attends to the whole context
    wide = np.zeros((int(q_start[-1]), 4, 8))
    for b, L in enumerate(chunk):
        for i in range(L):
            o, _ = paged_decode(q[q_start[b] + i][None], w.k_pool, w.v_pool, w.block_tables[b:b + 1],
                                w.context_lens[b:b + 1], w.scale)
            wide[q_start[b] + i] = o[0]
    assert not np.allclose(wide, _brute(case, q, q_start, chunk), rtol=1e-6, atol=1e-6)


def test_chunk_longer_than_context_is_rejected():
    case, w, q, q_start = _case(13, [4], [4])
    with pytest.raises(ValueError):
        extend_attention(q, np.array([0, 4]), w.k_pool, w.v_pool, w.block_tables, np.array([3]), w.scale)
