"""The oracle's process pool returns the single-process oracle's results.

The pool only divides a batch's sequences among worker processes (one BLAS
thread each); each sequence goes through the same oracle function, so the
results must be bit-identical to a single-process call with one BLAS thread.
"""
import numpy as np
from threadpoolctl import threadpool_limits

from oracle import extend_attention, paged_decode, split_partials
from workloads import f32_to_bf16_bits, logical_case, page_case


def _case():
    lc = logical_case(5, 9, 16, 4, 64, [300, 47, 1, 0, 129, 513, 64, 700, 96], prefix_len=0)
    return page_case(lc, 6, poison=True)


def test_pool_decode_matches_single_process(oracle_pool):
    w = _case()
    with threadpool_limits(1):
        ref, rl = paged_decode(w.q, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale)
    out, lse = oracle_pool.decode_workload(w)
    assert np.array_equal(out, ref) and np.array_equal(lse, rl)
    sub, subl = oracle_pool.decode_workload(w, seqs=[7, 2, 0])
    assert np.array_equal(sub, ref[[7, 2, 0]]) and np.array_equal(subl, rl[[7, 2, 0]])


def test_pool_split_partials_match_single_process(oracle_pool):
    w = _case()
    with threadpool_limits(1):
        ro, rl = split_partials(w.q, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale, 128)
    o, lse = oracle_pool.split_partials(w.q, w.k_pool, w.v_pool, w.block_tables, w.context_lens,
                                        w.scale, 128)
    assert np.array_equal(o, ro) and np.array_equal(lse, rl)


def test_pool_extend_matches_single_process(oracle_pool):
    w = _case()
    chunk = np.array([20, 1, 1, 0, 129, 13, 64, 5, 96])
    q_start = np.concatenate([[0], np.cumsum(chunk)]).astype(np.int32)
    rng = np.random.default_rng(7)
    q = f32_to_bf16_bits(rng.standard_normal((int(q_start[-1]), 16, 64), dtype=np.float32))
    with threadpool_limits(1):
        ro, rl = extend_attention(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens,
                                  w.scale)
    o, lse = oracle_pool.extend(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens,
                                w.scale)
    assert np.array_equal(o, ro) and np.array_equal(lse, rl)
