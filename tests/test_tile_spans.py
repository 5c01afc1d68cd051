"""Host logic of the data-movement reference: the spans of a decode step cover
every distinct block the batch uses exactly once (so the gather helper reads
the step's algorithmic K/V bytes, no more and no fewer)."""
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402
from workloads import build_config, group_starts, grouped_case, logical_case, page_case  # noqa: E402


def batch_of(w, S, prefix_len=0, pps=256, **kw):
    from paper_2510_14126_amd.device import PagedBatch
    if w.k_pool is None:                        # structure only: placeholder pools, never read
        w.q = np.zeros((w.batch, w.num_q_heads, w.head_dim), np.uint16)
        n = w.num_blocks * w.num_kv_heads * 16 * w.head_dim
        dummy = torch.zeros(1, dtype=torch.int16).expand(n)     # the pool's size, no storage
        kw.update(k_pool=dummy, v_pool=dummy)
    return PagedBatch(w, "cpu", partition_size=S, prefix_len=prefix_len,
                      prefix_partition_size=pps, **kw)


def blocks_read(w, spans):
    return [int(i) for b, s, e in spans for i in w.block_tables[b, s // 16:(e + 15) // 16]]


def used_blocks(w):
    nb = (w.context_lens.astype(np.int64) + 15) // 16
    return sorted({int(i) for b in range(w.batch) for i in w.block_tables[b, :nb[b]]})


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_bench_configurations_read_each_block_once(k):
    w = build_config(k, values=k < 4)
    L = 16 * int(w.meta.get("prefix_blocks", 0))
    kw = {}
    if L and "groups" in w.meta and w.meta.get("mid_blocks", 0):
        kw = dict(group_start=group_starts(w), group_len=16 * int(w.meta["mid_blocks"]))
    pb = batch_of(w, bench.DEFAULT_PARTITION[k], L, bench.default_prefix_partition(k, L) if L else 256,
                  **kw)
    spans = pb.tile_spans()
    got = blocks_read(w, spans)
    assert sorted(got) == used_blocks(w)
    assert (spans[:, 2] > spans[:, 1]).all()
    pb.close()


def test_per_sequence_partitions_longest_first():
    lc = logical_case(3, 5, 32, 8, 128, [700, 0, 130, 1300, 520])
    w = page_case(lc, 4)
    pb = batch_of(w, 256)
    spans = pb.tile_spans()
    n = spans[:, 2] - spans[:, 1]
    assert (np.diff(n) <= 0).all()
    # every partition of every sequence, tokens [p*S, min((p+1)*S, ctx))
    expect = sorted((b, s, min(s + 256, c)) for b, c in enumerate(w.context_lens) for s in range(0, c, 256))
    assert sorted(map(tuple, spans.tolist())) == expect
    assert sorted(blocks_read(w, spans)) == used_blocks(w)
    pb.close()


def test_groups_and_prefix_spans():
    w = grouped_case(11, 32, 8, 128, 256, [2, 1, 3], 64, [30, 0, 200, 5, 70, 16])
    pb = batch_of(w, 128, 256, 128, group_start=group_starts(w), group_len=64)
    spans = pb.tile_spans().tolist()
    assert spans[:2] == [[0, 0, 128], [0, 128, 256]]
    assert spans[2:5] == [[0, 256, 320], [2, 256, 320], [3, 256, 320]]
    assert sorted(blocks_read(w, spans)) == used_blocks(w)
    pb.close()
