"""Host-side block accounting of the footprint experiment (CPU only): the
pool allocator's blocks in use equal the distinct blocks the tables map, with
shared prompt blocks counted once, and equal the sum of per-sequence block
counts once every sequence holds private copies."""
import numpy as np

import bench
from workloads import build_config, duplicate_shared_blocks, logical_case, page_case


def test_stage_batches_count_shared_blocks_once():
    for k in (2, 3):
        w = build_config(k, values=False)
        assert bench._blocks_in_use(w) == w.meta["needed_blocks"]


def test_private_copies_count_every_sequence():
    case = logical_case(5, 6, 8, 2, 64, [40, 70, 33, 64, 100, 48], prefix_len=32)
    w = page_case(case, 6, share_prefix=True)
    shared = bench._blocks_in_use(w)
    wd = duplicate_shared_blocks(w)
    private = bench._blocks_in_use(wd)
    per_seq = int(((w.context_lens + 15) // 16).sum())
    assert private == per_seq
    assert shared == per_seq - (w.batch - 1) * (32 // 16)


def test_bench_launch_configurations():
    """The launch bench.py times: stated 512-token partitions on the
    long-context pool, the cascade wherever a prefix is shared, request groups
    on the fixer batch."""
    expect = {1: (512, None, False), 2: (512, 2048, False), 3: (1024, 2048, True),
              4: (8192, None, False), 5: (512, 4096, False)}
    for k, (S, L, groups) in expect.items():
        w = build_config(k, values=False)
        s, kw = bench.launch_configuration(k, w)
        assert s == S
        assert kw.get("prefix_len") == L
        assert ("group_len" in kw) == groups
    w = build_config(5, values=False)
    assert bench.launch_configuration(5, w)[1]["prefix_partition_size"] == 512
    assert bench.launch_configuration(5, w, cascade="off")[1] == {}
