"""GPU tests of host-built work lists.

A scheduled decode runs the same per-item arithmetic as the unscheduled grid,
only in another order and without the empty partitions, so every output must
be bit-identical to the unscheduled call (which the decode tests gate against
the oracle); the cheap configurations are gated against the oracle here too.
"""
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402
from oracle import compare, decode_workload  # noqa: E402
from workloads import logical_case, page_case  # noqa: E402

DEV = "cuda:0"


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_bench_launch_configurations(k, stage_batches):
    """Each workload in the launch configuration bench.py times (partition
    sizes, shared-prefix cascade with request groups, work list): every
    output against the oracle."""
    w = stage_batches.workload(k)
    S, kw = bench.launch_configuration(k, w)
    say(f"bench launch configuration {k} {w.name}: S={S} {sorted(kw)}")
    out = outputs(w, S, items=True, **kw)
    rep = compare(out, stage_batches.reference(k)[0])
    say(f"bench configuration {k} vs oracle, all {w.batch} sequences: {rep}")
    assert rep.passed


def outputs(w, S=None, items=None, **kw):
    """Output bits of one step; ``items``: True = the library's list, an array = that list."""
    from paper_2510_14126_amd.device import PagedBatch
    pb = PagedBatch(w, DEV, partition_size=S, schedule=items is True, **kw)
    if items is not None and items is not True:
        pb.set_items(items)
    pb.run()
    torch.cuda.synchronize()
    out = pb.out_bits()
    pb.close()
    return out


def assert_same(a, b, what):
    diff = int(np.count_nonzero(a != b))
    say(f"{what}: {diff} differing outputs of {a.size}")
    assert diff == 0, f"{what}: {diff} outputs differ"


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_scheduled_configs_bit_identical(k, stage_batches):
    w = stage_batches.workload(k)
    say(f"scheduled config {k} {w.name}")
    plain = outputs(w)
    sched = outputs(w, items=True)
    assert_same(sched, plain, f"config {k}")
    rep = compare(sched, stage_batches.reference(k)[0])
    say(f"config {k} vs oracle: {rep}")
    assert rep.passed


@pytest.mark.parametrize("k", [2, 3])
def test_scheduled_cascade_configs_bit_identical(k, stage_batches):
    w = stage_batches.workload(k)
    L = w.meta["prefix_blocks"] * 16
    say(f"scheduled cascade config {k}: prefix {L}")
    kw = dict(prefix_len=L, prefix_partition_size=256)
    assert_same(outputs(w, items=True, **kw), outputs(w, **kw), f"cascade config {k}")


def test_scheduled_long_context_bit_identical(stage_batches):
    w = stage_batches.workload(5)
    say("scheduled config 5")
    L = w.meta["prefix_blocks"] * 16
    plain = outputs(w, 512)
    assert_same(outputs(w, 512, items=True), plain, "config 5")
    kw = dict(prefix_len=L, prefix_partition_size=512)
    casc = outputs(w, 512, items=True, **kw)
    assert_same(casc, outputs(w, 512, **kw), "cascade config 5")
    rep = compare(casc, stage_batches.reference(5)[0])
    say(f"scheduled cascade config 5 vs oracle, all sequences: {rep}")
    assert rep.passed


EDGE = [
    # seed, B, Hq, Hkv, ctx, S (0 = one partition)
    (40, 7, 32, 8, [0, 1, 16, 17, 300, 0, 513], 128),
    (41, 5, 32, 8, [0, 1, 15, 16, 200], 0),
    (42, 4, 64, 8, [2049, 0, 31, 1024], 512),
    (43, 9, 16, 2, [5 * i for i in range(9)], 16),
    (44, 3, 8, 1, [0, 0, 0], 64),
]


@pytest.mark.parametrize("case", EDGE, ids=[f"seed{c[0]}" for c in EDGE])
def test_scheduled_edge_shapes(case):
    seed, B, hq, hkv, ctx, S = case
    say(f"scheduled edges seed={seed} B={B} Hq={hq} Hkv={hkv} S={S}")
    w = page_case(logical_case(seed, B, hq, hkv, 128, ctx), seed + 1, extra_blocks=4,
                  poison=True)
    sched = outputs(w, S, items=True)
    assert_same(sched, outputs(w, S), f"edges seed {seed}")
    rep = compare(sched, decode_workload(w)[0])
    say(f"edges seed {seed} vs oracle: {rep}")
    assert rep.passed


def test_any_item_order_gives_the_same_bits():
    """The list's order is free: a shuffled list and the grid order agree."""
    w = page_case(logical_case(50, 12, 32, 8, 128, [100 * i + 7 for i in range(12)]), 51)
    from paper_2510_14126_amd import binding
    S = 256
    items = binding.paged_attn_schedule(w.context_lens, w.max_context_len, S)
    rng = np.random.default_rng(52)
    ref = outputs(w, S)
    for order in (rng.permutation(items), np.sort(items)):
        assert_same(outputs(w, S, items=order), ref, "shuffled list")


def test_scheduled_cascade_edges():
    say("scheduled cascade: sequences shorter than and equal to the prefix")
    lc = logical_case(60, 5, 32, 8, 128, [700, 520, 900, 512, 1300], prefix_len=512)
    w = page_case(lc, 61, poison=True)
    w.context_lens = w.context_lens.copy()
    w.context_lens[1] = 492
    w.context_lens[3] = 0
    kw = dict(prefix_len=512, prefix_partition_size=128)
    sched = outputs(w, 256, items=True, **kw)
    assert_same(sched, outputs(w, 256, **kw), "cascade edges")
    rep = compare(sched, decode_workload(w)[0])
    say(f"cascade edges vs oracle: {rep}")
    assert rep.passed
