"""GPU tests of the two-level cascade (prefix, then per group of sequences).

Every output is gated against the fp64 oracle, which knows nothing of the
sharing: it gathers each sequence's own context through its own table.
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
from oracle.attention import bf16_to_f64  # noqa: E402
from workloads import build_config, group_starts, grouped_case  # noqa: E402

DEV = "cuda:0"


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


def outputs(w, S, prefix_len, pps, group_len=0, schedule=False, starts=None):
    from paper_2510_14126_amd.device import PagedBatch
    kw = {}
    if group_len:
        kw = dict(group_start=group_starts(w) if starts is None else starts, group_len=group_len)
    pb = PagedBatch(w, DEV, partition_size=S, prefix_len=prefix_len, prefix_partition_size=pps,
                    schedule=schedule, **kw)
    pb.out.fill_(0x7FC0)                       # NaN bits: every row must be written
    pb.run()
    torch.cuda.synchronize()
    out = pb.out_bits()
    pb.close()
    return out


def gate(out, w, what, seqs=None):
    ref = decode_workload(w, seqs=seqs)[0]
    rep = compare(out if seqs is None else out[seqs], ref)
    say(f"{what}: {rep}")
    assert rep.passed, f"{what}: {rep}"


@pytest.mark.parametrize("schedule", [False, True])
def test_fixer_batch_grouped(schedule):
    """The fixer batch with its requests as groups (their first attempts
    shared), in the bench launch configuration, against the oracle; the
    scheduled and full-grid launches give the same bits."""
    w = build_config(3)
    L = 16 * w.meta["prefix_blocks"]
    M = 16 * w.meta["mid_blocks"]
    S = bench.DEFAULT_PARTITION[3]
    pps = bench.default_prefix_partition(3, L)
    say(f"fixer grouped: prefix {L}, group {M}, S={S}, schedule={schedule}")
    out = outputs(w, S, L, pps, M, schedule)
    gate(out, w, "fixer grouped")
    if schedule:
        assert np.array_equal(out, outputs(w, S, L, pps, M, False)), "work list changed bits"
    plain = outputs(w, S, L, pps)
    assert compare(out, bf16_to_f64(plain), gpu_is_bf16_bits=True).passed


CASES = [
    # seed, Hq, Hkv, prefix, group sizes, group tokens, S, S_pre
    (5, 32, 8, 256, [1, 3, 2, 5, 4], 64, 128, 128),
    (6, 64, 8, 512, [2, 8, 1], 128, 256, 256),        # GQA 8: 8 sequences x 8 heads = 64 rows
    (7, 32, 8, 0, [4, 4, 1, 16], 256, 512, 64),       # no batch-wide prefix; 16 x 4 = 64 rows
    (8, 16, 4, 128, [1] * 6, 16, 64, 32),             # groups of one, one block shared
    (9, 32, 8, 64, [3, 2], 1024, 1024, 64),           # the largest group span
]


@pytest.mark.parametrize("case", CASES, ids=[f"seed{c[0]}" for c in CASES])
def test_grouped_shapes(case):
    seed, hq, hkv, L, sizes, M, S, pps = case
    rng = np.random.default_rng(seed)
    suffix = rng.integers(0, 400, size=sum(sizes))
    w = grouped_case(seed, hq, hkv, 128, L, sizes, M, suffix)
    say(f"grouped seed={seed} Hq={hq} Hkv={hkv} prefix={L} groups={sizes} M={M} S={S}")
    for schedule in (False, True):
        gate(outputs(w, S, L, pps, M, schedule), w, f"grouped seed {seed} schedule={schedule}")


def test_members_shorter_than_the_shared_parts():
    """Members that end inside the group's tokens or inside the prefix (the
    group's first sequence holds all of them) attend only to their own
    context; an empty sequence gives zeros."""
    w = grouped_case(20, 32, 8, 128, 256, [4, 3], 128, [100, 50, 0, 7, 30, 200, 1])
    w.context_lens = w.context_lens.copy()
    w.context_lens[1] = 256 + 20          # inside the group's tokens
    w.context_lens[2] = 200               # inside the prefix
    w.context_lens[3] = 0                 # empty
    w.context_lens[5] = 256 + 128         # exactly the shared parts
    say("grouped members shorter than the shared parts")
    out = outputs(w, 128, 256, 64, 128, True)
    gate(out, w, "short members")
    assert np.all(out[3] & 0x7FFF == 0)
