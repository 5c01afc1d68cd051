"""Index traces of the launches the benchmark times, checked bit for bit.

Block-table and context-length handling must be exact.  The trace entry
points run the production gather code and record, per work item, every KV
tile it loaded as (logical block, physical id read from the table, valid
rows).  The expected lists are computed here on the host from the tables and
lengths alone: the shared-prefix partitions read every sequence's prefix
through row 0, a group's shared tokens through its first row, and every
per-sequence partition its own tokens after the shared ones.  Slots that no
tile fills must keep the fill value.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import bench  # noqa: E402
from oracle import compare  # noqa: E402
from workloads import grouped_case, logical_case, page_case  # noqa: E402

DEV = "cuda:0"
FILL = -7


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


def expected_cascade(w, S, L, pps, lay, group_start=None, M=0, items=None):
    """Host-side trace of a cascade step (int32 array of lay['total'] values)."""
    hkv, G = w.num_kv_heads, w.num_q_heads // w.num_kv_heads
    bt, ctx = w.block_tables, w.context_lens.astype(np.int64)
    exp = np.full(lay["total"], FILL, dtype=np.int64)
    # prefix partitions: every row group reads the partition's blocks via row 0
    pre_parts = -(-L // pps) if L else 0
    row_groups = -(-(w.batch * G) // 64)
    pt = lay["prefix_tiles"]
    for p in range(pre_parts):
        s0, e0 = p * pps, min(L, (p + 1) * pps)
        tiles = [(j, int(bt[0, j]), min(16, e0 - 16 * j)) for j in range(s0 // 16, -(-e0 // 16))]
        for rg in range(row_groups):
            for g in range(hkv):
                base = lay["prefix_offset"] + ((p * row_groups + rg) * hkv + g) * pt * 3
                for i, t in enumerate(tiles):
                    exp[base + 3 * i: base + 3 * i + 3] = t
    # groups: each non-empty group reads its shared tokens via its first row
    if M:
        gt = lay["group_tiles"]
        for k in range(len(group_start) - 1):
            a, b = int(group_start[k]), int(group_start[k + 1])
            if b <= a:
                continue
            tiles = [(j, int(bt[a, j]), 16) for j in range(L // 16, (L + M) // 16)]
            for g in range(hkv):
                base = lay["group_offset"] + (k * hkv + g) * gt * 3
                for i, t in enumerate(tiles):
                    exp[base + 3 * i: base + 3 * i + 3] = t
    # per-sequence partitions after the shared tokens (those listed, if a list)
    first = L + M
    parts = -(-(int(ctx.max()) - first) // S) if int(ctx.max()) > first else 0
    listed = None if items is None else set(int(i) for i in items)
    dt = lay["decode_tiles"]
    for p in range(parts):
        for b in range(w.batch):
            if listed is not None and p * w.batch + b not in listed:
                continue
            n = int(ctx[b])
            lo, hi = first + p * S, min(n, first + (p + 1) * S)
            if hi <= lo:
                continue
            tiles = [(j, int(bt[b, j]), min(16, n - 16 * j)) for j in range(lo // 16, -(-hi // 16))]
            for g in range(hkv):
                base = lay["decode_offset"] + ((p * w.batch + b) * hkv + g) * dt * 3
                for i, t in enumerate(tiles):
                    exp[base + 3 * i: base + 3 * i + 3] = t
    return exp.astype(np.int32)


def cascade_trace(pb, lay, group_len=0):
    from paper_2510_14126_amd import binding
    tr = torch.full((lay["total"],), FILL, dtype=torch.int32, device=DEV)
    n = 0 if pb.items is None else int(pb.items.numel())
    binding.paged_attn_decode_cascade_trace(
        pb.pool, pb.q, pb.bt, pb.bt_stride, pb.ctx, pb.batch, pb.hq, pb.w.scale, pb.max_ctx,
        pb.partition_size, pb.prefix_len, pb.prefix_partition_size,
        pb.group_start if group_len else None, pb.num_groups if group_len else 0,
        pb.max_group_size if group_len else 0, group_len, pb.items if n else None, n,
        pb.part_o, pb.part_lse, tr, lay["total"])
    torch.cuda.synchronize()
    return tr.cpu().numpy()


def check_cascade(w, S, L, pps, group_start=None, M=0, schedule=False, what=""):
    from paper_2510_14126_amd import binding
    from paper_2510_14126_amd.device import PagedBatch
    kw = dict(group_start=group_start, group_len=M) if M else {}
    pb = PagedBatch(w, DEV, partition_size=S, prefix_len=L, prefix_partition_size=pps,
                    schedule=schedule, **kw)
    lay = binding.paged_attn_cascade_trace_layout(pb.pool, w.batch, w.num_q_heads, pb.max_ctx, S, L,
                                                  pps, pb.num_groups if M else 0, M)
    got = cascade_trace(pb, lay, M)
    items = None if pb.items is None else pb.items.cpu().numpy()
    exp = expected_cascade(w, S, L, pps, lay, group_start, M, items)
    bad = np.flatnonzero(got != exp)
    say(f"{what}: {lay['total'] // 3} trace slots, {bad.size} differ")
    assert bad.size == 0, f"{what}: first differing value {bad[0]}: got {got[bad[0]]} want {exp[bad[0]]}"
    # the trace launch is the production launch: its partials merge to the output
    pb.reduce()
    torch.cuda.synchronize()
    out = pb.out_bits()
    pb.close()
    return out


@pytest.mark.parametrize("schedule", [False, True], ids=["grid", "work_list"])
@pytest.mark.parametrize("hq", [32, 64])
def test_cascade_trace_edges(hq, schedule):
    """Short sequences (inside the prefix, at its end, empty), ragged tails."""
    say(f"cascade trace edges Hq={hq} schedule={schedule}")
    lc = logical_case(110, 6, hq, 8, 128, [700, 520, 900, 512, 1300, 515], prefix_len=512)
    w = page_case(lc, 111, poison=True)
    w.context_lens = w.context_lens.copy()
    w.context_lens[1] = 492
    w.context_lens[3] = 0
    out = check_cascade(w, 256, 512, 128, schedule=schedule, what=f"cascade edges Hq={hq}")
    from oracle import decode_workload
    assert compare(out, decode_workload(w)[0]).passed


@pytest.mark.parametrize("hq", [32, 64])
def test_grouped_cascade_trace(hq):
    say(f"grouped cascade trace Hq={hq}")
    sizes = [3, 1, 2, 4] if hq == 32 else [3, 1, 2]
    suffix = list(np.random.default_rng(120).integers(1, 400, sum(sizes)))
    w = grouped_case(121, hq, 8, 128, 256, sizes, 128, suffix)
    gs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    out = check_cascade(w, 128, 256, 128, group_start=gs, M=128, schedule=True,
                        what=f"grouped cascade Hq={hq}")
    from oracle import decode_workload
    assert compare(out, decode_workload(w)[0]).passed


@pytest.mark.parametrize("k", [2, 3, 5])
def test_bench_launch_configuration_traces(k, stage_batches):
    """The exact launches bench.py times on the stage batches with a shared
    prefix (cascade, request groups, work list), traced in full."""
    w = stage_batches.workload(k)
    S, kw = bench.launch_configuration(k, w)
    L, pps = kw["prefix_len"], kw["prefix_partition_size"]
    say(f"bench launch trace config {k} {w.name}: S={S} prefix={L}/{pps} groups={'group_len' in kw}")
    out = check_cascade(w, S, L, pps, kw.get("group_start"), kw.get("group_len", 0), schedule=True,
                        what=f"bench configuration {k}")
    assert compare(out, stage_batches.reference(k)[0]).passed


@pytest.mark.parametrize("hq", [32, 64])
def test_scheduled_decode_trace(hq):
    from paper_2510_14126_amd import binding
    from paper_2510_14126_amd.device import PagedBatch
    say(f"scheduled decode trace Hq={hq}")
    lc = logical_case(130, 7, hq, 8, 128, [0, 1, 16, 17, 300, 1025, 513])
    w = page_case(lc, 131, poison=True)
    S = 128
    pb = PagedBatch(w, DEV, partition_size=S, schedule=True)
    P = pb.num_parts
    tiles = S // 16
    total = P * w.batch * w.num_kv_heads * tiles * 3
    tr = torch.full((total,), FILL, dtype=torch.int32, device=DEV)
    n = int(pb.items.numel())
    binding.paged_attn_decode_scheduled_trace(pb.pool, pb.q, pb.bt, pb.bt_stride, pb.ctx, pb.batch,
                                              pb.hq, w.scale, pb.max_ctx, S, pb.items, n, pb.out,
                                              pb.part_o, pb.part_lse, tr, total)
    torch.cuda.synchronize()
    got = tr.cpu().numpy()
    exp = np.full(total, FILL, dtype=np.int64)
    for p in range(P):
        for b in range(w.batch):
            ctx = int(w.context_lens[b])
            lo, hi = p * S, min(ctx, (p + 1) * S)
            if hi <= lo:
                continue
            for g in range(w.num_kv_heads):
                base = ((p * w.batch + b) * w.num_kv_heads + g) * tiles * 3
                for i, j in enumerate(range(lo // 16, -(-hi // 16))):
                    exp[base + 3 * i: base + 3 * i + 3] = (j, w.block_tables[b, j], min(16, ctx - 16 * j))
    bad = np.flatnonzero(got != exp)
    say(f"scheduled decode trace: {bad.size} differing values of {total}")
    assert bad.size == 0
    pb.reduce()
    torch.cuda.synchronize()
    from oracle import decode_workload
    assert compare(pb.out_bits(), decode_workload(w)[0]).passed
    pb.close()
