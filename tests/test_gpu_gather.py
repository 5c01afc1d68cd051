"""GPU tests of the data-movement helper (pa_gather_tiles): every wavefront's
XOR of the words it read equals the same XOR taken on the host from the pool
arrays, bit for bit."""
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402
from workloads import build_config, group_starts, logical_case, page_case  # noqa: E402

DEV = "cuda:0"


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


def expected_sink(w, spans):
    """XOR of every 32-bit word of the K and V tiles wavefront w reads."""
    hkv = w.num_kv_heads
    tk = np.bitwise_xor.reduce(w.k_pool.view(np.uint32).reshape(w.num_blocks, hkv, -1), axis=2)
    tv = np.bitwise_xor.reduce(w.v_pool.view(np.uint32).reshape(w.num_blocks, hkv, -1), axis=2)
    t = tk ^ tv
    row_tokens = 16 * w.block_tables.shape[1]
    out = np.zeros((len(spans), hkv, 4), np.uint32)
    for i, (b, s, e) in enumerate(spans):
        b = min(max(int(b), 0), w.batch - 1)
        s = min(max(int(s), 0), row_tokens) & ~15
        e = min(max(int(e), s), row_tokens)
        ids = w.block_tables[b, s // 16:(e + 15) // 16]
        ids = np.clip(ids, 0, w.num_blocks - 1)
        for j, blk in enumerate(ids):
            out[i, :, j % 4] ^= t[blk]
    return out


def run(w, spans, S=256, tiles_in_flight=2):
    from paper_2510_14126_amd.device import PagedBatch
    pb = PagedBatch(w, DEV, partition_size=S)
    spans = np.ascontiguousarray(spans, dtype=np.int32).reshape(-1, 3)
    sd = torch.from_numpy(spans).to(DEV)
    sink = torch.full((max(1, spans.shape[0] * w.num_kv_heads * 4),), -1, dtype=torch.int32, device=DEV)
    pb.gather_tiles(sd, spans.shape[0], sink, tiles_in_flight=tiles_in_flight)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)[: spans.shape[0] * w.num_kv_heads * 4]
    pb.close()
    return got.reshape(-1, w.num_kv_heads, 4)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_bench_spans_match_host_xor(k):
    w = build_config(k)
    L = 16 * int(w.meta.get("prefix_blocks", 0))
    from paper_2510_14126_amd.device import PagedBatch
    kw = {}
    if L:
        kw = dict(prefix_len=L, prefix_partition_size=bench.default_prefix_partition(k, L))
    if L and "groups" in w.meta and w.meta.get("mid_blocks", 0):
        kw.update(group_start=group_starts(w), group_len=16 * int(w.meta["mid_blocks"]))
    pb = PagedBatch(w, DEV, partition_size=bench.DEFAULT_PARTITION[k], **kw)
    spans = pb.tile_spans()
    pb.close()
    say(f"gather tiles config {k}: {len(spans)} spans")
    ref = expected_sink(w, spans)
    for nif in (2, 4):
        assert np.array_equal(run(w, spans, tiles_in_flight=nif), ref), nif


def test_head_dim_64_and_clamped_spans():
    """D = 64 tiles, empty spans, a start inside a block, and spans whose
    sequence and tokens lie outside the table (clamped, as documented)."""
    w = page_case(logical_case(30, 6, 16, 4, 64, [0, 1, 17, 100, 513, 260]), 31, extra_blocks=3)
    row = 16 * w.block_tables.shape[1]
    spans = [[0, 0, 0], [1, 0, 1], [2, 5, 17], [3, 16, 100], [4, 0, 513], [5, 250, 260],
             [9, 0, 40], [-3, 0, 40], [4, -20, row + 500], [4, 600, 10]]
    say(f"gather tiles D=64 with clamped spans, table row {row} tokens")
    ref = expected_sink(w, spans)
    for nif in (2, 4):
        assert np.array_equal(run(w, spans, tiles_in_flight=nif), ref), nif
