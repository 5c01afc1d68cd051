"""Host-side tests of the C ABI: exports, allocator and argument validation.

No kernel is launched here: every call either manipulates host metadata or
fails validation before any HIP call, so these run without a GPU.
"""
import ctypes
import os
import re

import numpy as np

import pytest

from paper_2510_14126_amd import binding as pa

HERE = os.path.dirname(os.path.abspath(__file__))
HEADER = os.path.join(HERE, "..", "include", "paged_attn.h")
FAKE_K, FAKE_V = 0x10000, 0x20000     # aligned placeholder device addresses (never dereferenced)


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_][a-z_0-9]*)\s*\(",
                                 src, flags=re.M)))


def test_header_and_library_agree():
    names = declared_functions()
    assert len(names) == 37, names
    lib = pa.library()
    for n in names:
        assert hasattr(lib, n), f"library does not export {n}"
    assert set(names) == set(pa.SIGNATURES)
    assert pa.pa_version() >= 100


def make_pool(nb=10, hkv=8, d=128):
    return pa.kv_pool_create(nb, 16, hkv, d, FAKE_K, FAKE_V)


def test_pool_create_validation():
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_create(10, 32, 8, 128, FAKE_K, FAKE_V)
    assert e.value.code == pa.PA_EINVAL
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_create(10, 16, 8, 96, FAKE_K, FAKE_V)
    assert e.value.code == pa.PA_EUNSUPPORTED
    for bad in [(0, 16, 8, 128, FAKE_K, FAKE_V), (10, 16, 0, 128, FAKE_K, FAKE_V),
                (10, 16, 8, 128, 0, FAKE_V), (10, 16, 8, 128, FAKE_K + 2, FAKE_V)]:
        with pytest.raises(pa.PagedAttnError) as e:
            pa.kv_pool_create(*bad)
        assert e.value.code == pa.PA_EINVAL
    assert "kv_pool_create" in pa.pa_last_error()


def test_pool_layout():
    p = make_pool(nb=7, hkv=8, d=128)
    strides, nbytes = pa.kv_pool_layout(p)
    assert strides == [8 * 16 * 128, 16 * 128, 128, 1]
    assert nbytes == 7 * 8 * 16 * 128 * 2


def test_alloc_release_and_exhaustion():
    p = make_pool(nb=10)
    assert pa.kv_pool_num_free(p) == 10
    a = pa.kv_pool_alloc(p, 4)
    assert a == [0, 1, 2, 3] and pa.kv_pool_num_free(p) == 6
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_alloc(p, 7)
    assert e.value.code == pa.PA_ENOMEM and pa.kv_pool_num_free(p) == 6   # unchanged
    b = pa.kv_pool_alloc(p, 6)
    assert sorted(a + b) == list(range(10)) and pa.kv_pool_num_free(p) == 0
    pa.kv_pool_release(p, [2, 5])
    assert pa.kv_pool_num_free(p) == 2 and pa.kv_pool_refcount(p, 2) == 0
    assert sorted(pa.kv_pool_alloc(p, 2)) == [2, 5]


def test_shared_prefix_refcounts():
    p = make_pool(nb=8)
    prefix = pa.kv_pool_alloc(p, 3)
    pa.kv_pool_retain(p, prefix)          # a second sequence maps the prefix
    pa.kv_pool_retain(p, prefix)          # and a third
    assert [pa.kv_pool_refcount(p, i) for i in prefix] == [3, 3, 3]
    assert pa.kv_pool_num_shared(p) == 3
    pa.kv_pool_release(p, prefix)
    assert pa.kv_pool_num_shared(p) == 3
    pa.kv_pool_release(p, prefix)
    assert pa.kv_pool_num_free(p) == 5    # still held by the first sequence
    assert pa.kv_pool_num_shared(p) == 0
    pa.kv_pool_release(p, prefix)
    assert pa.kv_pool_num_free(p) == 8


def test_shared_block_count_follows_every_change():
    # Randomised retain/release sequences (repeated ids in one call included)
    # against a host model of the reference counts.
    import random
    rng = random.Random(7)
    p = make_pool(nb=12)
    ids = pa.kv_pool_alloc(p, 12)
    model = {i: 1 for i in ids}
    for _ in range(300):
        pick = [rng.choice(ids) for _ in range(rng.randint(1, 4))]
        if rng.random() < 0.55:
            if all(model[i] > 0 for i in pick):
                pa.kv_pool_retain(p, pick)
                for i in pick:
                    model[i] += 1
        else:
            need = {i: pick.count(i) for i in pick}
            if all(model[i] >= c for i, c in need.items()):
                pa.kv_pool_release(p, pick)
                for i in pick:
                    model[i] -= 1
            else:
                with pytest.raises(pa.PagedAttnError):
                    pa.kv_pool_release(p, pick)
        assert pa.kv_pool_num_shared(p) == sum(1 for c in model.values() if c >= 2)
        assert [pa.kv_pool_refcount(p, i) for i in ids] == [model[i] for i in ids]


def test_state_violations_change_nothing():
    p = make_pool(nb=6)
    ids = pa.kv_pool_alloc(p, 2)
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_release(p, [ids[0], ids[0]])   # double release in one call
    assert e.value.code == pa.PA_ESTATE and pa.kv_pool_refcount(p, ids[0]) == 1
    pa.kv_pool_release(p, [ids[0]])
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_release(p, [ids[0]])           # release of a free block
    assert e.value.code == pa.PA_ESTATE
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_retain(p, [ids[1], ids[0]])    # retain of a free block
    assert e.value.code == pa.PA_ESTATE and pa.kv_pool_refcount(p, ids[1]) == 1
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_release(p, [99])
    assert e.value.code == pa.PA_EINVAL


def test_claim_specific_blocks():
    p = make_pool(nb=6)
    pa.kv_pool_claim(p, [4, 1])
    assert pa.kv_pool_num_free(p) == 4
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_claim(p, [0, 4])
    assert e.value.code == pa.PA_ESTATE and pa.kv_pool_refcount(p, 0) == 0
    with pytest.raises(pa.PagedAttnError) as e:
        pa.kv_pool_claim(p, [2, 2])
    assert e.value.code == pa.PA_ESTATE
    assert pa.kv_pool_alloc(p, 4) == [0, 2, 3, 5]


def test_partition_planning():
    assert pa.paged_attn_num_partitions(0, 512) == 1
    assert pa.paged_attn_num_partitions(512, 512) == 1
    assert pa.paged_attn_num_partitions(513, 512) == 2
    assert pa.paged_attn_num_partitions(32768, 512) == 64
    assert pa.paged_attn_num_partitions(32768, 0) == 1
    assert pa.paged_attn_workspace_size(4, 8, 64, 300, 512) == (0, 0)
    assert pa.paged_attn_workspace_size(128, 64, 128, 32768, 512) == (128 * 64 * 64 * 128 * 4,
                                                                      128 * 64 * 64 * 4)
    with pytest.raises(pa.PagedAttnError):
        pa.paged_attn_num_partitions(100, 24)


def _decode(pool, **over):
    args = dict(q=0x1000, block_tables=0x2000, bt_stride=4, context_lens=0x3000, batch=2,
                num_q_heads=32, scale=0.088, max_context_len=64, partition_size=0, out=0x4000,
                partial_out=None, partial_lse=None)
    args.update(over)
    pa.paged_attn_decode(pool, **args)


@pytest.mark.parametrize("over,code", [
    (dict(num_q_heads=24), pa.PA_EUNSUPPORTED),        # G = 3
    (dict(num_q_heads=30), pa.PA_EINVAL),              # not a multiple of Hkv
    (dict(batch=-1), pa.PA_EINVAL),
    (dict(max_context_len=-5), pa.PA_EINVAL),
    (dict(partition_size=20), pa.PA_EINVAL),
    (dict(bt_stride=3), pa.PA_EINVAL),                 # ceil(64/16) = 4 needed
    (dict(q=0x1008), pa.PA_EINVAL),                    # misaligned q
    (dict(q=None), pa.PA_EINVAL),
    (dict(out=None), pa.PA_EINVAL),                    # single partition needs out
    (dict(max_context_len=1024, bt_stride=64, partition_size=512), pa.PA_EINVAL),  # no partials
    (dict(scale=float("nan")), pa.PA_EINVAL),
])
def test_decode_validation(over, code):
    p = make_pool()
    with pytest.raises(pa.PagedAttnError) as e:
        _decode(p, **over)
    assert e.value.code == code, pa.pa_last_error()


@pytest.mark.parametrize("over,code", [
    (dict(k_new=None), pa.PA_EINVAL),
    (dict(v_new=None), pa.PA_EINVAL),
    (dict(k_new=0x5008), pa.PA_EINVAL),                # misaligned
    (dict(v_new=0x6004), pa.PA_EINVAL),
    (dict(num_q_heads=24), pa.PA_EUNSUPPORTED),
    (dict(items=0x7000, num_items=-1), pa.PA_EINVAL),
])
def test_fused_append_validation(over, code):
    """Argument checks of the fused append + decode entry points, before any
    HIP call (fake device addresses)."""
    p = make_pool()
    args = dict(q=0x1000, k_new=0x5000, v_new=0x6000, block_tables=0x2000, bt_stride=4,
                context_lens=0x3000, batch=2, num_q_heads=32, scale=0.088, max_context_len=64,
                partition_size=0, items=None, num_items=0, out=0x4000, partial_out=None,
                partial_lse=None)
    args.update(over)
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_decode_append(p, **args)
    assert e.value.code == code, pa.pa_last_error()
    cargs = dict(q=0x1000, k_new=0x5000, v_new=0x6000, block_tables=0x2000, bt_stride=4,
                 context_lens=0x3000, batch=2, num_q_heads=32, scale=0.088, max_context_len=64,
                 partition_size=32, prefix_len=16, prefix_partition_size=16, group_start=None,
                 num_groups=0, max_group_size=0, group_len=0, items=None, num_items=0,
                 partial_out=0x8000, partial_lse=0x9000)
    cargs.update({k: v for k, v in over.items() if k in cargs})
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_decode_cascade_append(p, **cargs)
    assert e.value.code == code, pa.pa_last_error()


def test_empty_batch_is_a_no_op():
    p = make_pool()
    _decode(p, batch=0, q=None, block_tables=None, context_lens=None, out=None)


@pytest.mark.parametrize("over,code", [
    (dict(head_dim=96), pa.PA_EUNSUPPORTED),
    (dict(partition_size=0), pa.PA_EINVAL),
    (dict(max_partitions=0), pa.PA_EINVAL),
    (dict(out=None), pa.PA_EINVAL),
])
def test_reduce_validation(over, code):
    args = dict(partial_out=0x1000, partial_lse=0x2000, context_lens=0x3000, batch=2,
                num_q_heads=8, head_dim=128, partition_size=512, max_partitions=3, out=0x4000)
    args.update(over)
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_reduce(**args)
    assert e.value.code == code


def test_trace_capacity_checked():
    p = make_pool()
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_decode_trace(p, 0x1000, 0x2000, 4, 0x3000, 2, 32, 0.1, 64, 0, 0x4000, None,
                                   None, 0x5000, 10)
    assert e.value.code == pa.PA_EINVAL and "trace_capacity" in pa.pa_last_error()


def test_stream_copy_validation():
    with pytest.raises(pa.PagedAttnError):
        pa.pa_stream_copy(0x1000, 0x2000, 17)


def test_gather_tiles_validation():
    """Host checks of the data-movement helper; no span is ever launched."""
    p = make_pool()
    ok = dict(block_tables=0x50000, bt_stride=4, batch=2, spans=0x60000, num_spans=3, sink=0x70000)
    cases = [(dict(num_spans=-1), "num_spans"), (dict(block_tables=0), "NULL"),
             (dict(spans=0), "NULL"), (dict(sink=0), "NULL"), (dict(spans=0x60002), "aligned"),
             (dict(batch=0), "batch"), (dict(bt_stride=0), "bt_stride"),
             (dict(bt_stride=1 << 27), "2^31 tokens"),
             (dict(num_spans=1 << 28), "grid"), (dict(tiles_in_flight=3), "tiles_in_flight"),
             (dict(tiles_in_flight=0, num_spans=0), "tiles_in_flight")]
    for over, msg in cases:
        a = {**ok, **over}
        with pytest.raises(pa.PagedAttnError) as e:
            pa.pa_gather_tiles(p, **a)
        assert e.value.code == pa.PA_EINVAL and msg in pa.pa_last_error(), (over, pa.pa_last_error())
    with pytest.raises(pa.PagedAttnError):
        pa.pa_gather_tiles(None, **ok)
    pa.pa_gather_tiles(p, **{**ok, "num_spans": 0, "sink": 0})     # empty: no-op, no launch


# --------------------------------------------------------------- KV append

def _append(pool, **over):
    a = dict(k_new=0x30000, v_new=0x40000, block_tables=0x50000, bt_stride=4, context_lens=0x60000,
             batch=2)
    a.update(over)
    pa.paged_attn_append_kv(pool, a["k_new"], a["v_new"], a["block_tables"], a["bt_stride"],
                            a["context_lens"], a["batch"])


@pytest.mark.parametrize("over,code", [
    (dict(batch=-1), pa.PA_EINVAL),
    (dict(bt_stride=0), pa.PA_EINVAL),
    (dict(bt_stride=1 << 28), pa.PA_EINVAL),
    (dict(k_new=0), pa.PA_EINVAL),
    (dict(v_new=0), pa.PA_EINVAL),
    (dict(block_tables=0), pa.PA_EINVAL),
    (dict(context_lens=0), pa.PA_EINVAL),
    (dict(k_new=0x30008), pa.PA_EINVAL),       # not 16-byte aligned
    (dict(context_lens=0x60002), pa.PA_EINVAL),
])
def test_append_validation(over, code):
    p = make_pool()
    with pytest.raises(pa.PagedAttnError) as e:
        _append(p, **over)
    assert e.value.code == code, pa.pa_last_error()
    assert "paged_attn_append_kv" in pa.pa_last_error()


def test_append_empty_batch_is_a_no_op():
    p = make_pool()
    _append(p, batch=0, k_new=0, v_new=0, block_tables=0, context_lens=0)


# --------------------------------------------------------------- extend

def _extend(pool, **over):
    a = dict(q=0x30000, q_start=0x70000, total_q=64, block_tables=0x50000, bt_stride=8,
             context_lens=0x60000, batch=2, num_q_heads=32, scale=0.088, max_context_len=128,
             max_chunk=64, out=0x80000)
    a.update(over)
    pa.paged_attn_extend(pool, a["q"], a["q_start"], a["total_q"], a["block_tables"], a["bt_stride"],
                         a["context_lens"], a["batch"], a["num_q_heads"], a["scale"],
                         a["max_context_len"], a["max_chunk"], a["out"])


@pytest.mark.parametrize("over,code", [
    (dict(batch=-1), pa.PA_EINVAL),
    (dict(total_q=-1), pa.PA_EINVAL),
    (dict(max_chunk=-1), pa.PA_EINVAL),
    (dict(max_chunk=129), pa.PA_EINVAL),           # longer than the context bound
    (dict(max_context_len=8208, bt_stride=513), pa.PA_EUNSUPPORTED),
    (dict(bt_stride=7), pa.PA_EINVAL),
    (dict(num_q_heads=16), pa.PA_EUNSUPPORTED),     # G = 2
    (dict(q_start=0), pa.PA_EINVAL),
    (dict(out=0), pa.PA_EINVAL),
    (dict(out=0x80008), pa.PA_EINVAL),
    (dict(q=0x30004), pa.PA_EINVAL),
    (dict(scale=float("nan")), pa.PA_EINVAL),
])
def test_extend_validation(over, code):
    p = make_pool()
    with pytest.raises(pa.PagedAttnError) as e:
        _extend(p, **over)
    assert e.value.code == code, pa.pa_last_error()
    assert "paged_attn_extend" in pa.pa_last_error()


def test_extend_needs_head_dim_128():
    p = make_pool(d=64)
    with pytest.raises(pa.PagedAttnError) as e:
        _extend(p)
    assert e.value.code == pa.PA_EUNSUPPORTED


def test_extend_empty_is_a_no_op():
    p = make_pool()
    _extend(p, batch=0, q=0, q_start=0, block_tables=0, context_lens=0, out=0)
    _extend(p, total_q=0, q_start=0, out=0)
    _extend(p, max_chunk=0, q_start=0, out=0)


# --------------------------------------------------------------- work lists

def _brute_items(ctx, max_ctx, S, prefix):
    """Every (partition, sequence) item that holds tokens, by brute force.

    The partitioning is the decode call's own (paged_attn_num_partitions) or,
    with a prefix, S-token partitions after it."""
    if prefix == 0:
        parts = pa.paged_attn_num_partitions(max_ctx, S)
        size = S if parts > 1 else max_ctx + 16
    else:
        parts, size = -(-(max_ctx - prefix) // S), S
    keep_empty = prefix == 0 and parts == 1
    B = len(ctx)
    pairs = [(b, part) for b in range(B) for part in range(parts)] if parts >= 16 else \
        [(b, part) for part in range(parts) for b in range(B)]
    lst = []
    for pos, (b, part) in enumerate(pairs):
        n = min(max(int(ctx[b]), 0), max_ctx)
        toks = [t for t in range(prefix + part * size, prefix + (part + 1) * size) if t < n]
        if toks or keep_empty:
            lst.append((-len(toks), pos, part * B + b))
    return [it for _, _, it in sorted(lst)]


@pytest.mark.parametrize("seed", range(6))
def test_schedule_lists_every_item_longest_first(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 40))
    max_ctx = int(rng.integers(1, 3000))
    ctx = rng.integers(0, max_ctx + 1, B)
    ctx[0] = max_ctx
    for S in (0, 16, 128, 512, 4096):
        for prefix in (0, 16 * int(rng.integers(0, max_ctx // 16 + 1))):
            if S == 0 and prefix:
                with pytest.raises(pa.PagedAttnError):
                    pa.paged_attn_schedule(ctx, max_ctx, S, prefix)
                continue
            got = pa.paged_attn_schedule(ctx, max_ctx, S, prefix)
            assert list(got) == _brute_items(ctx, max_ctx, S, prefix), (S, prefix)


@pytest.mark.parametrize("max_ctx,S", [(0, 64), (0, 0), (20, 32), (32, 32), (33, 32)])
def test_schedule_matches_the_decode_partitioning(max_ctx, S):
    """A call whose decode runs one partition keeps every sequence's item,
    also when no sequence holds a token."""
    ctx = [0, max_ctx, max_ctx // 2]
    got = list(pa.paged_attn_schedule(ctx, max_ctx, S))
    assert got == _brute_items(ctx, max_ctx, S, 0)
    if pa.paged_attn_num_partitions(max_ctx, S) == 1:
        assert sorted(got) == [0, 1, 2]
    else:
        assert 0 not in got


def test_schedule_validation():
    with pytest.raises(pa.PagedAttnError):
        pa.paged_attn_schedule([10, 20], 20, 8)          # not a multiple of 16
    with pytest.raises(pa.PagedAttnError):
        pa.paged_attn_schedule([10, 20], 20, 16, prefix_len=32)
    ctx = np.array([100, 100], np.int32)
    items = np.zeros(1, np.int32)
    n = ctypes.c_int32()
    rc = pa._lib.paged_attn_schedule(ctx.ctypes.data_as(pa._pi32), 2, 100, 16, 0,
                                     items.ctypes.data_as(pa._pi32), 1, ctypes.byref(n))
    assert rc == pa.PA_EINVAL and n.value == 14


@pytest.mark.parametrize("num_items,items,code", [(-1, 0x90000, pa.PA_EINVAL), (100, 0x90000, pa.PA_EINVAL),
                                                  (2, 0, pa.PA_EINVAL), (2, 0x90002, pa.PA_EINVAL)])
def test_scheduled_decode_validation(num_items, items, code):
    p = make_pool()
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_decode_scheduled(p, 0x30000, 0x50000, 8, 0x60000, 2, 32, 0.1, 128, 64, items,
                                       num_items, 0x80000, 0xA0000, 0xB0000)
    assert e.value.code == code, pa.pa_last_error()


@pytest.mark.parametrize("kw,code", [
    (dict(group_len=24), "EINVAL"),                   # not a multiple of 16
    (dict(group_len=2048), "EINVAL"),                 # longer than 1024
    (dict(group_len=0), "EINVAL"),                    # the grouped call needs group tokens
    (dict(num_groups=0), "EINVAL"),
    (dict(num_groups=3), "EINVAL"),                   # more groups than sequences
    (dict(max_group_size=17), "EINVAL"),              # 17 x 4 rows > 64
    (dict(max_group_size=0), "EINVAL"),
    (dict(group_start=None), "EINVAL"),
    (dict(group_start=0x70002), "EINVAL"),            # misaligned
    (dict(prefix_len=96, group_len=48), "EINVAL"),    # past max_context_len = 128
])
def test_grouped_cascade_validation(kw, code):
    args = dict(prefix_len=64, group_len=32, group_start=0x70000, num_groups=2, max_group_size=2)
    args.update(kw)
    p = make_pool()
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_decode_cascade_groups(p, 0x30000, 0x50000, 8, 0x60000, 2, 32, 0.1, 128, 64,
                                            args["prefix_len"], 64, args["group_start"],
                                            args["num_groups"], args["max_group_size"],
                                            args["group_len"], None, 0, 0xA0000, 0xB0000)
    assert e.value.code == getattr(pa, "PA_" + code), pa.pa_last_error()


def test_grouped_workspace_and_reduce_validation():
    ob, lb, m = pa.paged_attn_cascade_groups_workspace_size(94, 32, 128, 3324, 1024, 2048, 1024, 256)
    assert m == 2 + 1 + 1 and ob == 94 * 32 * m * 128 * 4 and lb == 94 * 32 * m * 4
    with pytest.raises(pa.PagedAttnError):
        pa.paged_attn_cascade_groups_workspace_size(4, 32, 128, 300, 64, 256, 64, 64)  # past 300
    with pytest.raises(pa.PagedAttnError):
        pa.paged_attn_reduce_cascade_groups(0xA0000, 0xB0000, 0x60000, 2, 32, 128, 64, 64, 64, 0,
                                            4, 0x90000)


def test_grouped_cascade_empty_batch_is_a_no_op():
    p = make_pool()
    pa.paged_attn_decode_cascade_groups(p, 0, 0, 8, 0, 0, 32, 0.1, 128, 64, 64, 64, None, 0, 0, 32,
                                        None, 0, None, None)


# ------------------------------------------------------------ table check

def _shared_tables():
    """Three sequences sharing a 2-block prefix; sequences 1 and 2 form a
    group sharing one block after it."""
    bt = np.array([[0, 1, 2, 3, -1],
                   [0, 1, 4, 5, 6],
                   [0, 1, 4, 7, -1]], dtype=np.int32)
    ctx = np.array([64, 80, 60], dtype=np.int32)
    return bt, ctx


def test_check_tables_accepts_shared_prefix_and_groups():
    p = make_pool(nb=10)
    bt, ctx = _shared_tables()
    pa.paged_attn_check_tables(p, bt, ctx)
    pa.paged_attn_check_tables(p, bt, ctx, prefix_len=32)
    pa.paged_attn_check_tables(p, bt, ctx, prefix_len=32, group_start=[0, 1, 3], group_len=16)


def test_check_tables_rejects_a_prefix_mismatch():
    p = make_pool(nb=10)
    bt, ctx = _shared_tables()
    bt[2, 1] = 8                         # sequence 2's second prefix block differs from row 0
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_check_tables(p, bt, ctx, prefix_len=32)
    assert e.value.code == pa.PA_EINVAL and e.value.bad_seq == 2
    assert "block_tables[2][1] = 8" in pa.pa_last_error()
    pa.paged_attn_check_tables(p, bt, ctx, prefix_len=16)     # the first block still matches


def test_check_tables_rejects_a_group_mismatch():
    p = make_pool(nb=10)
    bt, ctx = _shared_tables()
    bt[2, 2] = 9                         # differs from the group's first row (sequence 1)
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_check_tables(p, bt, ctx, prefix_len=32, group_start=[0, 1, 3], group_len=16)
    assert e.value.bad_seq == 2
    # as groups of one, nothing is shared after the prefix
    pa.paged_attn_check_tables(p, bt, ctx, prefix_len=32, group_start=[0, 1, 2, 3], group_len=16)


def test_check_tables_short_sequences_only_need_what_they_read():
    p = make_pool(nb=10)
    bt, ctx = _shared_tables()
    ctx[1] = 10                          # inside the first prefix block
    bt[1, 1] = 9                         # an entry this sequence never reads
    pa.paged_attn_check_tables(p, bt, ctx, prefix_len=32)
    ctx[1] = 17                          # now it reads the second block as well
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_check_tables(p, bt, ctx, prefix_len=32)
    assert e.value.bad_seq == 1


@pytest.mark.parametrize("mutate", ["id_out_of_pool", "negative_id", "ctx_past_table", "bad_groups"])
def test_check_tables_rejects_bad_tables(mutate):
    p = make_pool(nb=10)
    bt, ctx = _shared_tables()
    kw = {}
    if mutate == "id_out_of_pool":
        bt[1, 4] = 10
    elif mutate == "negative_id":
        bt[2, 3] = -1
    elif mutate == "ctx_past_table":
        ctx[0] = 81
    else:
        kw = dict(prefix_len=32, group_start=[0, 2, 1, 3], group_len=16)
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_check_tables(p, bt, ctx, **kw)
    assert e.value.code == pa.PA_EINVAL


def test_check_tables_accepts_the_stage_workloads():
    from workloads import build_config, group_starts
    for k in (2, 3, 5):
        w = build_config(k, values=False)
        p = pa.kv_pool_create(w.num_blocks, 16, w.num_kv_heads, w.head_dim, FAKE_K, FAKE_V)
        kw = dict(prefix_len=16 * w.meta["prefix_blocks"])
        if "groups" in w.meta:
            kw.update(group_start=group_starts(w), group_len=16 * w.meta["mid_blocks"])
        pa.paged_attn_check_tables(p, w.block_tables, w.context_lens, **kw)
        p.close()


# ------------------------------------------------------------ trace layouts

def test_cascade_trace_layout():
    p = make_pool(nb=10, hkv=8)
    lay = pa.paged_attn_cascade_trace_layout(p, 10, 32, 2300, 512, 2048, 512)
    # prefix: 4 partitions x ceil(40 / 64) = 1 row group x 8 heads x 32 tiles
    assert lay["prefix_tiles"] == 32 and lay["group_offset"] == 3 * 4 * 1 * 8 * 32
    assert lay["group_tiles"] == 0 and lay["decode_offset"] == lay["group_offset"]
    # one 512-token partition after the prefix, 10 sequences, 8 heads, 32 tiles
    assert lay["decode_tiles"] == 32 and lay["total"] == lay["decode_offset"] + 3 * 10 * 8 * 32
    g = pa.paged_attn_cascade_trace_layout(p, 40, 64, 3000, 512, 2048, 1024, num_groups=5,
                                           group_len=256)
    # 40 x 8 = 320 rows -> 5 row groups; 2 prefix partitions of 64 tiles
    assert g["group_offset"] == 3 * 2 * 5 * 8 * 64 and g["group_tiles"] == 16
    assert g["decode_offset"] == g["group_offset"] + 3 * 5 * 8 * 16
    assert g["total"] == g["decode_offset"] + 3 * 2 * 40 * 8 * 32     # 696 tokens after: 2 parts
    with pytest.raises(pa.PagedAttnError):
        pa.paged_attn_cascade_trace_layout(p, 10, 30, 2300, 512, 2048, 512)


def test_cascade_trace_capacity_checked():
    p = make_pool(nb=10, hkv=8)
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_decode_cascade_trace(p, 0x30000, 0x50000, 160, 0x60000, 10, 32, 0.1, 2300, 512,
                                           2048, 512, None, 0, 0, 0, None, 0, 0xA0000, 0xB0000,
                                           0xC0000, 100)
    assert e.value.code == pa.PA_EINVAL and "trace_capacity" in pa.pa_last_error()
    with pytest.raises(pa.PagedAttnError) as e:
        pa.paged_attn_decode_scheduled_trace(p, 0x1000, 0x2000, 4, 0x3000, 2, 32, 0.1, 64, 0,
                                             0x4000, 2, 0x4000, None, None, 0x5000, 10)
    assert e.value.code == pa.PA_EINVAL and "trace_capacity" in pa.pa_last_error()


def test_noalloc_rejects_partials_beyond_the_scratch_array():
    """Checked on the host before any HIP call: 64 MiB hold the partials of
    the stage batches at 512-token partitions up to the fixer's, not more."""
    p = make_pool(nb=10)
    with pytest.raises(pa.PagedAttnError) as e:
        # 256 x 32 heads x 16 partitions x (128 + 1) fp32 > 64 MiB
        pa.paged_attn_decode_noalloc(p, 0x30000, 0x50000, 512, 0x60000, 256, 32, 0.1, 8192, 512,
                                     0x70000)
    assert e.value.code == pa.PA_EINVAL and "scratch" in pa.pa_last_error()
    ob, lb = pa.paged_attn_workspace_size(160, 32, 128, 3328, 512)
    assert -(-ob // 256) * 256 + lb <= pa.NOALLOC_SCRATCH_BYTES
