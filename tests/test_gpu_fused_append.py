"""GPU tests of the fused KV append + decode entry points: the same output
bits and the same pools as paged_attn_append_kv followed by the decode in the
same launch configuration, and the oracle's result with the new rows in
place.  The new token's slot holds NaN before the step, so a kernel that read
the slot instead of the new rows would fail.  Every case prints its name
before touching the GPU.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import compare, decode_workload  # noqa: E402
from workloads import f32_to_bf16_bits, group_starts, grouped_case, logical_case, page_case  # noqa: E402

DEV = "cuda:0"
NAN = 0x7FC0


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


def _new_rows(w, seed):
    rng = np.random.default_rng(seed)
    shape = (w.batch, w.num_kv_heads, w.head_dim)
    return (f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32)),
            f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32)))


def _slots(w):
    """(block, row) of token ctx - 1 of every non-empty sequence."""
    out = []
    for b in range(w.batch):
        n = int(w.context_lens[b])
        if n > 0:
            out.append((b, int(w.block_tables[b, (n - 1) // 16]), (n - 1) % 16))
    return out


def _dev16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV)


def check_fused(w, k_new, v_new, what, **kw):
    """Fused vs append + decode (bit for bit, outputs and pools) and the
    oracle with the new rows written on the host."""
    from paper_2510_14126_amd.device import PagedBatch
    for b, blk, r in _slots(w):                 # the slot holds NaN before the step
        w.k_pool[blk, :, r, :] = NAN
        w.v_pool[blk, :, r, :] = NAN
    kd, vd = _dev16(k_new), _dev16(v_new)
    pa_ = PagedBatch(w, DEV, **kw)
    pa_.append(kd, vd)
    pa_.run()
    pb_ = PagedBatch(w, DEV, **kw)
    pb_.decode_append(kd, vd)
    if pb_.needs_reduce:
        pb_.reduce()
    torch.cuda.synchronize()
    unfused, fused = pa_.out_bits(), pb_.out_bits()
    pools_equal = torch.equal(pa_.k, pb_.k) and torch.equal(pa_.v, pb_.v)
    pa_.close()
    pb_.close()
    assert pools_equal, f"{what}: the pools differ after the step"
    assert np.array_equal(unfused, fused), f"{what}: fused output differs from append + decode"
    for b, blk, r in _slots(w):                 # the oracle's pools after the append
        w.k_pool[blk, :, r, :] = k_new[b]
        w.v_pool[blk, :, r, :] = v_new[b]
    rep = compare(fused, decode_workload(w)[0])
    say(f"{what}: {rep}")
    assert rep.passed, f"{what}: {rep}"


CTX = [1, 16, 17, 33, 512, 513, 1000, 2048, 95]


@pytest.mark.parametrize("schedule", [False, True], ids=["grid", "list"])
@pytest.mark.parametrize("S", [0, 64, 512])
@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (64, 8, 128), (8, 2, 64)],
                         ids=["g4", "g8", "g4-d64"])
def test_fused_append_plain(hq, hkv, d, S, schedule):
    what = f"fused append Hq={hq} Hkv={hkv} D={d} S={S} schedule={schedule}"
    say(what)
    lc = logical_case(101, len(CTX), hq, hkv, d, CTX)
    w = page_case(lc, 102, extra_blocks=4)
    k_new, v_new = _new_rows(w, 103)
    check_fused(w, k_new, v_new, what, partition_size=S, schedule=schedule)


@pytest.mark.parametrize("schedule", [False, True], ids=["grid", "list"])
@pytest.mark.parametrize("hq", [32, 64], ids=["g4", "g8"])
def test_fused_append_cascade(hq, schedule):
    what = f"fused append cascade Hq={hq} schedule={schedule}"
    say(what)
    ctx = [513, 600, 1024, 1025, 700, 2000, 529]
    lc = logical_case(111, len(ctx), hq, 8, 128, ctx, prefix_len=512)
    w = page_case(lc, 112, extra_blocks=4)
    k_new, v_new = _new_rows(w, 113)
    check_fused(w, k_new, v_new, what, partition_size=256, prefix_len=512,
                prefix_partition_size=128, schedule=schedule)


@pytest.mark.parametrize("schedule", [False, True], ids=["grid", "list"])
@pytest.mark.parametrize("hq", [32, 64], ids=["g4", "g8"])
def test_fused_append_cascade_groups(hq, schedule):
    what = f"fused append grouped cascade Hq={hq} schedule={schedule}"
    say(what)
    sizes = [2, 3, 1, 2] if hq == 32 else [2, 1, 3]
    rng = np.random.default_rng(121)
    suffix = rng.integers(1, 500, size=sum(sizes))     # the new token after the shared parts
    w = grouped_case(121, hq, 8, 128, 256, sizes, 128, suffix)
    k_new, v_new = _new_rows(w, 122)
    check_fused(w, k_new, v_new, what, partition_size=128, prefix_len=256,
                prefix_partition_size=128, group_start=group_starts(w), group_len=128,
                schedule=schedule)
