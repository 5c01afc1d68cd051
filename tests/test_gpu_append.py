"""GPU tests of the KV append against the CPU oracle, and of the whole decode
loop (allocate at block boundaries, append, attend) over many steps.

Every case prints its name before touching the GPU.  Pools are compared bit
for bit with the oracle's append; attention outputs pass the parity gate.
"""
from dataclasses import replace

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import append_kv, compare, paged_decode  # noqa: E402
from workloads import f32_to_bf16_bits, logical_case, page_case  # noqa: E402

DEV = "cuda:0"


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


def _dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(DEV)


def _host_u16(t):
    return t.cpu().numpy().view(np.uint16)


def _bf16(rng, shape):
    return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def test_append_bit_exact_against_oracle():
    from paper_2510_14126_amd import binding
    say("append: bit-exact pools, contexts at block starts, middles, ends and 0")
    rng = np.random.default_rng(7)
    nb, hkv, d = 40, 8, 128
    kp, vp = _bf16(rng, (nb, hkv, 16, d)), _bf16(rng, (nb, hkv, 16, d))
    ctx = np.array([1, 16, 17, 31, 32, 33, 0, 200], np.int32)
    B, W = len(ctx), 16
    ids = rng.permutation(nb).astype(np.int32)
    bt = np.full((B, W), -1, np.int32)
    cur = 0
    for b, n in enumerate(ctx):
        m = (int(n) + 15) // 16
        bt[b, :m] = ids[cur: cur + m]
        cur += m
    kn, vn = _bf16(rng, (B, hkv, d)), _bf16(rng, (B, hkv, d))
    k_dev, v_dev = _dev(kp), _dev(vp)
    pool = binding.kv_pool_create(nb, 16, hkv, d, k_dev, v_dev)
    binding.paged_attn_append_kv(pool, _dev(kn), _dev(vn), _dev(bt), W, _dev(ctx), B)
    torch.cuda.synchronize()
    want_k, want_v = append_kv(kp, vp, bt, ctx, kn, vn)
    assert np.array_equal(_host_u16(k_dev), want_k)
    assert np.array_equal(_host_u16(v_dev), want_v)
    pool.close()


def test_append_out_of_range_ids_stay_inside_the_pool():
    from paper_2510_14126_amd import binding
    say("append: table ids out of range are clamped into the pool; guard rows untouched")
    rng = np.random.default_rng(8)
    nb, hkv, d = 6, 2, 64
    guard = 2                                   # blocks of sentinel data on each side
    full = _bf16(rng, (nb + 2 * guard, hkv, 16, d))
    fullv = _bf16(rng, (nb + 2 * guard, hkv, 16, d))
    k_all, v_all = _dev(full), _dev(fullv)
    k_dev, v_dev = k_all[guard: guard + nb], v_all[guard: guard + nb]
    bt = np.array([[-7, 0], [1, 99]], np.int32)
    ctx = np.array([5, 20], np.int32)
    kn, vn = _bf16(rng, (2, hkv, d)), _bf16(rng, (2, hkv, d))
    pool = binding.kv_pool_create(nb, 16, hkv, d, k_dev, v_dev)
    binding.paged_attn_append_kv(pool, _dev(kn), _dev(vn), _dev(bt), 2, _dev(ctx), 2)
    torch.cuda.synchronize()
    got_k, got_v = _host_u16(k_all), _host_u16(v_all)
    for lo, hi in ((0, guard), (guard + nb, nb + 2 * guard)):
        assert np.array_equal(got_k[lo:hi], full[lo:hi]) and np.array_equal(got_v[lo:hi], fullv[lo:hi])
    clamped = np.clip(bt, 0, nb - 1)
    want_k, want_v = append_kv(full[guard: guard + nb], fullv[guard: guard + nb], clamped, ctx, kn, vn)
    assert np.array_equal(got_k[guard: guard + nb], want_k)
    assert np.array_equal(got_v[guard: guard + nb], want_v)
    pool.close()


@pytest.mark.parametrize("fused", [False, True], ids=["append-then-decode", "fused"])
@pytest.mark.parametrize("hq,hkv,d,S", [(32, 8, 128, 64), (64, 8, 128, 0), (8, 2, 64, 32)],
                         ids=["g4-d128-split", "g8-d128", "g4-d64-split"])
def test_decode_loop_append_then_attend(hq, hkv, d, S, fused):
    """Prompts of several lengths grow token by token: a fresh block comes
    from the pool allocator whenever a token starts one, the step's K/V is
    appended on the GPU (by the append kernel, or inside the decode launch
    when fused), and the step's attention must match the oracle run on the
    oracle-appended pools; the pools stay bit-identical throughout."""
    from paper_2510_14126_amd import binding
    from paper_2510_14126_amd.device import PagedBatch
    steps = 40
    prompts = [1, 15, 16, 17, 100, 255]
    B = len(prompts)
    say(f"decode loop hq={hq} hkv={hkv} d={d} S={S} fused={fused} prompts={prompts} steps={steps}")
    case = logical_case(101, B, hq, hkv, d, prompts)
    growth = sum((p + steps + 15) // 16 - (p + 15) // 16 for p in prompts)
    w = page_case(case, 102, share_prefix=False, extra_blocks=growth + 3,
                  table_pad=(steps + 15) // 16 + 1, partition_size=S)
    k_dev, v_dev = _dev(w.k_pool), _dev(w.v_pool)
    alloc = binding.kv_pool_create(w.num_blocks, 16, hkv, d, k_dev, v_dev)
    used = np.unique(np.concatenate([w.block_tables[b, : (p + 15) // 16] for b, p in enumerate(prompts)]))
    binding.kv_pool_claim(alloc, used.tolist())
    kp, vp, bt = w.k_pool.copy(), w.v_pool.copy(), w.block_tables.copy()
    ctx = np.array(prompts, np.int32)
    rng = np.random.default_rng(103)
    W = bt.shape[1]
    for step in range(steps):
        ctx = ctx + 1
        for b in range(B):
            t = int(ctx[b]) - 1
            if t % 16 == 0:
                bt[b, t // 16] = binding.kv_pool_alloc(alloc, 1)[0]
        kn, vn, q = _bf16(rng, (B, hkv, d)), _bf16(rng, (B, hkv, d)), _bf16(rng, (B, hq, d))
        bt_dev, ctx_dev = _dev(bt), _dev(ctx)
        if not fused:
            binding.paged_attn_append_kv(alloc, _dev(kn), _dev(vn), bt_dev, W, ctx_dev, B)
        kp, vp = append_kv(kp, vp, bt, ctx, kn, vn)
        ws = replace(w, context_lens=ctx.copy(), block_tables=bt.copy(), q=q, k_pool=kp, v_pool=vp)
        pb = PagedBatch(ws, DEV, partition_size=S, register_blocks=False, k_pool=k_dev, v_pool=v_dev)
        if fused:
            pb.decode_append(_dev(kn), _dev(vn))
            if pb.needs_reduce:
                pb.reduce()
        else:
            pb.run()
        torch.cuda.synchronize()
        out = pb.out_bits()
        pb.close()
        ref, _ = paged_decode(q, kp, vp, bt, ctx, w.scale)
        rep = compare(out, ref)
        assert rep.passed, f"step {step}: {rep}"
    say(f"decode loop: {steps} steps passed; final contexts {ctx.tolist()}")
    assert np.array_equal(_host_u16(k_dev), kp) and np.array_equal(_host_u16(v_dev), vp)
    alloc.close()
