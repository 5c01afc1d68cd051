"""GPU parity and bit-exact tests of the HIP decode path against the CPU oracle.

Every case prints its name before touching the GPU.  Inputs come from the
seeded generators in ``workloads``; expected values come from ``oracle`` or
from hand-derived closed forms in ``tests/golden``.
"""
import json
import math
import os

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import compare, decode_workload, split_partials  # noqa: E402
from oracle.attention import bf16_to_f64  # noqa: E402
from workloads import (Workload, build_config, duplicate_shared_blocks, f32_to_bf16_bits,  # noqa: E402
                       logical_case, page_case, permute_blocks)

HERE = os.path.dirname(os.path.abspath(__file__))
DEV = "cuda:0"


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


def run(w, S=None, **kw):
    from paper_2510_14126_amd.device import PagedBatch
    pb = PagedBatch(w, DEV, partition_size=S, **kw)
    pb.run()
    torch.cuda.synchronize()
    return pb


def gpu_out(w, S=None, **kw):
    pb = run(w, S, **kw)
    if pb.needs_reduce and not pb.prefix_len and pb.num_parts == 1:
        raise AssertionError("inconsistent reduce plan")
    out = pb.out_bits()
    pb.close()
    return out


def assert_gate(out_bits, ref, what):
    rep = compare(out_bits, ref)
    say(f"{what}: {rep}")
    assert rep.passed, f"{what}: {rep}"
    return rep


# ------------------------------------------------------------------ configs

@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_config_parity_all_outputs(k, stage_batches):
    """Every output of each workload through the plain split-KV decode (its
    stated or default partition size) and the reduce, against the oracle."""
    w = stage_batches.workload(k)
    say(f"config {k} {w.name}: B={w.batch} Hq={w.num_q_heads} Hkv={w.num_kv_heads} D={w.head_dim} "
        f"NB={w.num_blocks} max_ctx={w.max_context_len} S={w.partition_size}")
    out = gpu_out(w)
    ref, _ = stage_batches.reference(k)
    assert_gate(out, ref, f"config {k} all {w.batch} sequences")
    if k == 5:
        # every output is a convex combination of V rows: finite and no larger
        # in magnitude than the largest |V| in the pool (+1 bf16 ulp of rounding)
        vmax = max(int((w.v_pool[i: i + 8192] & 0x7FFF).max()) for i in range(0, w.num_blocks, 8192))
        assert np.isfinite(bf16_to_f64(out)).all()
        assert int((out & 0x7FFF).max()) <= vmax + 1


# -------------------------------------------------------- shapes and edges

EDGE_CTX = [1, 2, 15, 16, 17, 511, 512, 513, 1024]


@pytest.mark.parametrize("S", [0, 16, 64, 512])
@pytest.mark.parametrize("d,hq,hkv", [(128, 32, 8), (64, 8, 2), (128, 8, 1), (128, 64, 8)])
def test_edge_contexts(S, d, hq, hkv):
    say(f"edge contexts S={S} D={d} Hq={hq} Hkv={hkv}")
    case = logical_case(100 + d + hq, len(EDGE_CTX), hq, hkv, d, EDGE_CTX)
    w = page_case(case, 7, extra_blocks=5)
    assert_gate(gpu_out(w, S), decode_workload(w)[0], f"edges S={S}")


@pytest.mark.parametrize("hq", [8, 16])
@pytest.mark.parametrize("S", [0, 64])
def test_empty_and_single_token_contexts(S, hq):
    say(f"ctx 0 and 1, S={S} Hq={hq}")
    case = logical_case(9, 5, hq, 2, 128, [0, 1, 33, 1, 200])
    w = page_case(case, 3)
    out = gpu_out(w, S)
    G = hq // 2
    assert np.all(out[0] & 0x7FFF == 0), "empty context must give zeros"
    for b in (1, 3):
        for h in range(hq):
            assert np.array_equal(out[b, h], case.v[b][h // G, 0]), "ctx=1 must return V exactly"
    assert_gate(out[2:3], decode_workload(w, seqs=[2])[0], "ctx 33 beside empty rows")


@pytest.mark.parametrize("S", [16, 64, 512, 4096])
def test_partition_sizes(S):
    say(f"partition size {S}")
    case = logical_case(12, 5, 32, 8, 128, [4100, 700, 520, 2049, 513], prefix_len=512)
    w = page_case(case, 13)
    assert_gate(gpu_out(w, S), decode_workload(w)[0], f"S={S}")


def test_split_partials_match_oracle():
    say("split partials vs oracle partials, S=64")
    case = logical_case(14, 3, 8, 2, 128, [300, 64, 129])
    w = page_case(case, 15)
    pb = run(w, 64)
    o, l = pb.partials()
    pb.close()
    ro, rl = split_partials(w.q, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale, 64)
    for b, n in enumerate(w.context_lens):
        pbn = -(-int(n) // 64)
        rep = compare(o[b, :, :pbn], ro[b, :, :pbn], gpu_is_bf16_bits=False)
        assert rep.passed, rep
        # Both kernels round each softmax weight to bf16 (RNE, relative error
        # <= 2^-9) before the PV product and sum the rounded weights, so the
        # partition's log-sum-exp is within log(1 + 2^-9) < 2^-9 of the exact
        # value, plus fp32 accumulation error.
        np.testing.assert_allclose(l[b, :, :pbn], rl[b, :, :pbn], rtol=0, atol=2 ** -9 + 1e-5)


# ---------------------------------------------------------- bit-exact tests

def _embed(q_rows, K, V, scale, d=64, group=4):
    """Embed a hand case (one KV head) into a D=64, G=4 pool by zero padding."""
    n = len(K)
    R = len(q_rows)
    q = np.zeros((1, group, d), np.uint16)
    for r in range(group):
        q[0, r, : len(q_rows[0])] = q_rows[r % R]
    nb = (n + 15) // 16 + 2
    kp = np.zeros((nb, 1, 16, d), np.uint16); vp = np.zeros_like(kp)
    ids = list(range(nb - 1, 0, -1))[: (n + 15) // 16]
    for t in range(n):
        kp[ids[t // 16], 0, t % 16, : len(K[t])] = K[t]
        vp[ids[t // 16], 0, t % 16, : len(V[t])] = V[t]
    bt = np.full((1, len(ids) + 1), -1, np.int32); bt[0, : len(ids)] = ids
    return Workload(name="hand", batch=1, num_q_heads=group, num_kv_heads=1, head_dim=d,
                    num_blocks=nb, context_lens=np.array([n], np.int32), block_tables=bt,
                    scale=scale, q=q, k_pool=kp, v_pool=vp)


with open(os.path.join(HERE, "golden", "hand_cases.json")) as f:
    HAND = json.load(f)["cases"]


@pytest.mark.parametrize("d,group", [(64, 4), (128, 8)], ids=["valu", "mfma"])
@pytest.mark.parametrize("case", HAND, ids=[c["name"] for c in HAND])
def test_hand_cases(case, d, group):
    say(f"hand case {case['name']} D={d} G={group}")
    w = _embed(case["q_bits"], case["K_bits"], case["V_bits"], case["scale"], d=d, group=group)
    out = gpu_out(w)
    R = len(case["q"])
    ncol = len(case["out"][0])
    for r in range(group):
        got = bf16_to_f64(out[0, r, :ncol])
        want = np.array(case["out"][r % R])
        np.testing.assert_allclose(got, want, rtol=2 ** -8, atol=0)
        assert np.all(out[0, r, ncol:] & 0x7FFF == 0)
        if "out_bf16_bits" in case:
            assert list(out[0, r, :ncol]) == case["out_bf16_bits"][r % R], "bf16 output must use RNE"
    if case["name"] in ("single_token", "argmax_group2") or case["name"].startswith("rne"):
        for r in range(group):
            want_bits = f32_to_bf16_bits(np.float32(case["out"][r % R]))
            assert np.array_equal(out[0, r, :ncol], want_bits)


def _argmax_workload(ctx, targets, d=128, hq=32, hkv=8, seed=3, poison=True):
    """K of each target token = 4096 e0 and q = e0, so out = V[target] exactly.

    Rows past the context and unused blocks hold K = 8192 e0 (they would win)
    and V = NaN, so any read of them shows up.  V encodes the physical slot:
    (block mod 256, block div 256, row) as exact bf16 integers.
    """
    case = logical_case(seed, len(ctx), hq, hkv, d, list(ctx))
    w = page_case(case, seed + 1, extra_blocks=6, poison=poison)
    e0 = np.zeros(d, np.float32); e0[0] = 1.0
    w.q[:] = f32_to_bf16_bits(e0)
    want = []
    nblk = (w.context_lens + 15) // 16
    used = {(int(w.block_tables[b, j]), r) for b in range(w.batch) for j in range(nblk[b])
            for r in range(min(16, int(w.context_lens[b]) - 16 * j))}
    for (pid, r) in used:
        w.k_pool[pid, :, r, :] = 0
        w.v_pool[pid, :, r, :] = 0
        w.v_pool[pid, :, r, 0:3] = f32_to_bf16_bits(np.float32([pid % 256, pid // 256, r]))
    for b, t in enumerate(targets):
        pid = int(w.block_tables[b, t // 16]); r = t % 16
        w.k_pool[pid, :, r, 0] = 0x4580  # 4096.0
        want.append((pid, r))
    return w, want


@pytest.mark.parametrize("hq", [32, 64])
@pytest.mark.parametrize("S", [0, 64, 512])
def test_argmax_reads_exact_slot(S, hq):
    ctx = [1, 40, 513, 1024, 1024, 700, 17]
    targets = [0, 39, 512, 511, 0, 64, 16]
    say(f"argmax slot selection S={S} Hq={hq}")
    w, want = _argmax_workload(ctx, targets, hq=hq)
    out = gpu_out(w, S)
    for b, (pid, r) in enumerate(want):
        got = bf16_to_f64(out[b, :, :3])
        assert np.all(got[:, 0] == pid % 256) and np.all(got[:, 1] == pid // 256) \
            and np.all(got[:, 2] == r), f"seq {b}: wanted slot ({pid},{r}), got {got[0]}"
        assert np.all(out[b, :, 3:] & 0x7FFF == 0)


def test_poison_past_context_is_never_used():
    say("NaN/huge poison past the context")
    case = logical_case(21, 4, 32, 8, 128, [17, 31, 5, 600])
    for S in (0, 64):
        clean = gpu_out(page_case(case, 7, poison=False), S)
        dirty = gpu_out(page_case(case, 7, poison=True), S)
        assert np.array_equal(clean, dirty)
        assert np.isfinite(bf16_to_f64(dirty)).all()


@pytest.mark.parametrize("hq", [32, 64])
def test_block_permutation_bit_identical(hq):
    say(f"physical block permutation Hq={hq}")
    w = page_case(logical_case(31, 6, hq, 8, 128, [900, 40, 600, 33, 48, 2048], prefix_len=32), 5)
    base = gpu_out(w, 512)
    for s in range(2):
        assert np.array_equal(base, gpu_out(permute_blocks(w, 60 + s), 512))


@pytest.mark.parametrize("hq", [32, 64])
def test_shared_prefix_equals_duplicated_bit_identical(hq):
    say(f"shared prefix vs duplicated copies Hq={hq}")
    w = page_case(logical_case(32, 6, hq, 8, 128, [900, 600, 2100, 520, 515, 1000], prefix_len=512), 6)
    assert w.meta["shared_blocks"] == 32
    a = gpu_out(w, 512)
    b = gpu_out(duplicate_shared_blocks(w), 512)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("S", [0, 512])
@pytest.mark.parametrize("hq", [32, 64])
def test_cache_policy_changes_no_bit(hq, S):
    """The plain decode loads its tiles with the streaming hint while the pool
    holds no shared block and with the default policy otherwise: one extra
    reference to a block switches the policy, never a result."""
    say(f"cache policy switch Hq={hq} S={S}")
    from paper_2510_14126_amd import binding
    from paper_2510_14126_amd.device import PagedBatch
    w = page_case(logical_case(34, 6, hq, 8, 128, [900, 40, 600, 33, 2048, 1500]), 8)
    pb = PagedBatch(w, DEV, partition_size=S)
    assert binding.kv_pool_num_shared(pb.pool) == 0
    pb.run()
    torch.cuda.synchronize()
    streamed = pb.out_bits().copy()
    some_block = int(w.block_tables[0, 0])
    binding.kv_pool_retain(pb.pool, [some_block])
    assert binding.kv_pool_num_shared(pb.pool) == 1
    pb.out.zero_()
    pb.run()
    torch.cuda.synchronize()
    cached = pb.out_bits().copy()
    binding.kv_pool_release(pb.pool, [some_block])
    pb.close()
    assert np.array_equal(streamed, cached)
    assert_gate(streamed, decode_workload(w)[0], f"cache policy Hq={hq} S={S}")


@pytest.mark.parametrize("k", [2, 1])
def test_repeat_runs_bit_identical(k, stage_batches):
    say(f"determinism config {k}")
    w = stage_batches.workload(k)
    from paper_2510_14126_amd.device import PagedBatch
    pb = PagedBatch(w, DEV)
    outs = []
    for _ in range(3):
        pb.out.zero_()
        pb.run()
        torch.cuda.synchronize()
        outs.append(pb.out_bits().copy())
    pb.close()
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


@pytest.mark.parametrize("hq", [32, 64])
def test_single_partition_through_reduce_matches_single_pass(hq):
    say(f"P_b = 1 through the reduce vs single pass Hq={hq}")
    case = logical_case(33, 3, hq, 8, 128, [2000, 300, 512])
    w = page_case(case, 8)
    split = gpu_out(w, 512)            # sequence 0 splits, 1 and 2 have one partition
    single = gpu_out(w, 0)
    assert np.array_equal(split[1:], single[1:])


def test_large_pool_offsets_above_4gib():
    """Blocks whose byte offsets exceed 4 GiB (64-bit address arithmetic)."""
    say("pool offsets above 4 GiB")
    case = logical_case(34, 3, 32, 8, 128, [300, 47, 1000])
    small = page_case(case, 9)
    tile = 8 * 16 * 128 * 2  # bytes per block of one pool
    nb_big = (5 << 30) // tile + 64
    remap = np.arange(small.num_blocks) + (nb_big - small.num_blocks)
    kbig = torch.empty((nb_big, 8, 16, 128), dtype=torch.int16, device=DEV)
    vbig = torch.empty_like(kbig)
    kbig[remap[0]: remap[-1] + 1] = torch.from_numpy(small.k_pool.view(np.int16)).to(DEV)
    vbig[remap[0]: remap[-1] + 1] = torch.from_numpy(small.v_pool.view(np.int16)).to(DEV)
    big = Workload(**{**small.__dict__})
    bt = small.block_tables.copy(); bt[bt >= 0] = remap[bt[bt >= 0]]
    big.block_tables = bt; big.num_blocks = nb_big
    assert int(bt.max()) * tile > (4 << 30)
    out = gpu_out(big, 512, k_pool=kbig, v_pool=vbig, register_blocks=False)
    del kbig, vbig
    torch.cuda.empty_cache()
    assert np.array_equal(out, gpu_out(small, 512))
    assert_gate(out, decode_workload(small)[0], "offsets > 4 GiB")


# ------------------------------------------------------------- index trace

def expected_trace(w, part_tokens, num_parts):
    """Host-side list of (j, phys, valid) per work item, from tables and lengths."""
    exp = {}
    for p in range(num_parts):
        for b in range(w.batch):
            n = int(w.context_lens[b])
            lo, hi = p * part_tokens, min(n, (p + 1) * part_tokens)
            tiles = []
            for j in range(lo // 16, (hi + 15) // 16 if hi > lo else lo // 16):
                tiles.append((j, int(w.block_tables[b, j]), min(16, n - 16 * j)))
            for g in range(w.num_kv_heads):
                exp[(p, b, g)] = tiles
    return exp


@pytest.mark.parametrize("hq", [32, 64])
@pytest.mark.parametrize("S", [0, 64, 512])
def test_index_trace_bit_exact(S, hq):
    from paper_2510_14126_amd import binding
    from paper_2510_14126_amd.device import PagedBatch
    say(f"index trace S={S} Hq={hq}")
    case = logical_case(40, 5, hq, 8, 128, [1, 16, 17, 700, 1300], prefix_len=0)
    w = page_case(case, 41, table_pad=3)
    pb = PagedBatch(w, DEV, partition_size=S)
    P = pb.num_parts
    part_tokens = S if P > 1 else ((w.max_context_len + 15) // 16) * 16
    tiles = part_tokens // 16
    cap = P * w.batch * w.num_kv_heads * tiles * 3
    trace = torch.full((cap,), -7, dtype=torch.int32, device=DEV)
    binding.paged_attn_decode_trace(pb.pool, pb.q, pb.bt, pb.bt_stride, pb.ctx, pb.batch, pb.hq,
                                    w.scale, pb.max_ctx, S, pb.out, pb.part_o, pb.part_lse, trace,
                                    cap)
    if P > 1:
        pb.reduce()
    torch.cuda.synchronize()
    tr = trace.cpu().numpy().reshape(P, w.batch, w.num_kv_heads, tiles, 3)
    for (p, b, g), tl in expected_trace(w, part_tokens, P).items():
        got = [tuple(int(x) for x in tr[p, b, g, i]) for i in range(tiles)]
        assert got[: len(tl)] == tl, f"item {(p, b, g)}"
        assert all(x == (-7, -7, -7) for x in got[len(tl):]), f"item {(p, b, g)} loaded extra tiles"
    # the trace build computes the same result as the production build
    assert np.array_equal(pb.out_bits(), gpu_out(w, S))
    pb.close()


# --------------------------------------------- negative controls (must fail)

def test_gate_rejects_planted_mistakes_on_gpu():
    say("negative controls through the GPU path")
    case = logical_case(50, 4, 32, 8, 128, [300, 150, 257, 100])
    w = page_case(case, 51)
    truth, _ = decode_workload(w)
    good = gpu_out(w)
    assert compare(good, truth).passed
    assert not compare(np.zeros_like(good), truth).passed
    dropped = Workload(**{**w.__dict__}); dropped.context_lens = w.context_lens - 1
    assert not compare(gpu_out(dropped), truth).passed
    bt = w.block_tables.copy()
    for b, n in enumerate(w.context_lens):
        last = (int(n) - 1) // 16
        bt[b, [0, last]] = bt[b, [last, 0]]
    swapped = Workload(**{**w.__dict__}); swapped.block_tables = bt
    assert not compare(gpu_out(swapped), truth).passed


@pytest.mark.parametrize("hq", [32, 64])
@pytest.mark.parametrize("S", [0, 512])
def test_growing_scores_force_rescales(S, hq):
    """Scores rising along the context make the running max grow many times."""
    say(f"growing scores S={S} Hq={hq}")
    case = logical_case(60, 3, hq, 8, 128, [2500, 1200, 777])
    for b in range(3):
        n = case.k[b].shape[1]
        k = bf16_to_f64(case.k[b]).astype(np.float32)
        k[:, :, 0] = np.arange(n, dtype=np.float32)[None, :] / 24.0
        case.k[b] = f32_to_bf16_bits(k)
    qf = bf16_to_f64(case.q).astype(np.float32)
    qf[:, :, 0] = 6.0
    case.q[:] = f32_to_bf16_bits(qf)
    w = page_case(case, 61)
    ref, lse = decode_workload(w)
    assert np.ptp(lse) > 10
    assert_gate(gpu_out(w, S), ref, f"growing scores S={S} Hq={hq}")


# ------------------------------------------------- shared-prefix cascade

@pytest.mark.parametrize("k", [2, 3, 5])
def test_cascade_stage_configs_all_outputs(k, stage_batches):
    """The full-grid cascade (no work list) on every workload with a shared
    prefix, every output against the oracle."""
    w = stage_batches.workload(k)
    L = w.meta["prefix_blocks"] * 16
    pps = 512 if k == 5 else 256
    say(f"cascade config {k} {w.name}: prefix {L}, prefix partitions {pps}")
    out = gpu_out(w, prefix_len=L, prefix_partition_size=pps)
    assert_gate(out, stage_batches.reference(k)[0], f"cascade config {k} all {w.batch} sequences")


CASCADE_CASES = [
    # seed, B, Hq, Hkv, ctx, prefix, S, S_pre
    (70, 5, 32, 8, [300, 47, 1000, 64, 129], 32, 512, 16),
    (71, 6, 32, 8, [512, 512, 600, 1100, 513, 700], 512, 64, 256),
    (72, 3, 64, 8, [2100, 2048, 4000], 2048, 512, 1024),
    (73, 17, 32, 8, list(range(240, 240 + 17 * 13, 13)), 224, 512, 128),
    (74, 9, 16, 2, [100 + 37 * i for i in range(9)], 96, 128, 32),
    (75, 4, 8, 1, [16, 17, 33, 80], 16, 16, 16),
]


@pytest.mark.parametrize("case", CASCADE_CASES, ids=[f"seed{c[0]}" for c in CASCADE_CASES])
def test_cascade_edge_shapes(case):
    seed, B, hq, hkv, ctx, pre, S, Spre = case
    say(f"cascade edges seed={seed} B={B} Hq={hq} Hkv={hkv} prefix={pre} S={S} S_pre={Spre}")
    lc = logical_case(seed, B, hq, hkv, 128, ctx, prefix_len=pre)
    w = page_case(lc, seed + 1, extra_blocks=4)
    ref = decode_workload(w)[0]
    out = gpu_out(w, S, prefix_len=pre, prefix_partition_size=Spre)
    assert_gate(out, ref, f"cascade seed {seed}")
    # same result as the per-sequence path up to rounding
    plain = gpu_out(w, S)
    assert compare(out, bf16_to_f64(plain), gpu_is_bf16_bits=True).passed


def test_cascade_sequence_shorter_than_prefix():
    say("cascade with a sequence shorter than the prefix")
    lc = logical_case(80, 4, 32, 8, 128, [700, 520, 900, 512], prefix_len=512)
    w = page_case(lc, 81)
    w.context_lens = w.context_lens.copy()
    w.context_lens[1] = 492          # attends only to the first 492 prefix tokens
    w.context_lens[3] = 0            # empty
    ref = decode_workload(w)[0]
    out = gpu_out(w, 512, prefix_len=512, prefix_partition_size=128)
    assert np.all(out[3] & 0x7FFF == 0)
    assert_gate(out, ref, "cascade short sequence")


@pytest.mark.parametrize("where", ["prefix", "suffix"])
@pytest.mark.parametrize("hq", [32, 64])
def test_cascade_argmax_exact_slot(hq, where):
    """One dominant token -- in the shared prefix (every sequence must select
    the same slot) or in each sequence's own suffix -- is selected exactly;
    rows past the context and unused blocks are poisoned."""
    say(f"cascade argmax Hq={hq} target in {where}")
    ctx = [600, 700, 530, 1000]
    lc = logical_case(90, 4, hq, 8, 128, ctx, prefix_len=512)
    w = page_case(lc, 91, extra_blocks=6, poison=True)
    e0 = np.zeros(128, np.float32); e0[0] = 1.0
    w.q[:] = f32_to_bf16_bits(e0)
    nblk = (w.context_lens + 15) // 16
    for b in range(4):
        for j in range(nblk[b]):
            pid = int(w.block_tables[b, j])
            for r in range(min(16, int(w.context_lens[b]) - 16 * j)):
                w.k_pool[pid, :, r, :] = 0
                w.v_pool[pid, :, r, :] = 0
                w.v_pool[pid, :, r, 0:3] = f32_to_bf16_bits(np.float32([pid % 256, pid // 256, r]))
    targets = [300] * 4 if where == "prefix" else [599, 512, 529, 999]
    want = []
    for b, t in enumerate(targets):
        pid = int(w.block_tables[b, t // 16])
        w.k_pool[pid, :, t % 16, 0] = 0x4580   # 4096.0
        want.append((pid, t % 16))
    out = gpu_out(w, 512, prefix_len=512, prefix_partition_size=128)
    for b, (pid, r) in enumerate(want):
        got = bf16_to_f64(out[b, :, :3])
        assert np.all(got[:, 0] == pid % 256) and np.all(got[:, 1] == pid // 256) \
            and np.all(got[:, 2] == r), f"seq {b}: wanted slot ({pid},{r}), got {got[0]}"
        assert np.all(out[b, :, 3:] & 0x7FFF == 0)


# ------------------------------------------------ batch-independent partials

@pytest.mark.parametrize("S,lo,hi,B", [(128, 2000, 4500, 48), (512, 8000, 12000, 40),
                                       (1024, 15000, 17000, 40)])
def test_partials_do_not_depend_on_the_batch(S, lo, hi, B, oracle_pool):
    """A sequence's split-KV partials have the same bits whether it is decoded
    in a large batch (thousands of work items) or in a batch of three, and
    the large batch passes the gate."""
    from dataclasses import replace
    rng = np.random.default_rng(160 + S)
    ctx = rng.integers(lo, hi, size=B)
    say(f"batch-independent partials S={S}: {B} sequences of {lo}..{hi} tokens, G = 8")
    w = page_case(logical_case(160 + S, B, 64, 8, 128, ctx), 161, extra_blocks=7)
    pb = run(w, S)
    o, lse = pb.partials()
    out = pb.out_bits()
    pb.close()
    assert_gate(out, oracle_pool.decode_workload(w)[0], f"large batch S={S}")
    idx = [0, B // 2, B - 1]
    sub = replace(w, batch=3, q=w.q[idx], block_tables=w.block_tables[idx],
                  context_lens=w.context_lens[idx])
    pb = run(sub, S)
    o1, lse1 = pb.partials()
    pb.close()
    for i, b in enumerate(idx):
        P = -(-int(w.context_lens[b]) // S)
        assert np.array_equal(lse[b, :, :P], lse1[i, :, :P]), f"lse of sequence {b}"
        assert np.array_equal(o[b, :, :P], o1[i, :, :P]), f"partials of sequence {b}"
