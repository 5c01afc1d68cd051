"""GPU parity tests of the extend (chunked prefill) attention against the CPU
oracle.  Every case prints its name before touching the GPU.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import compare, extend_attention, paged_decode  # noqa: E402
from oracle.attention import bf16_to_f64  # noqa: E402
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


def make_extend(seed, ctx, chunk, hq=32, hkv=8, prefix_len=0, poison=False):
    ctx, chunk = list(map(int, ctx)), list(map(int, chunk))
    case = logical_case(seed, len(ctx), hq, hkv, 128, ctx, prefix_len=prefix_len)
    w = page_case(case, seed + 1, share_prefix=prefix_len > 0, poison=poison)
    rng = np.random.default_rng(seed + 2)
    q_start = np.concatenate([[0], np.cumsum(chunk)]).astype(np.int32)
    q = f32_to_bf16_bits(rng.standard_normal((int(q_start[-1]), hq, 128), dtype=np.float32))
    return w, q, q_start


def gpu_extend(w, q, q_start, max_chunk=None):
    from paper_2510_14126_amd import binding
    total = int(q_start[-1])
    max_chunk = int(np.max(np.diff(q_start))) if max_chunk is None else max_chunk
    k_dev, v_dev = _dev(w.k_pool), _dev(w.v_pool)
    pool = binding.kv_pool_create(w.num_blocks, 16, w.num_kv_heads, 128, k_dev, v_dev)
    out = torch.zeros((max(total, 1), w.num_q_heads, 128), dtype=torch.int16, device=DEV)
    q_dev = _dev(q) if total else out
    binding.paged_attn_extend(pool, q_dev, _dev(q_start), total, _dev(w.block_tables),
                              int(w.block_tables.shape[1]), _dev(w.context_lens), w.batch,
                              w.num_q_heads, w.scale, int(w.context_lens.max()), max_chunk, out)
    torch.cuda.synchronize()
    pool.close()
    return out[:total].cpu().numpy().view(np.uint16)


def check(w, q, q_start, what, **kw):
    out = gpu_extend(w, q, q_start, **kw)
    ref, _ = extend_attention(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale)
    rep = compare(out, ref)
    say(f"{what}: {rep}")
    assert rep.passed, f"{what}: {rep}"
    return out


@pytest.mark.parametrize("hq", [32, 64], ids=["g4", "g8"])
def test_extend_fixer_shaped(hq):
    """Retries of one request: a shared schema prefix, a first attempt, and a
    chunk of new tokens per retry that attends to both and to itself."""
    rng = np.random.default_rng(50)
    B = 12
    chunk = rng.integers(32, 257, B)
    ctx = 512 + 64 + chunk
    say(f"extend fixer-shaped hq={hq}: B={B} chunks={chunk.tolist()}")
    w, q, q_start = make_extend(51, ctx, chunk, hq=hq, prefix_len=512)
    check(w, q, q_start, f"fixer-shaped g{hq // 8}")


CASES = [
    ("fresh prefill", [1, 15, 16, 17, 100], [1, 15, 16, 17, 100]),
    ("one-token chunks", [5, 300, 1000], [1, 1, 1]),
    ("ragged with an empty chunk", [40, 10, 21, 77], [3, 0, 21, 64]),
    ("chunk across many tiles", [700], [300]),
    # unmasked-stage count even, odd (rounded down to the ring's two slot
    # sets) and equal to the whole stream, and long chunks whose workgroups
    # cross the causal diagonal at different stages
    ("diagonal and ring parity", [64, 96, 1024, 1056, 333], [1, 1, 200, 37, 129]),
]


@pytest.mark.parametrize("hq", [32, 64], ids=["g4", "g8"])
@pytest.mark.parametrize("name,ctx,chunk", CASES, ids=[c[0] for c in CASES])
def test_extend_edge_shapes(name, ctx, chunk, hq):
    say(f"extend {name} hq={hq}: ctx={ctx} chunk={chunk}")
    w, q, q_start = make_extend(61, ctx, chunk, hq=hq, poison=True)
    check(w, q, q_start, f"{name} g{hq // 8}")


def test_extend_loose_max_chunk_bound():
    say("extend with max_chunk above every chunk")
    w, q, q_start = make_extend(71, [90, 33], [40, 33])
    check(w, q, q_start, "loose bound", max_chunk=90)


def test_one_token_extend_matches_gpu_decode():
    from paper_2510_14126_amd.device import PagedBatch
    say("extend with one-token chunks vs the decode kernel")
    w, q, q_start = make_extend(81, [200, 513, 47], [1, 1, 1])
    ext = gpu_extend(w, q, q_start)
    w.q = q.copy()
    pb = PagedBatch(w, DEV, partition_size=0)
    pb.run()
    torch.cuda.synchronize()
    dec = pb.out_bits()
    pb.close()
    ref, _ = paged_decode(q, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale)
    assert compare(ext, ref).passed and compare(dec, ref).passed
    diff = np.abs(ext.astype(np.int32) - dec.astype(np.int32))
    say(f"extend vs decode: max bf16 ulp difference {int(diff.max())}")


@pytest.mark.parametrize("factor", [-1.0, 0.0], ids=["negative", "zero"])
def test_extend_scale_sign(factor):
    """A negative scale (carried by the sign of Q inside the kernel) and a zero
    scale (uniform weights over the visible tokens), with masked tails."""
    ctx, chunk = [333, 64, 1056], [129, 1, 37]
    say(f"extend scale x{factor}: ctx={ctx} chunk={chunk}")
    w, q, q_start = make_extend(71, ctx, chunk, poison=True)
    w.scale = float(w.scale) * factor
    check(w, q, q_start, f"scale x{factor}")


LONG = [
    # contexts in (4096, 8192] (exactly 8192 included), chunks of at least 1024
    # tokens: the block-id staging takes a second pass above 4096 tokens
    ("long contexts", [8192, 6000, 4097, 7777], [1024, 2000, 1100, 1500]),
    ("one full-length chunk", [8192], [8192]),
]


@pytest.mark.parametrize("hq", [32, 64], ids=["g4", "g8"])
@pytest.mark.parametrize("name,ctx,chunk", LONG, ids=[c[0] for c in LONG])
def test_extend_long_contexts(name, ctx, chunk, hq, oracle_pool):
    say(f"extend {name} hq={hq}: ctx={ctx} chunk={chunk}")
    w, q, q_start = make_extend(91, ctx, chunk, hq=hq, prefix_len=2048, poison=True)
    out = gpu_extend(w, q, q_start)
    ref, _ = oracle_pool.extend(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens,
                                w.scale)
    rep = compare(out, ref)
    say(f"{name} g{hq // 8}: {rep}")
    assert rep.passed, f"{name}: {rep}"


@pytest.mark.parametrize("k", [2, 3])
def test_extend_bench_batches_all_rows(k, stage_batches, oracle_pool):
    """The batches bench.py --extend times (each sequence's tokens after its
    shared prompt as the chunk, its seeded queries), every output row."""
    import bench
    w = stage_batches.workload(k)
    chunk, q_start, q = bench.extend_inputs(w)
    say(f"extend bench batch config {k}: {int(q_start[-1])} rows, chunks "
        f"{int(chunk.min())}..{int(chunk.max())}")
    out = gpu_extend(w, q, q_start)
    ref, _ = oracle_pool.extend(q, q_start, w.k_pool, w.v_pool, w.block_tables, w.context_lens,
                                w.scale)
    rep = compare(out, ref)
    say(f"extend bench batch config {k}, all rows: {rep}")
    assert rep.passed, f"config {k}: {rep}"


def _extend_argmax(ctx, chunk, targets, hq):
    """Every chunk row's query is e0; K of one cached target token is 4096 e0
    and K of each sequence's last token 8192 e0, every other used slot K = 0;
    V encodes the physical slot (block mod 256, block div 256, row) as exact
    bf16 integers.  Rows past the context and unused blocks hold K = 8192 e0
    and V = NaN.  So chunk row i must return exactly V[target] if it does
    not see the last token (i < L - 1, causal mask) and V[last] if it does."""
    w, q, q_start = make_extend(77, ctx, chunk, hq=hq, poison=True)
    e0 = np.zeros(128, np.float32)
    e0[0] = 1.0
    q[:] = f32_to_bf16_bits(e0)
    nblk = (w.context_lens + 15) // 16
    used = {(int(w.block_tables[b, j]), r) for b in range(w.batch) for j in range(nblk[b])
            for r in range(min(16, int(w.context_lens[b]) - 16 * j))}
    for (pid, r) in used:
        w.k_pool[pid, :, r, :] = 0
        w.v_pool[pid, :, r, :] = 0
        w.v_pool[pid, :, r, 0:3] = f32_to_bf16_bits(np.float32([pid % 256, pid // 256, r]))
    want = []
    for b, t in enumerate(targets):
        n, L = int(ctx[b]), int(chunk[b])
        assert t < n - L, "the target lies in the cached context, seen by every chunk row"
        slot_t = (int(w.block_tables[b, t // 16]), t % 16)
        slot_l = (int(w.block_tables[b, (n - 1) // 16]), (n - 1) % 16)
        w.k_pool[slot_t[0], :, slot_t[1], 0] = 0x4580   # 4096.0
        w.k_pool[slot_l[0], :, slot_l[1], 0] = 0x4600   # 8192.0
        want.append((slot_t, slot_l))
    return w, q, q_start, want


@pytest.mark.parametrize("hq", [32, 64], ids=["g4", "g8"])
def test_extend_argmax_reads_exact_slot_and_causal_mask(hq):
    ctx = [40, 513, 1024, 4100, 8192]
    chunk = [1, 17, 512, 1000, 2048]
    targets = [16, 495, 0, 3099, 4096]
    say(f"extend argmax slot selection and causal mask Hq={hq}")
    w, q, q_start, want = _extend_argmax(ctx, chunk, targets, hq)
    out = gpu_extend(w, q, q_start)
    for b, (slot_t, slot_l) in enumerate(want):
        rows = out[q_start[b]:q_start[b + 1]]
        codes = np.stack([np.asarray([s[0] % 256, s[0] // 256, s[1]], np.float64)
                          for s in (slot_t, slot_l)])
        got = bf16_to_f64(rows[:, :, :3])
        L = rows.shape[0]
        assert np.all(got[:L - 1] == codes[0]), f"seq {b}: rows before the last must read {slot_t}"
        assert np.all(got[L - 1] == codes[1]), f"seq {b}: the last row must read {slot_l}"
        assert np.all(rows[:, :, 3:] & 0x7FFF == 0)
