"""Seeded random sweep of the decode entry points against the CPU oracle.

Each case draws a geometry (GQA 4 or 8, head_dim 64 or 128), a batch of
1-8 sequences with mixed lengths (block-boundary lengths included), a
partition size, optionally a shared prefix run through the cascade,
optionally a host-built work list and poisoned unused slots, and gates
every output against the oracle.  Every case prints its draw before it
touches the GPU.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import compare, decode_workload  # noqa: E402
from workloads import logical_case, page_case  # noqa: E402

DEV = "cuda:0"
GEOMETRIES = [(8, 2, 64), (16, 2, 64), (32, 8, 128), (64, 8, 128), (8, 1, 128), (4, 1, 128)]


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


def draw(seed):
    """Seeds from 16 on always run the cascade (head_dim 128 with a prefix)."""
    rng = np.random.default_rng(5000 + seed)
    geoms = GEOMETRIES if seed < 16 else [g for g in GEOMETRIES if g[2] == 128]
    hq, hkv, d = geoms[int(rng.integers(len(geoms)))]
    batch = int(rng.integers(1, 9))
    ctx = []
    for _ in range(batch):
        kind = rng.random()
        if kind < 0.15:
            n = 1
        elif kind < 0.45:
            n = 16 * int(rng.integers(1, 100)) + int(rng.integers(-1, 2))
        else:
            n = int(rng.integers(2, 2500))
        ctx.append(max(1, n))
    prefix = 0
    if d == 128 and (seed >= 16 or rng.random() < 0.5):
        prefix = 16 * int(rng.integers(1, 129))              # up to 2048 tokens
        ctx = [max(n, prefix + int(rng.integers(0, 600))) for n in ctx]
    S = [0, 16, 64, 256, 512][int(rng.integers(5))]
    if prefix and S == 0:
        S = 256
    spre = 16 * int(rng.integers(1, 65))
    schedule = bool(rng.random() < 0.5)
    poison = bool(rng.random() < 0.5)
    return dict(hq=hq, hkv=hkv, d=d, ctx=ctx, prefix=prefix, S=S, spre=spre, schedule=schedule,
                poison=poison)


@pytest.mark.parametrize("seed", range(32))
def test_random_decode_against_oracle(seed):
    c = draw(seed)
    say(f"random seed={seed}: {c}")
    lc = logical_case(6000 + seed, len(c["ctx"]), c["hq"], c["hkv"], c["d"], c["ctx"],
                      prefix_len=c["prefix"])
    w = page_case(lc, 7000 + seed, share_prefix=c["prefix"] > 0, poison=c["poison"], extra_blocks=4)
    ref = decode_workload(w)[0]
    from paper_2510_14126_amd.device import PagedBatch
    kw = dict(schedule=c["schedule"])
    if c["prefix"]:
        kw.update(prefix_len=c["prefix"], prefix_partition_size=c["spre"])
    pb = PagedBatch(w, DEV, partition_size=c["S"], **kw)
    pb.run()
    torch.cuda.synchronize()
    out = pb.out_bits()
    pb.close()
    rep = compare(out, ref)
    say(f"random seed={seed}: {rep}")
    assert rep.passed, f"seed {seed} {c}: {rep}"
