"""Worst case for the precision of the softmax weights: the near-tie input of
tests/precision_case.py (weights near 0.5 that straddle bf16 rounding points,
correlated with the sign of V, over contexts up to 32k tokens), through every
decode path, gated against the oracle.  Weights rounded to bf16 before the PV
product fail this gate; the kernels carry each weight as a bf16 pair (high
and low part) and the row sums in fp32."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import compare, decode_workload  # noqa: E402
from precision_case import near_tie_case  # noqa: E402

DEV = "cuda:0"
CTX = [32768, 4099, 513, 16, 1]


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    yield
    torch.cuda.empty_cache()


def gated(w, what, S, **kw):
    from paper_2510_14126_amd.device import PagedBatch
    pb = PagedBatch(w, DEV, partition_size=S, **kw)
    pb.run()
    torch.cuda.synchronize()
    out = pb.out_bits()
    pb.close()
    rep = compare(out, decode_workload(w)[0])
    say(f"{what}: {rep}")
    assert rep.passed, f"{what}: {rep}"


@pytest.mark.parametrize("S", [512, 0])
@pytest.mark.parametrize("hq", [32, 64], ids=["g4_valu", "g8_mfma"])
def test_near_ties_split_and_single_pass(hq, S):
    ctx = CTX if S else [4099, 513, 16, 1]
    w = near_tie_case(ctx, hq=hq, hkv=8, seed=150)
    say(f"near-tie weights Hq={hq} S={S} ctx={ctx}")
    gated(w, f"near ties Hq={hq} S={S}", S)


@pytest.mark.parametrize("hq", [32, 64], ids=["g4", "g8"])
def test_near_ties_cascade(hq):
    w = near_tie_case(CTX[:3], hq=hq, hkv=8, seed=151, prefix_len=512)
    say(f"near-tie weights, cascade over a 512-token shared prefix, Hq={hq}")
    gated(w, f"near ties cascade Hq={hq}", 512, prefix_len=512, prefix_partition_size=256,
          schedule=True)
