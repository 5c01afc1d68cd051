"""The decode entry point that allocates nothing against paged_attn_decode.

paged_attn_decode_noalloc runs the same decode and reduce kernels as
paged_attn_decode + paged_attn_reduce with caller-provided partials, only
with the partials in the library's own scratch array, so its output must be
bit-identical; two calls in a row, the second on a smaller batch, check that
what the first call left in the array does not leak into the second.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import compare, decode_workload  # noqa: E402
from workloads import build_config, logical_case, page_case  # noqa: E402

DEV = "cuda:0"


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


def reference_and_noalloc(w, S):
    from paper_2510_14126_amd import binding
    from paper_2510_14126_amd.device import PagedBatch
    pb = PagedBatch(w, DEV, partition_size=S)
    pb.run()
    torch.cuda.synchronize()
    ref = pb.out_bits()
    out = torch.full_like(pb.out, -1)
    binding.paged_attn_decode_noalloc(pb.pool, pb.q, pb.bt, pb.bt_stride, pb.ctx, pb.batch, pb.hq,
                                      w.scale, pb.max_ctx, S, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    pb.close()
    return ref, got


def test_noalloc_matches_decode_two_calls_in_a_row():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    big = build_config(2)                      # 64 sequences, 5 partitions of 512 tokens
    small = page_case(logical_case(140, 5, 32, 8, 128, [700, 1, 0, 129, 1500]), 141, poison=True)
    for name, w, S in (("generator batch", big, 512), ("small batch", small, 256),
                       ("small batch, one pass", small, 0)):
        say(f"noalloc vs decode + reduce: {name}, S={S}")
        ref, got = reference_and_noalloc(w, S)
        diff = int(np.count_nonzero(ref != got))
        say(f"{name}: {diff} differing outputs of {ref.size}")
        assert diff == 0
        rep = compare(got, decode_workload(w)[0])
        say(f"{name} vs oracle: {rep}")
        assert rep.passed


def test_noalloc_g8_long_partitions():
    say("noalloc vs decode + reduce: G = 8, 4096-token contexts in 256-token partitions")
    w = page_case(logical_case(142, 6, 64, 8, 128, [4096, 4000, 17, 2049, 0, 3001]), 143)
    ref, got = reference_and_noalloc(w, 256)
    assert np.array_equal(ref, got)
    assert compare(got, decode_workload(w)[0]).passed
