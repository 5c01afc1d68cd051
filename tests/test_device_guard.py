"""Host-side guards of the device layer (CPU only): a pool tensor smaller
than the geometry the pool handle will declare is refused before anything is
launched -- the library clamps block ids to the declared pool, so it cannot
tell a short buffer from a full one."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads import logical_case, page_case  # noqa: E402


def test_short_pool_tensor_is_refused():
    from paper_2510_14126_amd.device import PagedBatch
    w = page_case(logical_case(3, 2, 8, 2, 64, [40, 17]), 4)
    need = w.num_blocks * w.num_kv_heads * 16 * w.head_dim
    short = torch.zeros(need - 16 * w.head_dim, dtype=torch.int16)
    full = torch.zeros(need, dtype=torch.int16)
    with pytest.raises(ValueError, match="k_pool"):
        PagedBatch(w, "cpu", k_pool=short, v_pool=full, register_blocks=False)
    with pytest.raises(ValueError, match="v_pool"):
        PagedBatch(w, "cpu", k_pool=full, v_pool=short, register_blocks=False)


def test_replica_timing_refuses_mismatched_pool_values():
    import bench
    from workloads import stage_units
    deps = bench.footprint_deployments(1024, stage_units(9, 200))
    rep = deps["isolated"][1]
    k = np.zeros((1024, 8, 16, 128), np.uint16)              # budget != 1024
    assert rep.budget != 1024
    with pytest.raises(ValueError, match="replica"):
        bench._time_replica(rep, k, k, 1, 0, 0)
    for reps in deps.values():
        for r in reps:
            r.close()
