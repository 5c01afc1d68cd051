"""Host-side block accounting of the footprint experiment (CPU only): the
pool allocator's blocks in use equal the distinct blocks the tables map, with
shared prompt blocks counted once, and equal the sum of per-sequence block
counts once every sequence holds private copies."""
import numpy as np

import bench
from workloads import build_config, duplicate_shared_blocks, logical_case, page_case


def test_stage_batches_count_shared_blocks_once():
    for k in (2, 3):
        w = build_config(k, values=False)
        assert bench._blocks_in_use(w) == w.meta["needed_blocks"]


def test_private_copies_count_every_sequence():
    case = logical_case(5, 6, 8, 2, 64, [40, 70, 33, 64, 100, 48], prefix_len=32)
    w = page_case(case, 6, share_prefix=True)
    shared = bench._blocks_in_use(w)
    wd = duplicate_shared_blocks(w)
    private = bench._blocks_in_use(wd)
    per_seq = int(((w.context_lens + 15) // 16).sum())
    assert private == per_seq
    assert shared == per_seq - (w.batch - 1) * (32 // 16)


def test_bench_launch_configurations():
    """The launch bench.py times: stated 512-token partitions on the
    long-context pool, the cascade wherever a prefix is shared, request groups
    on the fixer batch."""
    expect = {1: (512, None, False), 2: (512, 2048, False), 3: (1024, 2048, True),
              4: (8192, None, False), 5: (512, 4096, False)}
    for k, (S, L, groups) in expect.items():
        w = build_config(k, values=False)
        s, kw = bench.launch_configuration(k, w)
        assert s == S
        assert kw.get("prefix_len") == L
        assert ("group_len" in kw) == groups
    w = build_config(5, values=False)
    assert bench.launch_configuration(5, w)[1]["prefix_partition_size"] == 512
    assert bench.launch_configuration(5, w, cascade="off")[1] == {}


def _nb(t):
    return -(-t // 16)


def test_deployments_under_a_fixed_kv_budget():
    """Host accounting of the isolated / shared / private deployments: the
    same total budget, whole requests (a generator call and a fixer request)
    admitted in order, every replica within its budget, each stage's prompt
    resident once per replica that serves the stage (referenced by every
    sequence that maps it), exactly the blocks the sequences need; isolation
    admits the most requests."""
    from paper_2510_14126_amd import binding
    from workloads import FIRST_ATTEMPT, stage_units
    M = 1024
    deps = bench.footprint_deployments(M, stage_units(7, 600))
    requests = {}
    for kind, reps in deps.items():
        assert sum(r.budget for r in reps) == 2 * M
        requests[kind] = sum(len(r.groups) for r in reps)
        for r in reps:
            assert r.blocks_used() <= r.budget
            if not (r is deps["isolated"][0] or r is deps["isolated"][1]):
                assert len(r.seqs["generator"]) == len(r.groups)    # one generator call per request
            expect = r.prompt_blocks
            for st, rows in r.seqs.items():
                for ids, n in rows:
                    assert len(ids) == _nb(n)
                    assert len(set(ids)) == len(ids)
                    if r.private:
                        expect += _nb(n)
                    else:
                        expect += _nb(n) - 128 - (FIRST_ATTEMPT // 16 if st == "fixer" else 0)
            if not r.private:
                expect += len(r.groups) * (FIRST_ATTEMPT // 16)
            assert r.blocks_used() == expect, kind
            for st, ids in r.prompt.items():
                assert binding.kv_pool_refcount(r.pool, ids[0]) == 1 + len(r.seqs[st])
    gen, fix = deps["isolated"]
    assert gen.prompt_blocks == 128 and fix.prompt_blocks == 128
    assert all(r.prompt_blocks == 256 for r in deps["shared"])
    assert all(r.prompt_blocks == 0 for r in deps["private"])
    assert len(fix.seqs["generator"]) == 0 and len(gen.seqs["fixer"]) == 0
    assert len(gen.seqs["generator"]) == len(fix.groups)           # the same requests
    for r in deps["shared"] + deps["private"]:                      # both stages on each replica
        assert len(r.seqs["generator"]) > 0 and len(r.seqs["fixer"]) > 0
    assert requests["isolated"] >= requests["shared"] > requests["private"] > 0
    for reps in deps.values():
        for r in reps:
            r.close()
