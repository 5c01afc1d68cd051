"""Benchmark of one decode step of paged decode attention on one MI355X.

A step is one pass of the whole hot path over one batch: the split-KV decode
(for batches that share a schema prefix, the one-launch cascade: a
matrix-core pass over the shared prefix for all query rows plus the
per-sequence decode of the tokens after it) followed by the cross-split
reduce, for every sequence and head of the batch.

Workloads (seeded synthetic bf16 N(0,1) inputs, 16-token blocks, one layer):
the headline line is the long-context stage pool (batch 128, 64 query / 8 KV
heads, head_dim 128, contexts 8192..32768 tokens with a shared 4096-token
prefix, 512-token split-KV partitions), the largest of the five stage-shaped
batches; the same line carries a ``per_config`` entry for each of the other
four (tiny, SQL generator, SQL error fixer, shared pool), each with its own
step time, roofline fraction, parity spot check and CPU-oracle baseline.
``--config k`` measures batch k alone.

Timing: the pools and queries are replicated R times in HBM (R copies of the
same data at different addresses, like R layers of a model) and consecutive
steps rotate through them, so a step does not find its working set in the
256 MB Infinity Cache left over from the previous step.  W warmup steps,
then K timed steps bracketed by device synchronisation; per-kernel durations
come from HIP events around K back-to-back launches of each kernel on the
launch stream.

Output: exactly one JSON line on stdout.  `value` is KV GB/s counting the
algorithmic bytes of a step (each distinct cached token slot once, plus
queries, outputs, block tables and lengths) over the measured step time.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1..5]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
PROFILE_DIR = os.path.join(ROOT, "profiles")
_CSRC = "paper_2510_14126_amd/csrc/"
KERNEL_SOURCES = {
    "decode_valu": [_CSRC + f for f in ("decode_valu.hip", "valu_body.h", "pa_device.h", "kernels.h")],
    "decode_mfma": [_CSRC + f for f in ("decode_mfma.hip", "mfma_body.h", "pa_device.h", "kernels.h")],
    "cascade": [_CSRC + f for f in ("cascade.hip", "valu_body.h", "mfma_body.h", "pa_device.h",
                                    "kernels.h")],
    "reduce": [_CSRC + f for f in ("reduce.hip", "pa_device.h", "kernels.h")],
    "append": [_CSRC + f for f in ("append.hip", "pa_device.h", "kernels.h")],
    "extend": [_CSRC + f for f in ("extend.hip", "mfma_body.h", "pa_device.h", "kernels.h")],
    "gather_tiles": [_CSRC + f for f in ("gather_tiles.hip", "pa_device.h", "kernels.h")],
    "stream_copy": [_CSRC + f for f in ("stream_copy.hip", "kernels.h")],
}
LIBRARY_PATH = os.path.join(ROOT, "paper_2510_14126_amd", "libpaged_attn.so")
HEADLINE_CONFIG = 5            # the largest single-GPU stage batch (long-context pool)
PER_CONFIG = (1, 2, 3, 4)      # the other stage batches, reported in the same line
# Split-KV partition sizes used when --partition-size is not given.  The
# long-context pool states 512-token partitions; the other workloads state
# none and use the size that measured fastest on them with the host-built
# work list (the shared pool: one partition of up to 8192 tokens, no reduce).
DEFAULT_PARTITION = {1: 512, 2: 512, 3: 1024, 4: 8192, 5: 512}


# Prefix partition sizes (tokens) used when --prefix-partition-size is not
# given: the size that measured fastest on each workload with a shared prefix.
DEFAULT_PREFIX_PARTITION = {2: 512, 3: 1024, 5: 512}


def default_prefix_partition(config: int, prefix_len: int) -> int:
    size = DEFAULT_PREFIX_PARTITION.get(config, 1024)
    return max(16, min(size, -(-prefix_len // 16) * 16))


def launch_configuration(k, w, partition_size=None, prefix_partition_size=None, cascade="auto",
                         groups="auto"):
    """Partition size and PagedBatch keywords of the launch this benchmark
    times on workload k: the stated or measured-fastest partition size; the
    shared-prefix cascade when the batch shares a prefix; request groups when
    its sequences also share tokens per group after the prefix."""
    from workloads import group_starts
    S = partition_size or DEFAULT_PARTITION.get(k, w.partition_size)
    L = 16 * int(w.meta.get("prefix_blocks", 0))
    if cascade == "off" or (cascade == "auto" and L == 0):
        L = 0
    M = 16 * int(w.meta.get("mid_blocks", 0)) if "groups" in w.meta else 0
    if groups == "on" and (M == 0 or L == 0):
        raise SystemExit("--groups on: this workload has no groups sharing tokens after the prefix")
    kw = {}
    if L:
        kw = dict(prefix_len=L, prefix_partition_size=prefix_partition_size or default_prefix_partition(k, L))
        if M and groups != "off":
            kw.update(group_start=group_starts(w), group_len=M)
    return S, kw


def decode_kernel_of(w, prefix_len: int = 0) -> str:
    """Which decode kernel the library launches for this geometry."""
    if prefix_len:
        return "cascade"
    return "decode_mfma" if (w.group == 8 and w.head_dim == 128) else "decode_valu"


def kernel_display_name(w, kernel: str) -> str:
    return {"cascade": f"cascade_kernel<{w.group}>", "decode_mfma": "decode_mfma_g8_kernel",
            "decode_valu": f"decode_valu_kernel<{w.head_dim},{w.group}>"}[kernel]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash(kernel: str = "decode_valu") -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def library_source_hash() -> str:
    """Hash of every source of the library (kernels, C ABI, header)."""
    csrc = os.path.join(ROOT, _CSRC)
    files = sorted(os.path.join(csrc, f) for f in os.listdir(csrc))
    files.append(os.path.join(ROOT, "include", "paged_attn.h"))
    h = hashlib.sha256()
    for p in files:
        with open(p, "rb") as f:
            h.update(os.path.basename(p).encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def source_stamp() -> dict:
    """What a profiled run was built from: written by the run itself
    (--profile-loop --stamp) and checked when its results are ingested."""
    lib = None
    if os.path.exists(LIBRARY_PATH):
        with open(LIBRARY_PATH, "rb") as f:
            lib = hashlib.sha256(f.read()).hexdigest()[:16]
    return {"library_source_sha256_16": library_source_hash(),
            "kernel_source_sha256_16": {k: kernel_source_hash(k) for k in KERNEL_SOURCES},
            "library_sha256_16": lib}


def checked_stamp(path) -> dict:
    """The stamp of a profiled run; refuses one taken on other sources."""
    if not path:
        raise SystemExit("ingest needs --stamp: the source stamp the profiled run wrote")
    with open(path) as f:
        st = json.load(f)
    cur = library_source_hash()
    if st.get("library_source_sha256_16") != cur:
        raise SystemExit(f"profile stamp {st.get('library_source_sha256_16')} does not match the "
                         f"current library sources {cur}: profile again")
    return st


def byte_accounting(w):
    from workloads import logical_tokens, touched_slots
    per_tok = w.bytes_per_token
    qo = 2 * (w.batch * w.num_q_heads * w.head_dim * 2)               # q in + out
    meta = 4 * w.batch + 4 * int(w.blocks_per_seq().sum())              # lengths + table entries read
    alg = touched_slots(w) * per_tok + qo + meta
    logical = logical_tokens(w) * per_tok + qo + meta
    return alg, logical


# --------------------------------------------------------------- CPU baseline

_W = None


def _oracle_chunk(seqs):
    from threadpoolctl import threadpool_limits
    from oracle import decode_workload
    with threadpool_limits(1):
        decode_workload(_W, seqs=seqs)
    return len(seqs)


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, alg_bytes, min_seconds=10.0, logical_bytes=None):
    """Time the CPU oracle on whole decode steps of the same batch.

    The oracle runs over the batch's sequences in a process pool (one BLAS
    thread per worker) and the step is repeated until min_seconds pass.
    Called before the process touches the GPU: the pool is forked.  Workers:
    the CPUs this process may use, at most 16, the host share of one GPU.
    """
    import multiprocessing as mp
    global _W
    _W = w
    affinity = len(os.sched_getaffinity(0))
    cores = max(1, min(16, affinity))
    chunks = [list(range(i, w.batch, cores)) for i in range(cores)]
    chunks = [c for c in chunks if c]
    ctx = mp.get_context("fork")
    steps = 0
    pool = ctx.Pool(len(chunks))
    try:
        pool.map(_oracle_chunk, [chunks[0][:1]])                   # workers up
        t0 = time.perf_counter()
        while True:
            pool.map(_oracle_chunk, chunks)
            steps += 1
            el = time.perf_counter() - t0
            if el >= min_seconds:
                break
    finally:
        pool.close()
        pool.join()
    _W = None
    sec_per_step = el / steps
    return {"value": round(alg_bytes / sec_per_step / 1e9, 4), "unit": "GB/s", "cores": len(chunks),
            "kind": "oracle", "sample": f"{steps} full decode steps of the same batch "
            f"({w.batch} sequences) in {el:.1f} s; fp64 numpy oracle, process pool, "
            f"1 BLAS thread per worker", "seconds_per_step": round(sec_per_step, 4),
            "decode_steps_per_s": round(1.0 / sec_per_step, 3),
            "logical_kv_gbps": (round(logical_bytes / sec_per_step / 1e9, 4)
                                if logical_bytes else None),
            "affinity_cpus": affinity, "cpu_model": _cpu_model(), "numpy": np.__version__}


# ------------------------------------------------------------------ traffic

def traffic_from_profiles(workload_name, kernel="decode_valu"):
    """Counter-derived HBM bytes per decode launch, if the profile summary was
    taken on the current kernel source; else None."""
    path = os.path.join(PROFILE_DIR, f"{kernel}_{workload_name}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_src = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    m_tr = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_src or not m_tr or m_src.group(1) != kernel_source_hash(kernel):
        return None
    return float(m_tr.group(1))


def ingest_counters(fetch_csv, write_csv, workload_name, kernel_prefix, command_note, stamp):
    """Write the traffic summary from two rocprofv3 --pmc CSVs (FETCH_SIZE, WRITE_SIZE).

    Each counter is scaled by what it reads for the calibration copy of
    268435456 bytes each way (pa_stream_copy) in the same run.
    """
    import csv
    import collections
    from workloads import CONFIG_NAMES, build_config
    k = [c for c, n in CONFIG_NAMES.items() if n == workload_name][0]
    alg, _ = byte_accounting(build_config(k, values=False))
    res = {}
    for path, cname in ((fetch_csv, "FETCH_SIZE"), (write_csv, "WRITE_SIZE")):
        per = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == cname:
                per[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        copy = [v for n, v in per.items() if "stream_copy_kernel" in n][0]
        kern = [(n, v) for n, v in per.items() if kernel_prefix + "_" in n]
        if not kern:
            raise SystemExit(f"no {kernel_prefix} dispatches in {path}")
        name, vals = kern[0]
        factor = (268435456 / 1024) / (sum(copy) / len(copy))
        res[cname] = dict(kernel=name, n=len(vals), mean_kib=sum(vals) / len(vals),
                          copy_kib=sum(copy) / len(copy), factor=factor)
    f, wr = res["FETCH_SIZE"], res["WRITE_SIZE"]
    fetched = f["mean_kib"] * f["factor"] * 1024
    written = wr["mean_kib"] * wr["factor"] * 1024
    out = os.path.join(PROFILE_DIR, f"{kernel_prefix}_{workload_name}_counters.md")
    with open(out, "w") as fh:
        fh.write(f"# HBM traffic counters: {f['kernel']} on the {workload_name} workload\n\n"
                 f"Commands (run from /tmp with TMPDIR=/tmp):\n\n{command_note}\n\n"
                 "Calibration: pa_stream_copy of 268435456 bytes read + 268435456 bytes written "
                 "in the same runs.\n\n"
                 f"| counter | calibration copy reads (KiB) | factor | kernel mean (KiB/dispatch) | "
                 f"dispatches | scaled bytes/dispatch |\n|---|---|---|---|---|---|\n"
                 f"| FETCH_SIZE | {f['copy_kib']:.1f} | {f['factor']:.4f} | {f['mean_kib']:.2f} | "
                 f"{f['n']} | {fetched:,.0f} |\n"
                 f"| WRITE_SIZE | {wr['copy_kib']:.1f} | {wr['factor']:.4f} | {wr['mean_kib']:.2f} | "
                 f"{wr['n']} | {written:,.0f} |\n\n"
                 f"algorithmic_bytes_per_launch: {alg}\n"
                 f"traffic_bytes_per_launch: {fetched + written:.6e}\n"
                 f"traffic_over_algorithmic: {(fetched + written) / alg:.4f}\n"
                 f"kernel_source_sha256_16: {stamp['kernel_source_sha256_16'][kernel_prefix]}\n"
                 f"library_source_sha256_16: {stamp['library_source_sha256_16']}\n")
    print(out)


def ingest_sq(csv_paths, workload_name, kernel_substr, command_note, stem, stamp):
    """Write a per-dispatch summary of SQ (shader sequencer) counters for one kernel."""
    import csv
    import collections
    m, n = {}, 0
    name = None
    for path in csv_paths:
        per = collections.defaultdict(lambda: collections.defaultdict(list))
        for r in csv.DictReader(open(path)):
            per[r["Kernel_Name"]][r["Counter_Name"]].append(float(r["Counter_Value"]))
        ks = [k for k in per if kernel_substr in k]
        if not ks:
            raise SystemExit(f"no {kernel_substr} dispatches in {path}")
        name = ks[0]
        for c, v in per[name].items():
            m[c] = sum(v) / len(v)
            n = len(v)
    simds = 1024                      # 256 CUs x 4 SIMDs
    xcds = 8
    lines = []
    if "GRBM_GUI_ACTIVE" in m and "SQ_VALU_MFMA_BUSY_CYCLES" in m:
        gpu_cycles = m["GRBM_GUI_ACTIVE"] / xcds
        lines.append(f"| matrix-core busy (SQ_VALU_MFMA_BUSY_CYCLES / (SIMDs x GRBM_GUI_ACTIVE per XCD)) | "
                     f"{100 * m['SQ_VALU_MFMA_BUSY_CYCLES'] / (simds * gpu_cycles):.1f}% |")
    if "SQ_WAVE_CYCLES" in m:
        for c, label in (("SQ_WAIT_INST_ANY", "wave cycles waiting on an instruction dependency"),
                         ("SQ_WAIT_INST_LDS", "wave cycles waiting on LDS"),
                         ("SQ_ACTIVE_INST_VALU", "wave cycles issuing VALU"),
                         ("SQ_ACTIVE_INST_LDS", "wave cycles issuing LDS")):
            if c in m:
                lines.append(f"| {label} ({c} / SQ_WAVE_CYCLES) | {100 * m[c] / m['SQ_WAVE_CYCLES']:.1f}% |")
    if "SQ_LDS_BANK_CONFLICT" in m and "SQ_LDS_IDX_ACTIVE" in m:
        lines.append(f"| LDS bank-conflict cycles / LDS active cycles | "
                     f"{100 * m['SQ_LDS_BANK_CONFLICT'] / max(1.0, m['SQ_LDS_IDX_ACTIVE']):.1f}% |")
    if "SQ_INSTS_VALU" in m and "SQ_INSTS_MFMA" in m and m["SQ_INSTS_MFMA"] > 0:
        lines.append(f"| VALU instructions per MFMA | {m['SQ_INSTS_VALU'] / m['SQ_INSTS_MFMA']:.2f} |")
    out = os.path.join(PROFILE_DIR, f"{stem}.md")
    with open(out, "w") as fh:
        fh.write(f"# SQ counters: {name} on the {workload_name} workload\n\n"
                 f"Commands (run from /tmp with TMPDIR=/tmp):\n\n{command_note}\n\n"
                 f"Per-dispatch means over {n} dispatches (whole GPU).\n\n"
                 "| counter | per dispatch |\n|---|---|\n")
        for c in sorted(m):
            fh.write(f"| {c} | {m[c]:,.0f} |\n")
        fh.write("\n| derived | value |\n|---|---|\n" + "\n".join(lines) + "\n")
        fh.write(f"\nlibrary_source_sha256_16: {stamp['library_source_sha256_16']}\n")
    print(out)


def ingest_stats(stats_csv, workload_name, command_note, stamp, stem=None):
    """Write the kernel-duration summary from a rocprofv3 --stats kernel_stats.csv."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    out = os.path.join(PROFILE_DIR, f"{stem or f'kernels_{workload_name}_stats'}.md")
    with open(out, "w") as fh:
        fh.write(f"# Kernel durations on the {workload_name} workload (rocprofv3 --kernel-trace --stats)\n\n"
                 f"Command (run from /tmp with TMPDIR=/tmp):\n\n{command_note}\n\n"
                 "| kernel | calls | average (us) | min (us) | max (us) | share |\n|---|---|---|---|---|---|\n")
        for r in rows:
            fh.write(f"| `{r['Name'][:90]}` | {r['Calls']} | {float(r['AverageNs'])/1e3:.2f} | "
                     f"{float(r['MinNs'])/1e3:.2f} | {float(r['MaxNs'])/1e3:.2f} | {float(r['Percentage']):.1f}% |\n")
        fh.write("".join(f"\nkernel_source_sha256_16 ({k}): {h}"
                         for k, h in stamp["kernel_source_sha256_16"].items()) +
                 f"\nlibrary_source_sha256_16: {stamp['library_source_sha256_16']}\n")
    print(out)


# ------------------------------------------------------------------ extend

MFMA_BF16_PEAK_TFLOPS = 2500.0


def extend_chunks(w) -> np.ndarray:
    """Chunk per sequence: the tokens after the shared prompt (schema prefix and,
    for the fixer, the request's first attempt); the whole context without one."""
    shared = 16 * (int(w.meta.get("prefix_blocks", 0)) + int(w.meta.get("mid_blocks", 0)))
    return np.maximum(w.context_lens.astype(np.int64) - shared, 1).astype(np.int32)


def extend_inputs(w):
    """(chunk lengths, q_start, bf16 query rows) of the extend batch timed here:
    each sequence's chunk as ``extend_chunks``, queries N(0,1) from seed 4242."""
    from workloads import f32_to_bf16_bits
    chunk = extend_chunks(w)
    q_start = np.concatenate([[0], np.cumsum(chunk)]).astype(np.int32)
    rng = np.random.default_rng(4242)
    q = f32_to_bf16_bits(rng.standard_normal((int(q_start[-1]), w.num_q_heads, w.head_dim),
                                             dtype=np.float32))
    return chunk, q_start, q


def extend_flops(w, chunk) -> int:
    """Causal flops of one extend call: 4 Hq D per (row, visible token)."""
    ctx = w.context_lens.astype(np.int64)
    L = chunk.astype(np.int64)
    # row i of sequence b sees n - L + i + 1 tokens: the sum over i of a chunk
    vis = L * (ctx - L) + L * (L + 1) // 2
    return int(4 * w.num_q_heads * w.head_dim * int(vis.sum()))


def run_extend(w, base, reps, R, K, stream, sh, binding):
    """Time paged_attn_extend on the workload's batch and spot-check two sequences."""
    import torch
    if w.head_dim != 128 or w.max_context_len > 8192:
        return {"skipped": "extend needs head_dim 128 and contexts up to 8192 tokens"}
    chunk, q_start, q = extend_inputs(w)
    total = int(q_start[-1])
    dev = base.q.device
    q_dev = torch.from_numpy(q.view(np.int16)).to(dev)
    qs_dev = torch.from_numpy(q_start).to(dev)
    out = torch.zeros_like(q_dev)
    max_chunk = int(chunk.max())

    def call(i):
        binding.paged_attn_extend(reps[i % R][0], q_dev, qs_dev, total, base.bt, base.bt_stride, base.ctx,
                                  w.batch, w.num_q_heads, w.scale, base.max_ctx, max_chunk, out, sh)
    for i in range(3):
        call(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_calls = max(5, min(K, 50))
    e0.record(stream)
    for i in range(n_calls):
        call(i)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / n_calls
    flops = extend_flops(w, chunk)
    from workloads import touched_slots
    alg_bytes = touched_slots(w) * w.bytes_per_token + 2 * total * w.num_q_heads * w.head_dim * 2
    # parity spot check on the first and the longest-chunk sequence
    call(0)
    torch.cuda.synchronize()
    from oracle import compare, extend_attention
    seqs = sorted({0, int(np.argmax(chunk))})
    rows = np.concatenate([np.arange(q_start[b], q_start[b + 1]) for b in seqs])
    sub_start = np.concatenate([[0], np.cumsum(chunk[seqs])]).astype(np.int32)
    ref, _ = extend_attention(q[rows], sub_start, w.k_pool, w.v_pool, w.block_tables[seqs],
                              w.context_lens[seqs], w.scale)
    rep = compare(out.cpu().numpy().view(np.uint16)[rows], ref)
    log(f"extend spot check on sequences {seqs}: {rep}")
    del q_dev, qs_dev, out
    tflops = flops / (ms * 1e-3) / 1e12
    return {"workload": f"{w.name} batch, chunk = tokens after the shared prompt "
                        f"({int(chunk.min())}..{max_chunk}, {total} rows)",
            "kernel": f"extend_mfma_kernel<{w.group}>", "ms_per_call": round(ms, 5),
            "flops_per_call": flops, "tflops": round(tflops, 1),
            "roofline": {"bound": "mfma", "achieved": round(tflops, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4)},
            "alg_kv_gbps": round(alg_bytes / (ms * 1e-3) / 1e9, 1),
            "parity_spot_check": {"passed": rep.passed, "max_abs": rep.max_abs,
                                  "worst_row_rel_l2": rep.worst_row_rel_l2, "sequences": seqs}}


# --------------------------------------------------------------- footprint

def _blocks_in_use(w) -> int:
    """Blocks the pool allocator holds for a batch: claim every referenced
    block once, retain it once per extra table that maps it."""
    from paper_2510_14126_amd import binding
    pool = binding.kv_pool_create(w.num_blocks, 16, w.num_kv_heads, w.head_dim, 0x10000, 0x20000)
    nb = (w.context_lens.astype(np.int64) + 15) // 16
    used = np.concatenate([w.block_tables[b, : nb[b]] for b in range(w.batch)])
    ids, counts = np.unique(used, return_counts=True)
    binding.kv_pool_claim(pool, ids.tolist())
    extra = np.repeat(ids, counts - 1)
    if extra.size:
        binding.kv_pool_retain(pool, extra.tolist())
    in_use = w.num_blocks - binding.kv_pool_num_free(pool)
    pool.close()
    return int(in_use)


FOOTPRINT_BUDGETS = (1024, 2048, 4096)   # KV blocks per engine replica and layer (64 KiB each)
_FP_HQ, _FP_HKV, _FP_D = 32, 8, 128         # head geometry of the generator and fixer stages


class Replica:
    """One engine replica of a stage pool: a host-side block allocator over a
    fixed KV budget, the prompt contexts it keeps resident, and the sequences
    it admitted.  Shared prompt blocks are allocated once and retained once
    per sequence that maps them; with ``private`` every sequence holds its own
    copy of its prompt blocks (no prefix sharing)."""

    def __init__(self, budget, stages, private=False):
        from paper_2510_14126_amd import binding
        from workloads import FIXER_PROMPT, GENERATOR_PROMPT
        self.b = binding
        self.budget = budget
        self.stages = tuple(stages)
        self.private = private
        self.pool = binding.kv_pool_create(budget, 16, _FP_HKV, _FP_D, 0x10000, 0x20000)
        self.prompt = {}
        if not private:
            for st, tokens in (("generator", GENERATOR_PROMPT), ("fixer", FIXER_PROMPT)):
                if st in self.stages:
                    self.prompt[st] = binding.kv_pool_alloc(self.pool, tokens // 16)
        self.prompt_blocks = sum(len(v) for v in self.prompt.values())
        self.seqs = {"generator": [], "fixer": []}    # stage -> [(table ids, context length)]
        self.groups = []                              # fixer: sequences per request, in order

    def free(self) -> int:
        return self.b.kv_pool_num_free(self.pool)

    def need(self, unit) -> int:
        """Blocks a generator call or a whole fixer request (all retries) takes."""
        from workloads import FIRST_ATTEMPT, FIXER_PROMPT, GENERATOR_PROMPT
        stage, suffixes = unit
        nb = lambda t: -(-t // 16)                     # noqa: E731
        plen = GENERATOR_PROMPT if stage == "generator" else FIXER_PROMPT
        first = FIRST_ATTEMPT if stage == "fixer" else 0
        if self.private:
            return sum(nb(plen) + nb(first) + nb(s) for s in suffixes)
        return nb(first) + sum(nb(s) for s in suffixes)

    def admit(self, unit) -> bool:
        """Admit a generator call or a whole fixer request (all retries), or
        nothing if its blocks do not fit in the free blocks."""
        from workloads import FIRST_ATTEMPT, FIXER_PROMPT, GENERATOR_PROMPT
        stage, suffixes = unit
        if stage not in self.stages or self.need(unit) > self.free():
            return False
        nb = lambda t: -(-t // 16)                     # noqa: E731
        plen = GENERATOR_PROMPT if stage == "generator" else FIXER_PROMPT
        first = FIRST_ATTEMPT if stage == "fixer" else 0
        shared_first = [] if self.private or not first else self.b.kv_pool_alloc(self.pool, nb(first))
        for s in suffixes:
            if self.private:
                ids = self.b.kv_pool_alloc(self.pool, nb(plen) + nb(first) + nb(s))
            else:
                self.b.kv_pool_retain(self.pool, self.prompt[stage])
                if shared_first:
                    self.b.kv_pool_retain(self.pool, shared_first)
                ids = list(self.prompt[stage]) + list(shared_first) + self.b.kv_pool_alloc(self.pool, nb(s))
            self.seqs[stage].append((ids, plen + first + s))
        if stage == "fixer":
            self.groups.append(len(suffixes))
        return True

    @property
    def sequences(self) -> int:
        return sum(len(v) for v in self.seqs.values())

    def blocks_used(self) -> int:
        return self.budget - self.free()

    def close(self) -> None:
        self.pool.close()


def footprint_deployments(budget, units):
    """Three two-replica deployments with the same total KV budget (2 x
    budget blocks) serving the same demand, a sequence of requests that each
    make one generator call and one fixer request (units 2i, 2i + 1); each
    admits whole requests in order until the next no longer fits:
      isolated  a generator pool and a fixer pool, each keeping its own stage's
                prompt resident once; the 2 x budget blocks are split between
                them in proportion to the demand (each stage pool scaled on its
                own), so both stages admit the same requests;
      shared    two replicas of one engine, each keeping both stages' prompts
                resident, taking the requests alternately;
      private   the shared engine without prefix sharing (every sequence holds
                its own prompt blocks)."""
    pairs = [(units[i], units[i + 1]) for i in range(0, len(units) - 1, 2)]
    # isolated: the most requests whose two stage pools fit in 2 x budget
    from workloads import FIXER_PROMPT, GENERATOR_PROMPT
    need_g, need_f = GENERATOR_PROMPT // 16, FIXER_PROMPT // 16
    k = 0
    pg, pf = Replica(2 * budget, ["generator"]), Replica(2 * budget, ["fixer"])
    for gu, fu in pairs:
        if need_g + pg.need(gu) + need_f + pf.need(fu) > 2 * budget:
            break
        need_g += pg.need(gu)
        need_f += pf.need(fu)
        k += 1
    pg.close()
    pf.close()
    spare = 2 * budget - need_g - need_f
    iso = [Replica(need_g + spare // 2, ["generator"]), Replica(need_f + spare - spare // 2, ["fixer"])]
    for gu, fu in pairs[:k]:
        assert iso[0].admit(gu) and iso[1].admit(fu)
    out = {"isolated": iso}
    for kind, private in (("shared", False), ("private", True)):
        reps = [Replica(budget, ["generator", "fixer"], private) for _ in range(2)]
        full = [False, False]
        for j, (gu, fu) in enumerate(pairs):
            r = j % 2                          # requests alternate between the replicas
            if full[r]:
                r = 1 - r
            if full[r]:
                break
            if reps[r].need(gu) + reps[r].need(fu) > reps[r].free():
                full[r] = True
                continue
            assert reps[r].admit(gu) and reps[r].admit(fu)
        out[kind] = reps
    return out


def _replica_batches(rep, k_np, v_np, seed):
    """Decode launches of one replica's step: [(workload, PagedBatch keywords)]."""
    from workloads import FIRST_ATTEMPT, FIXER_PROMPT, GENERATOR_PROMPT, batch_from_tables
    out = []
    if rep.private:
        seqs = rep.seqs["generator"] + rep.seqs["fixer"]
        if seqs:
            w = batch_from_tables("private", [s[0] for s in seqs], [s[1] for s in seqs], rep.budget,
                                  _FP_HQ, _FP_HKV, _FP_D, seed, k_np, v_np)
            out.append((w, dict(partition_size=512)))
        return out
    gen = rep.seqs["generator"]
    if gen:
        w = batch_from_tables("generator", [s[0] for s in gen], [s[1] for s in gen], rep.budget,
                              _FP_HQ, _FP_HKV, _FP_D, seed, k_np, v_np)
        out.append((w, dict(partition_size=512, prefix_len=GENERATOR_PROMPT, prefix_partition_size=512)))
    fix = rep.seqs["fixer"]
    if fix:
        w = batch_from_tables("fixer", [s[0] for s in fix], [s[1] for s in fix], rep.budget,
                              _FP_HQ, _FP_HKV, _FP_D, seed + 1, k_np, v_np)
        starts = np.concatenate([[0], np.cumsum(rep.groups)]).astype(np.int32)
        out.append((w, dict(partition_size=1024, prefix_len=FIXER_PROMPT, prefix_partition_size=1024,
                            group_start=starts, group_len=FIRST_ATTEMPT)))
    return out


def _time_replica(rep, k_np, v_np, steps, warmup, seed):
    """Microseconds per decode step of one replica's admitted batch (all its
    launches), rotating over copies of its pool so that no step finds its
    blocks in the Infinity Cache.  k_np, v_np: the replica's pool values, one
    block per block of its budget."""
    import torch
    from paper_2510_14126_amd.device import PagedBatch
    if k_np.shape[0] != rep.budget or v_np.shape[0] != rep.budget:
        raise ValueError(f"pool values hold {k_np.shape[0]} blocks, the replica {rep.budget}")
    dev = torch.device("cuda:0")
    batches = _replica_batches(rep, k_np, v_np, seed)
    if not batches:
        return 0.0
    k0 = torch.from_numpy(k_np.view(np.int16)).to(dev)
    v0 = torch.from_numpy(v_np.view(np.int16)).to(dev)
    R = max(1, min(8, -(-(1 << 30) // (2 * k0.numel() * 2))))
    copies = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(R - 1)]
    pbs = [[PagedBatch(w, dev, register_blocks=False, k_pool=k, v_pool=v, schedule=True, **kw)
            for w, kw in batches] for k, v in copies]

    def step(i):
        for pb in pbs[i % R]:
            pb.run()
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    us = 1e3 * e0.elapsed_time(e1) / steps
    for row in pbs:
        for pb in row:
            pb.close()
    del pbs, copies, k0, v0
    torch.cuda.empty_cache()
    return us


def run_footprint(args):
    """Analogue of the paper's isolated-vs-shared comparison (Fig. 2, section 2
    "Cortex Benefits"): under a fixed KV budget per engine replica, how many
    sequences each deployment admits (the pool allocator's block counts) and
    the decode tokens/s it sustains at that batch (measured)."""
    from workloads import normal_bf16, stage_units
    units = stage_units(2510, 4000)
    results = []
    for M in FOOTPRINT_BUDGETS:
        deps = footprint_deployments(M, units)
        entry = {"blocks_per_replica": M, "total_blocks": 2 * M,
                 "mb_per_replica_and_layer": round(M * 2 * _FP_HKV * 16 * _FP_D * 2 / 1e6, 1)}
        for kind, reps in deps.items():
            recs = []
            for i, rep in enumerate(reps):
                shape = (rep.budget, _FP_HKV, 16, _FP_D)      # the replica's own pool
                k_np, v_np = normal_bf16(shape, 77, 1), normal_bf16(shape, 77, 2)
                us = _time_replica(rep, k_np, v_np, args.steps, args.warmup, 300 + i)
                recs.append({"stages": list(rep.stages), "prompt_blocks": rep.prompt_blocks,
                             "blocks_used": rep.blocks_used(),
                             "generator_sequences": len(rep.seqs["generator"]),
                             "fixer_sequences": len(rep.seqs["fixer"]),
                             "us_per_step": round(us, 2),
                             "tokens_per_s": round(rep.sequences / (us * 1e-6), 1) if us else 0.0})
                rep.close()
            entry[kind] = {"replicas": recs, "requests": len([1 for r in reps for _ in r.groups]),
                           "sequences": sum(r["generator_sequences"] + r["fixer_sequences"] for r in recs),
                           "prompt_blocks": sum(r["prompt_blocks"] for r in recs),
                           "tokens_per_s": round(sum(r["tokens_per_s"] for r in recs), 1)}
        entry["isolated_over_shared"] = {
            "requests": round(entry["isolated"]["requests"] / max(1, entry["shared"]["requests"]), 3),
            "sequences": round(entry["isolated"]["sequences"] / max(1, entry["shared"]["sequences"]), 3),
            "tokens_per_s": round(entry["isolated"]["tokens_per_s"] / max(1.0, entry["shared"]["tokens_per_s"]), 3)}
        log(f"footprint M={M}: " + ", ".join(f"{k}: {entry[k]['sequences']} seqs "
                                            f"{entry[k]['tokens_per_s'] / 1e6:.2f} M tok/s"
                                            for k in ("isolated", "shared", "private")))
        results.append(entry)
    line = {
        "metric": "sequences admitted and decode tokens/s of two engine replicas under a fixed KV "
                  "budget per replica: isolated stage pools vs one shared engine vs no prefix sharing",
        "budgets": results, "n_gpus": 1, "steps": args.steps, "data": "synthetic",
        "note": "one layer; generator calls and fixer requests alternate in the demand; each "
                "replica admits until a unit no longer fits; replicas are timed one at a time",
    }
    print(json.dumps(line), flush=True)


# ---------------------------------------------------------------- GPU timing

def measure(k, w, args, cpu, copy_gbps, headline, with_extend):
    """Time one workload's decode steps in its launch configuration and return
    its record (the headline fields, or one per_config entry)."""
    import torch
    from paper_2510_14126_amd import binding
    from paper_2510_14126_amd.device import PagedBatch

    over = dict(partition_size=args.partition_size, prefix_partition_size=args.prefix_partition_size,
                cascade=args.cascade, groups=args.groups) if headline else {}
    S, kw = launch_configuration(k, w, **over)
    w.partition_size = S
    alg_bytes, logical_bytes = byte_accounting(w)
    prefix_len = kw.get("prefix_len", 0)
    group_len = kw.get("group_len", 0)
    dev = torch.device("cuda:0")
    pool_bytes = 2 * w.k_pool.nbytes
    R = (args.replicas if headline and args.replicas else
         max(1, min(16, -(-(1 << 30) // pool_bytes))))
    base = PagedBatch(w, dev, partition_size=S, schedule=args.schedule == "on", **kw)
    sched_host_us = None
    if base.items is not None:
        # host cost of the work list (a serving loop rebuilds it every step
        # from its host context lengths, like the block tables)
        ts = []
        for _ in range(50):
            t1 = time.perf_counter()
            binding.paged_attn_schedule(w.context_lens, base.max_ctx, base.partition_size,
                                        prefix_len + group_len)
            ts.append(time.perf_counter() - t1)
        sched_host_us = round(1e6 * float(np.median(ts)), 1)
    reps = [(base.pool, base.q)]
    keep = []
    for _ in range(1, R):
        kk, vv, qq = base.k.clone(), base.v.clone(), base.q.clone()
        keep.append((kk, vv, qq))
        reps.append((binding.kv_pool_create(w.num_blocks, 16, w.num_kv_heads, w.head_dim, kk, vv), qq))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    split = base.needs_reduce

    def decode_on(i, st):
        pool, q = reps[i % R]
        base.decode(st, pool=pool, q=q)

    def decode(i):
        decode_on(i, sh)

    def reduce():
        base.reduce(sh)

    for i in range(args.warmup):
        decode(i)
        if split:
            reduce()
    torch.cuda.synchronize()

    K = args.steps
    graphs = None
    if args.graph and headline:
        # one captured step per replica; replays carry no host launch cost
        graphs = []
        for r in range(R):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                cs = torch.cuda.current_stream().cuda_stream
                decode_on(r, cs)
                if split:
                    base.reduce(cs)
            graphs.append(g)
        for g in graphs:
            g.replay()
        torch.cuda.synchronize()

    def step(i):
        if graphs is not None:
            graphs[i % R].replay()
        else:
            decode(i)
            if split:
                reduce()

    # timed region: K whole steps, no instrumentation between launches
    e_start = torch.cuda.Event(enable_timing=True)
    e_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    e_start.record(stream)
    for i in range(K):
        step(i)
    e_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_step = e_start.elapsed_time(e_end) / K

    # per-kernel durations: K decode launches back to back between two events
    # on the launch stream, then K reduce launches the same way
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(K):
        decode(i)
    ev[1].record(stream)
    for i in range(K if split else 0):
        reduce()
    ev[2].record(stream)
    torch.cuda.synchronize()
    dec_avg = ev[0].elapsed_time(ev[1]) / K
    red_avg = ev[1].elapsed_time(ev[2]) / K if split else 0.0

    # data-movement reference: the tiles the step reads (each distinct one
    # once), in the decode's grid shape, read with no arithmetic
    spans = base.tile_spans()
    n_spans = int(spans.shape[0])
    sink = torch.empty(max(1, n_spans * w.num_kv_heads * 4), dtype=torch.int32, device=dev)

    def time_gather(table, stride, rows, span_arr):
        """us per call at ring depths 2 and 4, rotating the replicas like the decode."""
        sd = torch.from_numpy(np.ascontiguousarray(span_arr, dtype=np.int32)).to(dev)
        us = {}
        for nif in (2, 4):
            call = lambda i: binding.pa_gather_tiles(reps[i % R][0], table, stride, rows, sd,  # noqa: E731
                                                     n_spans, sink, sh, nif)
            for i in range(3):
                call(i)
            torch.cuda.synchronize()
            ev[0].record(stream)
            for i in range(K):
                call(i)
            ev[1].record(stream)
            torch.cuda.synchronize()
            us[nif] = 1e3 * ev[0].elapsed_time(ev[1]) / K
        return us

    gather_us = time_gather(base.bt, base.bt_stride, base.batch, spans)
    best_nif = min(gather_us, key=gather_us.get)
    gather_avg = gather_us[best_nif] / 1e3
    span_blocks = [(int(e) - (int(s0) & ~15) + 15) // 16 for _, s0, e in spans]
    tiles_read = int(sum(span_blocks)) * w.num_kv_heads
    gather_bytes = tiles_read * 2 * 16 * w.head_dim * 2
    gather_line = {"us_per_call": round(gather_avg * 1e3, 3), "kv_bytes": gather_bytes,
                   "tiles_in_flight": best_nif,
                   "us_by_tiles_in_flight": {str(a): round(b, 3) for a, b in gather_us.items()},
                   "gbps": round(gather_bytes / (gather_avg * 1e-3) / 1e9, 1),
                   "spans": n_spans,
                   "decode_time_over_gather": round(dec_avg / gather_avg, 3)}
    if headline:
        # the same spans with every span's blocks laid out contiguously (ids in
        # order, one table row per span): the same bytes without fragmentation
        crow = max(1, max(span_blocks, default=1))
        ctab = np.zeros((max(1, n_spans), crow), dtype=np.int32)
        nxt = 0
        for i, nb in enumerate(span_blocks):
            ctab[i, :nb] = np.arange(nxt, nxt + nb) % w.num_blocks
            nxt += nb
        cspans = np.stack([np.arange(n_spans), np.zeros(n_spans, np.int64),
                           16 * np.asarray(span_blocks, np.int64)], axis=1) if n_spans else spans
        contig_us = time_gather(torch.from_numpy(ctab).to(dev), crow, max(1, n_spans), cspans)
        contig_avg = min(contig_us.values()) / 1e3
        gather_line.update({
            "contiguous_us_per_call": round(contig_avg * 1e3, 3),
            "contiguous_gbps": round(gather_bytes / (contig_avg * 1e-3) / 1e9, 1),
            "note": "pa_gather_tiles: the K/V tiles of this step (each once) read in the "
                    "decode's grid shape with no arithmetic (the faster ring depth); "
                    "contiguous: the same spans with each span's blocks stored in order"})
    log(f"[{w.name}] gather reference: {gather_line}")

    # hot: K steps back to back on one replica (its working set stays in the
    # caches), timed like the main loop
    hot_ms = None
    if args.hot:
        decode(0)
        if split:
            reduce()
        torch.cuda.synchronize()
        ev[0].record(stream)
        for i in range(K):
            decode(0)
            if split:
                reduce()
        ev[1].record(stream)
        torch.cuda.synchronize()
        hot_ms = ev[0].elapsed_time(ev[1]) / K

    # KV append of the step's new token, timed the same way.  The rows written
    # are the ones already stored at slot ctx-1, so the pools stay unchanged
    # for the parity check below.
    nz = w.context_lens > 0
    last = np.maximum(w.context_lens.astype(np.int64) - 1, 0)
    phys = w.block_tables[np.arange(w.batch), last // 16]
    k_new = torch.from_numpy(np.ascontiguousarray(w.k_pool[phys, :, last % 16, :]).view(np.int16)).to(dev)
    v_new = torch.from_numpy(np.ascontiguousarray(w.v_pool[phys, :, last % 16, :]).view(np.int16)).to(dev)
    for i in range(3):
        binding.paged_attn_append_kv(reps[i % R][0], k_new, v_new, base.bt, base.bt_stride, base.ctx,
                                     base.batch, sh)
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(K):
        binding.paged_attn_append_kv(reps[i % R][0], k_new, v_new, base.bt, base.bt_stride, base.ctx,
                                     base.batch, sh)
    ev[1].record(stream)
    torch.cuda.synchronize()
    app_ms = ev[0].elapsed_time(ev[1]) / K
    app_bytes = 4 * int(nz.sum()) * w.num_kv_heads * w.head_dim * 2      # K+V rows read and written
    append_line = {"us_per_call": round(app_ms * 1e3, 3), "bytes_per_call": app_bytes,
                   "gbps": round(app_bytes / (app_ms * 1e-3) / 1e9, 2),
                   "note": "one launch per step; launch-latency bound at these sizes"}

    # A serving loop's decode iteration: append, decode and reduce as three
    # launches, against the fused append + decode and the reduce (the same
    # rows as above, so the pools stay unchanged).
    def iteration(i, fused):
        pool, q = reps[i % R]
        if fused:
            base.decode_append(k_new, v_new, sh, pool=pool, q=q)
        else:
            binding.paged_attn_append_kv(pool, k_new, v_new, base.bt, base.bt_stride, base.ctx,
                                         base.batch, sh)
            base.decode(sh, pool=pool, q=q)
        if split:
            reduce()

    iter_us = {}
    for fused in (False, True):
        for i in range(3):
            iteration(i, fused)
        torch.cuda.synchronize()
        ev[0].record(stream)
        for i in range(K):
            iteration(i, fused)
        ev[1].record(stream)
        torch.cuda.synchronize()
        iter_us["fused" if fused else "append_then_decode"] = round(
            1e3 * ev[0].elapsed_time(ev[1]) / K, 3)
    iteration_line = {"append_then_decode_us": iter_us["append_then_decode"],
                      "fused_append_decode_us": iter_us["fused"],
                      "note": "append + decode (+ reduce) per step as separate launches, and with "
                              "paged_attn_decode(_cascade)_append; same replicas as the main loop"}

    extend_line = run_extend(w, base, reps, R, K, stream, sh, binding) if with_extend else None

    # parity spot check of the benchmarked launch configuration
    from oracle import compare, decode_workload
    torch.cuda.synchronize()
    base.out.zero_()
    decode(0)
    if split:
        reduce()
    torch.cuda.synchronize()
    seqs = sorted({0, int(np.argmax(w.context_lens)), w.batch - 1})
    ref, _ = decode_workload(w, seqs=seqs)
    rep = compare(base.out_bits()[seqs], ref)
    log(f"[{w.name}] parity spot check on sequences {seqs}: {rep}")

    achieved = alg_bytes / (dec_avg * 1e-3) / 1e9
    value = alg_bytes / (ms_step * 1e-3) / 1e9
    kern = decode_kernel_of(w, prefix_len)
    traffic = traffic_from_profiles(w.name, kern)
    rec = {
        "value": round(value, 2),
        "unit": "GB/s",
        "ms_per_step": round(ms_step, 5),
        "config": {"workload": f"{w.name}: {w.meta['description']}", "batch": w.batch,
                   "num_q_heads": w.num_q_heads, "num_kv_heads": w.num_kv_heads,
                   "head_dim": w.head_dim, "block_size": 16, "partition_size": base.partition_size,
                   "num_partitions": base.num_parts, "replicas_rotated": R,
                   "shared_prefix_cascade": {"prefix_len": prefix_len,
                                             "prefix_partition_size": base.prefix_partition_size,
                                             "groups": {"count": base.num_groups,
                                                        "shared_tokens": group_len}
                                             if group_len else None}
                   if prefix_len else None,
                   "work_list": (f"host-built, {int(base.items.numel())} non-empty items longest first"
                                 if base.items is not None else "full grid"),
                   "work_list_host_us": sched_host_us,
                   "max_context_len": w.max_context_len, "parallelism": "single GPU"},
        "pct_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "frac_hbm_peak_step": round(value / HBM_PEAK_GBPS, 4),
        "meets_70pct_hbm_target": bool(value >= 0.7 * HBM_PEAK_GBPS),
        "decode_steps_per_s": round(1000.0 / ms_step, 2),
        "tokens_per_s": round(w.batch * 1000.0 / ms_step, 1),
        "algorithmic_bytes_per_step": int(alg_bytes),
        "logical_kv_gbps_effective": round(logical_bytes / (ms_step * 1e-3) / 1e9, 2),
        "hot_ms_per_step": round(hot_ms, 5) if hot_ms is not None else None,
        "launch": "hip graph replay per step" if graphs is not None else "direct launches",
        "kernel_ms": {"decode_avg": round(dec_avg, 5), "reduce_avg": round(red_avg, 5)},
        "pct_of_copy_probe": round(100 * value / copy_gbps, 2),
        "wall_s_timed_region": round(wall, 4),
        "parity_spot_check": {"passed": rep.passed, "max_abs": rep.max_abs,
                              "worst_row_rel_l2": rep.worst_row_rel_l2, "sequences": seqs},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic,
                     "kernel": kernel_display_name(w, kern),
                     "launch": "decode call (all kernels it launches)",
                     "bytes_per_launch": int(alg_bytes)},
        "gather_reference": gather_line,
        "append_kv": append_line,
        "decode_iteration": iteration_line,
        "cpu_baseline": cpu,
    }
    if extend_line is not None:
        rec["extend"] = extend_line
    # free this workload's device memory before the next one
    for pool, _ in reps[1:]:
        pool.close()
    base.close()
    del reps, keep, base, k_new, v_new, sink
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def profile_loop(k, w, args):
    """Only the decode launches (plus one calibration copy): for hardware-counter
    and kernel-trace runs under rocprofv3.  With --stamp, first writes the
    sources this run was built from."""
    import torch
    from paper_2510_14126_amd import binding
    from paper_2510_14126_amd.device import PagedBatch
    S, kw = launch_configuration(k, w, args.partition_size, args.prefix_partition_size,
                                 args.cascade, args.groups)
    dev = torch.device("cuda:0")
    base = PagedBatch(w, dev, partition_size=S, schedule=args.schedule == "on", **kw)
    pool_bytes = 2 * w.k_pool.nbytes
    R = args.replicas or max(1, min(16, -(-(1 << 30) // pool_bytes)))
    reps = [(base.pool, base.q)]
    keep = []
    for _ in range(1, R):
        kk, vv, qq = base.k.clone(), base.v.clone(), base.q.clone()
        keep.append((kk, vv, qq))
        reps.append((binding.kv_pool_create(w.num_blocks, 16, w.num_kv_heads, w.head_dim, kk, vv), qq))
    sh = torch.cuda.current_stream().cuda_stream
    src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    binding.pa_stream_copy(src, dst, src.numel(), sh)      # calibration: 256 MiB each way
    if args.extend:
        chunk, q_start, q = extend_inputs(w)
        q_dev = torch.from_numpy(q.view(np.int16)).to(dev)
        qs_dev = torch.from_numpy(q_start).to(dev)
        out = torch.zeros_like(q_dev)
        for i in range(args.profile_loop):
            binding.paged_attn_extend(reps[i % R][0], q_dev, qs_dev, int(q_start[-1]), base.bt,
                                      base.bt_stride, base.ctx, w.batch, w.num_q_heads, w.scale,
                                      base.max_ctx, int(chunk.max()), out, sh)
    else:
        for i in range(args.profile_loop):
            pool, q = reps[i % R]
            base.decode(sh, pool=pool, q=q)
            if base.needs_reduce:
                base.reduce(sh)
    torch.cuda.synchronize()
    log(f"profile loop done: {args.profile_loop} {'extend' if args.extend else 'decode'} launches, "
        f"replicas={R}, calibration copy 268435456 bytes")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=None,
                    help="measure batch k alone (default: the long-context headline plus a "
                         "per_config entry for each other batch)")
    ap.add_argument("--partition-size", type=int, default=None)
    ap.add_argument("--replicas", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle time of the headline CPU baseline")
    ap.add_argument("--cpu-seconds-per-config", type=float, default=3.0,
                    help="oracle time of each per_config CPU baseline")
    ap.add_argument("--hot", action=argparse.BooleanOptionalAction, default=True,
                    help="also time steps on a single replica (cache-warm); --no-hot skips it")
    ap.add_argument("--cascade", choices=["auto", "on", "off"], default="auto",
                    help="shared-prefix cascade (auto: on when the batch shares a prefix)")
    ap.add_argument("--prefix-partition-size", type=int, default=None,
                    help="tokens per prefix partition (default: per workload, see DEFAULT_PREFIX_PARTITION)")
    ap.add_argument("--schedule", choices=["on", "off"], default="on",
                    help="run the decode over a host-built work list (non-empty items, longest first)")
    ap.add_argument("--groups", choices=["auto", "on", "off"], default="auto",
                    help="second level of sharing: groups of sequences (a fixer request's retries) "
                         "that share tokens after the prefix (auto: when the workload has them)")
    ap.add_argument("--graph", action="store_true",
                    help="replay each step from a captured HIP graph (one per replica)")
    ap.add_argument("--ingest-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--ingest-stats", metavar="KERNEL_STATS_CSV")
    ap.add_argument("--ingest-sq", nargs="+", metavar="COUNTER_CSV",
                    help="write an SQ-counter summary (with --sq-kernel and --profile-name)")
    ap.add_argument("--sq-kernel", default="cascade_kernel")
    ap.add_argument("--command-note", default="")
    ap.add_argument("--stamp", default=None,
                    help="measuring runs: write the source stamp here; ingest: the stamp to check")
    ap.add_argument("--extend", action="store_true",
                    help="also time extend (chunked prefill) attention on --config k: each "
                         "sequence's tokens after its shared prompt as the chunk (the default run "
                         "times it on the fixer batch)")
    ap.add_argument("--footprint", action="store_true",
                    help="isolated stage pools vs one shared engine under a fixed KV budget; "
                         "prints its own JSON line")
    ap.add_argument("--profile-name", default=None,
                    help="file stem for --ingest-stats (default kernels_<workload>_stats)")
    ap.add_argument("--profile-loop", type=int, default=0,
                    help="only run this many decode (or, with --extend, extend) launches of "
                         "--config (default the headline batch) plus one calibration copy, and "
                         "exit; for rocprofv3 runs")
    args = ap.parse_args()

    from workloads import CONFIG_NAMES, build_config
    if args.ingest_sq or args.ingest_counters or args.ingest_stats:
        k = args.config or HEADLINE_CONFIG
        name = CONFIG_NAMES[k]
        stamp = checked_stamp(args.stamp)
        if args.ingest_sq:
            ingest_sq(args.ingest_sq, name, args.sq_kernel, args.command_note,
                      args.profile_name or f"sq_{name}", stamp)
        if args.ingest_counters:
            wc = build_config(k, values=False)
            S, kw = launch_configuration(k, wc, args.partition_size, args.prefix_partition_size,
                                         args.cascade, args.groups)
            ingest_counters(*args.ingest_counters, name, decode_kernel_of(wc, kw.get("prefix_len", 0)),
                            args.command_note, stamp)
        if args.ingest_stats:
            ingest_stats(args.ingest_stats, name, args.command_note, stamp, args.profile_name)
        return

    if args.stamp:
        # the sources this (profiled) run was built from, checked at ingest
        os.makedirs(os.path.dirname(os.path.abspath(args.stamp)), exist_ok=True)
        with open(args.stamp, "w") as f:
            json.dump(source_stamp(), f)

    if args.footprint:
        run_footprint(args)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE={world}); "
              "the decode-attention path runs on a single GPU", file=sys.stderr)
        sys.exit(2)

    head_k = args.config or HEADLINE_CONFIG
    extra = [] if args.config or args.profile_loop else [c for c in PER_CONFIG if c != head_k]
    t0 = time.perf_counter()
    ws = {}
    for k in [head_k] + extra:
        ws[k] = build_config(k)
        S, _ = launch_configuration(k, ws[k])
        ws[k].partition_size = S
        alg, logical = byte_accounting(ws[k])
        log(f"workload {ws[k].name}: B={ws[k].batch} Hq={ws[k].num_q_heads} Hkv={ws[k].num_kv_heads} "
            f"D={ws[k].head_dim} NB={ws[k].num_blocks} max_ctx={ws[k].max_context_len} "
            f"alg={alg/1e6:.1f} MB logical={logical/1e6:.1f} MB ({time.perf_counter()-t0:.1f} s)")

    if args.profile_loop:
        profile_loop(head_k, ws[head_k], args)
        return

    # CPU baselines first: the oracle's worker pools are forked before the
    # process touches the GPU
    cpu = {}
    if not args.no_cpu_baseline:
        for k in [head_k] + extra:
            alg, logical = byte_accounting(ws[k])
            secs = args.cpu_seconds if k == head_k else args.cpu_seconds_per_config
            log(f"cpu baseline (oracle) {ws[k].name} ...")
            cpu[k] = cpu_baseline(ws[k], alg, secs, logical)
            log(f"cpu baseline {ws[k].name}: {cpu[k]}")

    import torch
    from paper_2510_14126_amd import binding
    dev = torch.device("cuda:0")
    sh = torch.cuda.current_stream().cuda_stream
    # achievable copy bandwidth on this machine (read + write bytes)
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        binding.pa_stream_copy(src, dst, src.numel(), sh)
    c0 = torch.cuda.Event(enable_timing=True); c1 = torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(10):
        binding.pa_stream_copy(src, dst, src.numel(), sh)
    c1.record()
    torch.cuda.synchronize()
    copy_gbps = 10 * 2 * src.numel() / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()

    head = measure(head_k, ws.pop(head_k), args, cpu.get(head_k), copy_gbps, True,
                   args.extend)
    per_config = []
    extend_line = head.pop("extend", None)
    for k in extra:
        w = ws.pop(k)
        rec = measure(k, w, args, cpu.get(k), copy_gbps, False, with_extend=(k == 3))
        if "extend" in rec:
            extend_line = rec.pop("extend")
        rec = {"config_index": k, "workload": w.name, **rec}
        per_config.append(rec)
        log(f"per_config {w.name}: {rec['ms_per_step']} ms/step, {rec['value']} GB/s "
            f"({rec['pct_hbm_peak']}% of peak), decode {rec['kernel_ms']['decode_avg']} ms, "
            f"parity {rec['parity_spot_check']['passed']}")
        del w

    line = {
        "metric": "paged decode-attention KV GB/s (algorithmic bytes) and % of HBM peak; "
                  "decode steps/s per batch",
        "value": head["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 K/V/Q; stage-shaped block tables and lengths)",
        **{k: v for k, v in head.items() if k not in ("value", "unit", "ms_per_step")},
        "copy_probe_gbps": round(copy_gbps, 1),
        "per_config": per_config,
        "target_70pct_hbm_on_configs_1_to_4": (
            {r["workload"]: r["meets_70pct_hbm_target"] for r in per_config} if per_config else None),
        "extend": extend_line,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
