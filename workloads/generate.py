"""Seeded synthetic inputs for batched paged decode attention.

This module only *builds inputs*: context lengths, block tables, K/V block
pools and query rows, all bf16 values stored as their 16-bit patterns
(``uint16``).  It holds no attention arithmetic.  The CPU oracle and the GPU
path both consume what it returns and neither is imported here.

The stage shapes mirror the NL2SQL agent of the paper (section 1 and section 2,
Fig. 1): an SQL-generator stage whose calls all share one resident schema
prompt, an SQL-error-fixer stage whose retries (up to five per request) share
the schema prompt and the first attempt, a single
shared engine pool that mixes both stages without stage isolation (Fig. 2's
contrast case), and a long-context stage pool.

Physical layout of a pool (token-major tiles, one tile per block and KV head)::

    k_pool[num_blocks][num_kv_heads][block_size][head_dim]   uint16 (bf16 bits)
    v_pool  same shape

Block tables are ``int32[batch][max_blocks_per_seq]``; entries past
``ceil(ctx / block_size)`` hold -1 and must never be read.

Values are N(0, 1) drawn in float32 and rounded to bf16 with round-to-nearest-
even.  Large arrays are drawn in fixed 4 Mi-element chunks, chunk ``c`` of
stream ``s`` coming from ``numpy.random.default_rng([seed, s, c])``; the
result therefore depends only on (seed, stream, shape) and not on how many
threads fill it.
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

BLOCK_SIZE = 16
CHUNK = 1 << 22

# bf16 bit patterns used as poison.
BF16_QNAN = 0x7FC0
BF16_ONE = 0x3F80

STREAM_K, STREAM_V, STREAM_Q = 1, 2, 3


# --------------------------------------------------------------------------
# value generation
# --------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even) and return bits.

    Used only to encode generated inputs; NaN maps to the canonical quiet NaN.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    rounded = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        rounded[nan] = BF16_QNAN
    return rounded


def _fill_chunk(out: np.ndarray, seed: int, stream: int, c: int) -> None:
    lo = c * CHUNK
    hi = min(lo + CHUNK, out.size)
    rng = np.random.default_rng([seed, stream, c])
    x = rng.standard_normal(hi - lo, dtype=np.float32)
    b = x.view(np.uint32)
    b += np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    out[lo:hi] = (b >> np.uint32(16)).astype(np.uint16)


def normal_bf16(shape, seed: int, stream: int, threads: int | None = None) -> np.ndarray:
    """N(0,1) values rounded to bf16, as uint16 bits, chunk-keyed by (seed, stream)."""
    n = int(np.prod(shape, dtype=np.int64))
    out = np.empty(n, dtype=np.uint16)
    nchunks = (n + CHUNK - 1) // CHUNK
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))
    if nchunks <= 1 or threads <= 1:
        for c in range(nchunks):
            _fill_chunk(out, seed, stream, c)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(lambda c: _fill_chunk(out, seed, stream, c), range(nchunks)))
    return out.reshape(shape)


# --------------------------------------------------------------------------
# workload container
# --------------------------------------------------------------------------

@dataclass
class Workload:
    """One decode step of one layer: everything the hot path reads."""

    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    num_blocks: int
    context_lens: np.ndarray          # int32 [B]
    block_tables: np.ndarray          # int32 [B][max_blocks]
    scale: float
    partition_size: int = 512
    block_size: int = BLOCK_SIZE
    q: np.ndarray | None = None       # uint16 [B][Hq][D]
    k_pool: np.ndarray | None = None  # uint16 [NB][Hkv][BS][D]
    v_pool: np.ndarray | None = None
    meta: dict = field(default_factory=dict)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def max_context_len(self) -> int:
        return int(self.context_lens.max()) if self.batch else 0

    @property
    def bytes_per_token(self) -> int:
        """K plus V bytes of one token over all KV heads."""
        return 2 * self.num_kv_heads * self.head_dim * 2

    def blocks_per_seq(self) -> np.ndarray:
        return (self.context_lens.astype(np.int64) + self.block_size - 1) // self.block_size


def touched_slots(w: Workload) -> int:
    """Distinct (physical block, row) token slots read by one decode step."""
    seen: dict[int, int] = {}
    for b in range(w.batch):
        n = int(w.context_lens[b])
        nb = (n + w.block_size - 1) // w.block_size
        for j in range(nb):
            pid = int(w.block_tables[b, j])
            valid = min(w.block_size, n - j * w.block_size)
            if seen.get(pid, 0) < valid:
                seen[pid] = valid
    return sum(seen.values())


def logical_tokens(w: Workload) -> int:
    return int(w.context_lens.astype(np.int64).sum())


def _tables_from_lists(lists, width=None) -> np.ndarray:
    width = width if width is not None else max((len(x) for x in lists), default=0)
    bt = np.full((len(lists), max(width, 1)), -1, dtype=np.int32)
    for i, ids in enumerate(lists):
        bt[i, : len(ids)] = ids
    return bt


def _fill_values(w: Workload, seed: int) -> Workload:
    shape = (w.num_blocks, w.num_kv_heads, w.block_size, w.head_dim)
    w.k_pool = normal_bf16(shape, seed, STREAM_K)
    w.v_pool = normal_bf16(shape, seed, STREAM_V)
    w.q = normal_bf16((w.batch, w.num_q_heads, w.head_dim), seed, STREAM_Q)
    return w


def _nblk(n: int) -> int:
    return (n + BLOCK_SIZE - 1) // BLOCK_SIZE


# --------------------------------------------------------------------------
# the five stage-shaped configurations
# --------------------------------------------------------------------------

CONFIG_NAMES = {
    1: "tiny",
    2: "sql_generator",
    3: "sql_error_fixer",
    4: "shared_pool",
    5: "long_context",
}

CONFIG_DESCRIPTIONS = {
    1: "tiny: batch 4, 8 q / 2 kv heads, head_dim 64, ctx U[100,300], 128-block permuted pool",
    2: "SQL-generator stage: batch 64, 32 q / 8 kv heads, head_dim 128, shared 2048-token "
       "schema prefix + unique suffix U[64,512], pool 1.2x needed, shuffled",
    3: "SQL-error-fixer stage: 32 requests x U{1..5} retries, 32 q / 8 kv heads, head_dim 128, "
       "shared 2048 prefix + per-request 256-token first attempt + unique retry U[128,1024]",
    4: "shared pool (no stage isolation): batch 256, generator/fixer 50/50, 32 q / 8 kv, "
       "head_dim 128, lognormal lengths (mean 1500, sigma 0.8, clip 64..8192), 50% holes",
    5: "long-context stage pool: batch 128, 64 q / 8 kv heads, head_dim 128, ctx U[8192,32768] "
       "with shared 4096-token prefix, 512-token split-KV partitions",
}


def _stage_with_prefix(name, rng, batch, hq, hkv, d, prefix_tokens, suffix_lens, pool_factor=1.2,
                       mid_groups=None, mid_tokens=0):
    """Sequences = shared prefix [+ per-group shared middle] + unique suffix.

    ``mid_groups[b]`` names the group (request) sequence b belongs to; all
    sequences of a group share ``mid_tokens`` tokens after the prefix.
    Both shared parts must be whole blocks.
    """
    assert prefix_tokens % BLOCK_SIZE == 0 and mid_tokens % BLOCK_SIZE == 0
    n_pre = prefix_tokens // BLOCK_SIZE
    n_mid = mid_tokens // BLOCK_SIZE
    groups = sorted(set(mid_groups)) if mid_groups is not None else []
    suffix_blocks = [_nblk(int(s)) for s in suffix_lens]
    needed = n_pre + n_mid * len(groups) + sum(suffix_blocks)
    nb = int(math.ceil(pool_factor * needed))
    perm = rng.permutation(nb).astype(np.int32)
    cursor = 0
    pre_ids = perm[cursor: cursor + n_pre]; cursor += n_pre
    mid_ids = {}
    for gidx in groups:
        mid_ids[gidx] = perm[cursor: cursor + n_mid]; cursor += n_mid
    lists = []
    for b in range(batch):
        ids = list(pre_ids)
        if mid_groups is not None:
            ids += list(mid_ids[mid_groups[b]])
        ids += list(perm[cursor: cursor + suffix_blocks[b]]); cursor += suffix_blocks[b]
        lists.append(ids)
    ctx = np.array([prefix_tokens + mid_tokens + int(s) for s in suffix_lens], dtype=np.int32)
    w = Workload(name=name, batch=batch, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                 num_blocks=nb, context_lens=ctx, block_tables=_tables_from_lists(lists),
                 scale=1.0 / math.sqrt(d))
    w.meta.update(prefix_blocks=n_pre, mid_blocks=n_mid, needed_blocks=needed,
                  used_ids=perm[:needed].copy())
    if mid_groups is not None:
        w.meta["groups"] = np.asarray(mid_groups, dtype=np.int32)
    return w


def build_config(k: int, values: bool = True) -> Workload:
    """Configuration ``k`` (1..5) with seed ``1000 + k``.

    Draw order: structure, then physical placement (both from
    ``default_rng(1000 + k)``), then K, V and Q values (chunk-keyed streams).
    ``values=False`` returns the structure only (tables, lengths, pool size).
    """
    seed = 1000 + k
    rng = np.random.default_rng(seed)
    if k == 1:
        batch, hq, hkv, d, nb = 4, 8, 2, 64, 128
        ctx = rng.integers(100, 300, size=batch, endpoint=True).astype(np.int32)
        perm = rng.permutation(nb).astype(np.int32)
        lists, cur = [], 0
        for n in ctx:
            m = _nblk(int(n)); lists.append(list(perm[cur: cur + m])); cur += m
        w = Workload(name=CONFIG_NAMES[1], batch=batch, num_q_heads=hq, num_kv_heads=hkv,
                     head_dim=d, num_blocks=nb, context_lens=ctx,
                     block_tables=_tables_from_lists(lists), scale=1.0 / math.sqrt(d))
        w.meta.update(needed_blocks=cur, used_ids=perm[:cur].copy())
    elif k == 2:
        batch = 64
        suffix = rng.integers(64, 512, size=batch, endpoint=True)
        w = _stage_with_prefix(CONFIG_NAMES[2], rng, batch, 32, 8, 128, 2048, suffix)
    elif k == 3:
        n_req = 32
        retries = rng.integers(1, 5, size=n_req, endpoint=True)
        groups = np.repeat(np.arange(n_req), retries)
        batch = int(groups.size)
        suffix = rng.integers(128, 1024, size=batch, endpoint=True)
        w = _stage_with_prefix(CONFIG_NAMES[3], rng, batch, 32, 8, 128, 2048, suffix,
                               mid_groups=list(groups), mid_tokens=256)
        w.meta["retries"] = retries.astype(np.int32)
    elif k == 4:
        batch, hq, hkv, d = 256, 32, 8, 128
        tags = rng.permutation(np.array(["generator"] * 128 + ["fixer"] * 128))
        sigma = 0.8
        mu = math.log(1500.0) - sigma * sigma / 2.0
        raw = rng.lognormal(mu, sigma, size=batch)
        ctx = np.clip(np.rint(raw), 64, 8192).astype(np.int32)
        nblocks = [_nblk(int(n)) for n in ctx]
        needed = int(sum(nblocks))
        nb = 2 * needed
        ids = rng.choice(nb, size=needed, replace=False).astype(np.int32)
        lists, cur = [], 0
        for m in nblocks:
            lists.append(list(ids[cur: cur + m])); cur += m
        w = Workload(name=CONFIG_NAMES[4], batch=batch, num_q_heads=hq, num_kv_heads=hkv,
                     head_dim=d, num_blocks=nb, context_lens=ctx,
                     block_tables=_tables_from_lists(lists), scale=1.0 / math.sqrt(d))
        w.meta.update(needed_blocks=needed, used_ids=ids.copy(), tags=tags)
    elif k == 5:
        batch = 128
        ctx = rng.integers(8192, 32768, size=batch, endpoint=True)
        w = _stage_with_prefix(CONFIG_NAMES[5], rng, batch, 64, 8, 128, 4096, ctx - 4096)
    else:
        raise ValueError(f"unknown configuration {k}")
    w.meta["config"] = k
    w.meta["seed"] = seed
    w.meta["description"] = CONFIG_DESCRIPTIONS[k]
    if values:
        _fill_values(w, seed)
    return w


def group_starts(w: Workload) -> np.ndarray:
    """First sequence of each group of a workload whose sequences come in
    consecutive groups (``meta["groups"]``), plus the batch size at the end."""
    g = np.asarray(w.meta["groups"])
    assert np.all(np.diff(g) >= 0), "groups must be consecutive"
    return np.concatenate([[0], np.flatnonzero(np.diff(g)) + 1, [g.size]]).astype(np.int32)


def grouped_case(seed: int, hq: int, hkv: int, d: int, prefix_tokens: int, group_sizes,
                 mid_tokens: int, suffix_lens) -> Workload:
    """A small stage batch with two levels of sharing: all sequences share
    ``prefix_tokens``, and the sequences of each group (consecutive, sizes
    ``group_sizes``) share ``mid_tokens`` more; random N(0,1) bf16 values."""
    rng = np.random.default_rng(seed)
    groups = np.repeat(np.arange(len(group_sizes)), group_sizes)
    w = _stage_with_prefix("grouped_case", rng, int(groups.size), hq, hkv, d, prefix_tokens,
                           np.asarray(suffix_lens), mid_groups=list(groups), mid_tokens=mid_tokens)
    return _fill_values(w, seed)


# --------------------------------------------------------------------------
# small cases for pins and edge tests
# --------------------------------------------------------------------------

@dataclass
class LogicalCase:
    """Un-paged inputs: per sequence K/V as [Hkv][n][D] bf16 bits."""

    q: np.ndarray                 # uint16 [B][Hq][D]
    k: list                       # per sequence uint16 [Hkv][n_b][D]
    v: list
    scale: float
    num_kv_heads: int
    prefix_len: int = 0

    @property
    def context_lens(self):
        return np.array([x.shape[1] for x in self.k], dtype=np.int32)


def logical_case(seed: int, batch: int, hq: int, hkv: int, d: int, ctx_lens,
                 prefix_len: int = 0, scale: float | None = None) -> LogicalCase:
    """Random N(0,1) bf16 inputs before paging; the first ``prefix_len``
    tokens of every sequence are identical (a shared prompt)."""
    rng = np.random.default_rng(seed)
    ctx_lens = [int(n) for n in ctx_lens]
    assert all(n >= prefix_len for n in ctx_lens)
    q = f32_to_bf16_bits(rng.standard_normal((batch, hq, d), dtype=np.float32))
    pk = f32_to_bf16_bits(rng.standard_normal((hkv, prefix_len, d), dtype=np.float32))
    pv = f32_to_bf16_bits(rng.standard_normal((hkv, prefix_len, d), dtype=np.float32))
    ks, vs = [], []
    for n in ctx_lens:
        sk = f32_to_bf16_bits(rng.standard_normal((hkv, n - prefix_len, d), dtype=np.float32))
        sv = f32_to_bf16_bits(rng.standard_normal((hkv, n - prefix_len, d), dtype=np.float32))
        ks.append(np.concatenate([pk, sk], axis=1))
        vs.append(np.concatenate([pv, sv], axis=1))
    return LogicalCase(q=q, k=ks, v=vs, scale=(1.0 / math.sqrt(d)) if scale is None else scale,
                       num_kv_heads=hkv, prefix_len=prefix_len)


def page_case(case: LogicalCase, seed: int, share_prefix: bool = True, extra_blocks: int = 3,
              poison: bool = False, table_pad: int = 2, name: str = "case",
              partition_size: int = 512) -> Workload:
    """Scatter a logical case into a randomly placed block pool.

    With ``share_prefix`` the whole blocks of the common prefix are stored
    once and referenced from every table.  ``poison`` fills every slot that a
    correct kernel must not use (rows past a sequence's context in its last
    block, and unused blocks) with K = 8192 on dim 0 and V = NaN; otherwise
    those slots hold N(0,1) values (stale data).
    """
    rng = np.random.default_rng(seed)
    B, hq, d = case.q.shape
    hkv = case.num_kv_heads
    ctx = case.context_lens
    nblocks = [_nblk(int(n)) for n in ctx]
    n_shared = (case.prefix_len // BLOCK_SIZE) if (share_prefix and B > 1) else 0
    needed = n_shared + sum(m - n_shared for m in nblocks)
    nb = needed + extra_blocks
    perm = rng.permutation(nb).astype(np.int32)
    shape = (nb, hkv, BLOCK_SIZE, d)
    if poison:
        kp = np.zeros(shape, np.uint16); kp[..., 0] = 0x4600  # 8192.0
        vp = np.full(shape, BF16_QNAN, np.uint16)
    else:
        kp = f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
        vp = f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    shared_ids = perm[:n_shared]
    cursor = n_shared
    lists = []
    for b in range(B):
        n = int(ctx[b])
        ids = list(shared_ids) + list(perm[cursor: cursor + nblocks[b] - n_shared])
        cursor += nblocks[b] - n_shared
        lists.append(ids)
        for j, pid in enumerate(ids):
            lo, hi = j * BLOCK_SIZE, min(n, (j + 1) * BLOCK_SIZE)
            kp[pid, :, : hi - lo, :] = case.k[b][:, lo:hi, :]
            vp[pid, :, : hi - lo, :] = case.v[b][:, lo:hi, :]
    width = max(nblocks) + table_pad if B else 1
    w = Workload(name=name, batch=B, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                 num_blocks=nb, context_lens=ctx.astype(np.int32),
                 block_tables=_tables_from_lists(lists, width), scale=case.scale,
                 partition_size=partition_size, q=case.q.copy(), k_pool=kp, v_pool=vp)
    w.meta.update(needed_blocks=needed, used_ids=perm[:needed].copy(), shared_blocks=n_shared)
    return w


def permute_blocks(w: Workload, seed: int) -> Workload:
    """Same logical inputs, every physical block moved by one random permutation."""
    rng = np.random.default_rng(seed)
    pi = rng.permutation(w.num_blocks).astype(np.int32)   # old id -> new id
    k = np.empty_like(w.k_pool); v = np.empty_like(w.v_pool)
    k[pi] = w.k_pool; v[pi] = w.v_pool
    bt = w.block_tables.copy()
    m = bt >= 0
    bt[m] = pi[bt[m]]
    return replace(w, block_tables=bt, k_pool=k, v_pool=v, meta=dict(w.meta, permutation=pi))


def duplicate_shared_blocks(w: Workload) -> Workload:
    """Give every sequence a private copy of each block it shares with others."""
    refs: dict[int, int] = {}
    for b in range(w.batch):
        for j in range(_nblk(int(w.context_lens[b]))):
            pid = int(w.block_tables[b, j]); refs[pid] = refs.get(pid, 0) + 1
    extra = sum(c - 1 for c in refs.values() if c > 1)
    nb = w.num_blocks + extra
    k = np.concatenate([w.k_pool, np.zeros((extra,) + w.k_pool.shape[1:], np.uint16)])
    v = np.concatenate([w.v_pool, np.zeros((extra,) + w.v_pool.shape[1:], np.uint16)])
    bt = w.block_tables.copy()
    nxt = w.num_blocks
    first_owner: dict[int, int] = {}
    for b in range(w.batch):
        for j in range(_nblk(int(w.context_lens[b]))):
            pid = int(bt[b, j])
            if refs[pid] > 1:
                if pid not in first_owner:
                    first_owner[pid] = b
                else:
                    k[nxt] = w.k_pool[pid]; v[nxt] = w.v_pool[pid]
                    bt[b, j] = nxt; nxt += 1
    return replace(w, num_blocks=nb, block_tables=bt, k_pool=k, v_pool=v,
                   meta=dict(w.meta, duplicated=extra))


# --------------------------------------------------------------------------
# stage demand for the isolated-vs-shared footprint experiment
# --------------------------------------------------------------------------

GENERATOR_PROMPT = 2048    # schema prompt tokens of the SQL-generator stage
FIXER_PROMPT = 2048        # schema prompt tokens of the SQL-error-fixer stage
FIRST_ATTEMPT = 256        # a fixer request's failed first attempt, shared by its retries


def stage_units(seed: int, n_units: int):
    """Seeded demand of the two LLM stages as in configurations 2 and 3:
    alternately a generator call (its tokens after the prompt: U[64, 512])
    and a fixer request (1..5 retries, each U[128, 1024] tokens after the
    prompt and the first attempt).  Returns [(stage, [suffix tokens, ...])]."""
    rng = np.random.default_rng(seed)
    units = []
    for i in range(n_units):
        if i % 2 == 0:
            units.append(("generator", [int(rng.integers(64, 512, endpoint=True))]))
        else:
            r = int(rng.integers(1, 5, endpoint=True))
            units.append(("fixer", [int(x) for x in rng.integers(128, 1024, size=r, endpoint=True)]))
    return units


def batch_from_tables(name: str, tables, context_lens, num_blocks: int, hq: int, hkv: int,
                      d: int, seed: int, k_pool=None, v_pool=None, meta=None) -> Workload:
    """A decode batch over given block tables: N(0,1) bf16 queries (and pools,
    unless given) from seed."""
    w = Workload(name=name, batch=len(tables), num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                 num_blocks=num_blocks, context_lens=np.asarray(context_lens, dtype=np.int32),
                 block_tables=_tables_from_lists(tables), scale=1.0 / math.sqrt(d))
    if k_pool is None:
        shape = (num_blocks, hkv, BLOCK_SIZE, d)
        k_pool = normal_bf16(shape, seed, STREAM_K)
        v_pool = normal_bf16(shape, seed, STREAM_V)
    w.k_pool, w.v_pool = k_pool, v_pool
    w.q = normal_bf16((w.batch, hq, d), seed, STREAM_Q)
    w.meta.update(meta or {})
    return w
