"""The oracle run over the sequences of a batch by a pool of worker processes.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
does.  It shares no code with the HIP path.

Nothing here computes attention.  Each worker runs the oracle's own functions
(``paged_decode``, ``split_partials``, ``extend_attention``) on a subset of the
batch's sequences with one BLAS thread, so every sequence's result has the
same bits as a single-process call with one BLAS thread, however the
sequences are divided.  The large inputs reach the workers as files in memory-backed
storage (``/dev/shm`` where it exists), mapped read-only, so the pool can be
forked once -- before the parent process touches a GPU -- and still serve
batches built afterwards.
"""

from __future__ import annotations

import multiprocessing as mp
import os
import shutil
import tempfile
from types import SimpleNamespace

import numpy as np

from .attention import paged_decode, split_partials
from .extend import extend_attention


def default_workers() -> int:
    """Worker processes: the CPUs this process may use, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _init_worker() -> None:
    # one BLAS thread per worker process: the pool supplies the parallelism
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except ImportError:
        pass


def _load(paths: dict) -> SimpleNamespace:
    return SimpleNamespace(**{k: np.load(p, mmap_mode="r") for k, p in paths.items()})


def _decode_task(args):
    paths, seqs, scale, block_size = args
    a = _load(paths)
    out, lse = paged_decode(a.q, a.k_pool, a.v_pool, a.block_tables, a.context_lens, scale,
                            block_size, seqs=seqs)
    return seqs, out, lse


def _split_task(args):
    paths, seqs, scale, partition_size, block_size = args
    a = _load(paths)
    o, lse = split_partials(a.q, a.k_pool, a.v_pool, a.block_tables, a.context_lens, scale,
                            partition_size, block_size, seqs=seqs)
    return seqs, o, lse


def _extend_task(args):
    paths, seqs, scale, block_size = args
    a = _load(paths)
    qs = np.asarray(a.q_start)
    rows = np.concatenate([np.arange(qs[b], qs[b + 1]) for b in seqs]) if seqs else np.zeros(0, np.int64)
    sub_start = np.concatenate([[0], np.cumsum([qs[b + 1] - qs[b] for b in seqs])]).astype(np.int64)
    out, lse = extend_attention(np.asarray(a.q[rows]), sub_start, a.k_pool, a.v_pool,
                                np.asarray(a.block_tables)[seqs], np.asarray(a.context_lens)[seqs],
                                scale, block_size)
    return seqs, rows, out, lse


class OraclePool:
    """A fork-started process pool that runs the oracle over sequences."""

    def __init__(self, workers: int | None = None):
        self.workers = workers or default_workers()
        self._pool = mp.get_context("fork").Pool(self.workers, initializer=_init_worker)

    def close(self) -> None:
        if self._pool is not None:
            self._pool.close()
            self._pool.join()
            self._pool = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- plumbing ---------------------------------------------------------
    @staticmethod
    def _share(arrays: dict):
        base = "/dev/shm" if os.path.isdir("/dev/shm") and os.access("/dev/shm", os.W_OK) else None
        d = tempfile.mkdtemp(prefix="oracle_", dir=base)
        paths = {}
        for name, arr in arrays.items():
            p = os.path.join(d, name + ".npy")
            arr = np.asarray(arr)
            m = np.lib.format.open_memmap(p, mode="w+", dtype=arr.dtype, shape=arr.shape)
            m[...] = arr
            m.flush()
            del m
            paths[name] = p
        return d, paths

    def _chunks(self, seqs, lengths):
        """Deal the sequences, longest first, round-robin to 4 tasks per worker."""
        order = sorted(seqs, key=lambda b: -int(lengths[b]))
        n = max(1, min(len(order), 4 * self.workers))
        return [sorted(order[i::n]) for i in range(n) if order[i::n]]

    # -- oracle calls -----------------------------------------------------
    def decode(self, q, k_pool, v_pool, block_tables, context_lens, scale, block_size: int = 16,
               seqs=None):
        """``paged_decode`` over every (or each listed) sequence."""
        B, hq, d = q.shape
        seqs = list(range(B)) if seqs is None else [int(b) for b in seqs]
        out = np.zeros((len(seqs), hq, d))
        lse = np.zeros((len(seqs), hq))
        if not seqs:
            return out, lse
        pos = {b: i for i, b in enumerate(seqs)}
        d_, paths = self._share(dict(q=q, k_pool=k_pool, v_pool=v_pool, block_tables=block_tables,
                                     context_lens=context_lens))
        try:
            tasks = [(paths, c, float(scale), block_size) for c in self._chunks(seqs, context_lens)]
            for cs, o, l in self._pool.imap_unordered(_decode_task, tasks):
                idx = [pos[b] for b in cs]
                out[idx], lse[idx] = o, l
        finally:
            shutil.rmtree(d_, ignore_errors=True)
        return out, lse

    def decode_workload(self, w, seqs=None):
        return self.decode(w.q, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale,
                           w.block_size, seqs=seqs)

    def split_partials(self, q, k_pool, v_pool, block_tables, context_lens, scale, partition_size,
                       block_size: int = 16, seqs=None):
        """``split_partials`` over every (or each listed) sequence."""
        B, hq, d = q.shape
        seqs = list(range(B)) if seqs is None else [int(b) for b in seqs]
        p_max = max(1, -(-int(np.max(np.asarray(context_lens)[seqs], initial=0)) // partition_size))
        o = np.zeros((len(seqs), hq, p_max, d))
        lse = np.full((len(seqs), hq, p_max), -np.inf)
        pos = {b: i for i, b in enumerate(seqs)}
        d_, paths = self._share(dict(q=q, k_pool=k_pool, v_pool=v_pool, block_tables=block_tables,
                                     context_lens=context_lens))
        try:
            tasks = [(paths, c, float(scale), int(partition_size), block_size)
                     for c in self._chunks(seqs, context_lens)]
            for cs, oc, lc in self._pool.imap_unordered(_split_task, tasks):
                pc = oc.shape[2]
                idx = [pos[b] for b in cs]
                o[idx, :, :pc], lse[idx, :, :pc] = oc, lc
        finally:
            shutil.rmtree(d_, ignore_errors=True)
        return o, lse

    def extend(self, q, q_start, k_pool, v_pool, block_tables, context_lens, scale,
               block_size: int = 16):
        """``extend_attention`` over the whole batch."""
        total, hq, d = q.shape
        out = np.zeros((total, hq, d))
        lse = np.zeros((total, hq))
        B = len(q_start) - 1
        if B <= 0 or total == 0:
            return out, lse
        qs = np.asarray(q_start, dtype=np.int64)
        work = (np.diff(qs) * np.asarray(context_lens, dtype=np.int64)[:B]).tolist()
        d_, paths = self._share(dict(q=q, q_start=qs, k_pool=k_pool, v_pool=v_pool,
                                     block_tables=block_tables, context_lens=context_lens))
        try:
            tasks = [(paths, c, float(scale), block_size) for c in self._chunks(range(B), work)]
            for _, rows, o, l in self._pool.imap_unordered(_extend_task, tasks):
                out[rows], lse[rows] = o, l
        finally:
            shutil.rmtree(d_, ignore_errors=True)
        return out, lse
