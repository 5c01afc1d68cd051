"""Device residency for one decode step: torch allocates, the library computes.

``PagedBatch`` copies a generated workload's pools, queries, block tables and
context lengths into device memory, registers the physical placement with
the library's block pool (claim once, retain per extra reference), allocates
the output and split-KV partials, and runs the two C-ABI calls of a step.
Nothing here computes attention.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding


def _dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


class PagedBatch:
    def __init__(self, w, device="cuda:0", partition_size: int | None = None,
                 register_blocks: bool = True, k_pool=None, v_pool=None,
                 prefix_len: int = 0, prefix_partition_size: int = 256, schedule: bool = False,
                 group_start=None, group_len: int = 0, check_tables: bool = True):
        self.w = w
        self.device = torch.device(device)
        self.partition_size = w.partition_size if partition_size is None else partition_size
        self.k = k_pool if k_pool is not None else _dev(w.k_pool, self.device)
        self.v = v_pool if v_pool is not None else _dev(w.v_pool, self.device)
        # the library cannot see a device buffer's size: the pools must hold
        # every block the handle will declare
        need = w.num_blocks * w.num_kv_heads * 16 * w.head_dim
        for name, t in (("k_pool", self.k), ("v_pool", self.v)):
            if t.numel() < need or t.element_size() != 2:
                raise ValueError(f"{name} holds {t.numel()} 16-bit values; {w.num_blocks} blocks "
                                 f"of {w.num_kv_heads} x 16 x {w.head_dim} need {need}")
        self.q = _dev(w.q, self.device)
        self.bt = _dev(w.block_tables.astype(np.int32), self.device)
        self.ctx = _dev(w.context_lens.astype(np.int32), self.device)
        self.batch, self.hq, self.d = w.batch, w.num_q_heads, w.head_dim
        self.max_ctx = w.max_context_len
        self.out = torch.zeros((self.batch, self.hq, self.d), dtype=torch.int16, device=self.device)
        self.pool = binding.kv_pool_create(w.num_blocks, binding.BLOCK_SIZE, w.num_kv_heads,
                                           w.head_dim, self.k, self.v)
        if register_blocks:
            self.register_placement()
        self.prefix_len = prefix_len
        self.prefix_partition_size = prefix_partition_size
        if check_tables and (prefix_len or group_len):
            # the shared passes read shared entries from one row: verify the
            # host tables really share them before launching
            binding.paged_attn_check_tables(self.pool, w.block_tables, w.context_lens, prefix_len,
                                            group_start if group_len else None, group_len)
        # second level: groups of consecutive sequences sharing group_len tokens after the prefix
        self.group_len = group_len
        self.group_start = None
        if group_len:
            starts = np.ascontiguousarray(group_start, dtype=np.int32)
            self.num_groups = int(starts.size - 1)
            self.max_group_size = int(np.diff(starts).max()) if self.num_groups else 1
            self.group_start = torch.from_numpy(starts).to(self.device)
            ob, lb, self.num_parts = binding.paged_attn_cascade_groups_workspace_size(
                self.batch, self.hq, self.d, self.max_ctx, self.partition_size, prefix_len,
                prefix_partition_size, group_len)
        elif prefix_len:
            ob, lb, self.num_parts = binding.paged_attn_cascade_workspace_size(
                self.batch, self.hq, self.d, self.max_ctx, self.partition_size, prefix_len,
                prefix_partition_size)
        else:
            self.num_parts = binding.paged_attn_num_partitions(self.max_ctx, self.partition_size)
            ob, lb = binding.paged_attn_workspace_size(self.batch, self.hq, self.d, self.max_ctx,
                                                       self.partition_size)
        self.part_o = torch.empty(ob // 4, dtype=torch.float32, device=self.device) if ob else None
        self.part_lse = torch.empty(lb // 4, dtype=torch.float32, device=self.device) if lb else None
        self.items = None
        if schedule:
            self.set_items(binding.paged_attn_schedule(w.context_lens, self.max_ctx,
                                                       self.partition_size, prefix_len + group_len))

    def set_items(self, items) -> None:
        """Run the per-sequence partitions from a host work list (see paged_attn_schedule)."""
        self.items = torch.from_numpy(np.ascontiguousarray(items, dtype=np.int32)).to(self.device)

    def register_placement(self) -> None:
        """Claim every block the tables use; retain shared blocks once per extra user."""
        w = self.w
        nb = (w.context_lens.astype(np.int64) + 15) // 16
        used = np.concatenate([w.block_tables[b, : nb[b]] for b in range(w.batch)]) \
            if w.batch else np.zeros(0, np.int32)
        ids, counts = np.unique(used, return_counts=True)
        binding.kv_pool_claim(self.pool, ids.tolist())
        extra = np.repeat(ids, counts - 1)
        if extra.size:
            binding.kv_pool_retain(self.pool, extra.tolist())

    @property
    def bt_stride(self) -> int:
        return int(self.w.block_tables.shape[1])

    def decode(self, stream=None, out=None, pool=None, q=None) -> None:
        """The step's decode launch; ``pool``/``q`` replace the batch's own
        (a replica of the same data at other addresses)."""
        pool = self.pool if pool is None else pool
        q = self.q if q is None else q
        if self.group_len:
            n = 0 if self.items is None else int(self.items.numel())
            binding.paged_attn_decode_cascade_groups(
                pool, q, self.bt, self.bt_stride, self.ctx, self.batch, self.hq,
                self.w.scale, self.max_ctx, self.partition_size, self.prefix_len,
                self.prefix_partition_size, self.group_start, self.num_groups, self.max_group_size,
                self.group_len, self.items if n else None, n, self.part_o, self.part_lse, stream)
            return
        if self.items is not None:
            n = int(self.items.numel())
            if self.prefix_len:
                binding.paged_attn_decode_cascade_scheduled(
                    pool, q, self.bt, self.bt_stride, self.ctx, self.batch, self.hq,
                    self.w.scale, self.max_ctx, self.partition_size, self.prefix_len,
                    self.prefix_partition_size, self.items, n, self.part_o, self.part_lse, stream)
            else:
                binding.paged_attn_decode_scheduled(
                    pool, q, self.bt, self.bt_stride, self.ctx, self.batch, self.hq,
                    self.w.scale, self.max_ctx, self.partition_size, self.items, n,
                    self.out if out is None else out, self.part_o, self.part_lse, stream)
            return
        if self.prefix_len:
            binding.paged_attn_decode_cascade(
                pool, q, self.bt, self.bt_stride, self.ctx, self.batch, self.hq,
                self.w.scale, self.max_ctx, self.partition_size, self.prefix_len,
                self.prefix_partition_size, self.part_o, self.part_lse, stream)
            return
        binding.paged_attn_decode(pool, q, self.bt, self.bt_stride, self.ctx, self.batch,
                                  self.hq, self.w.scale, self.max_ctx, self.partition_size,
                                  self.out if out is None else out, self.part_o, self.part_lse,
                                  stream)

    def append(self, k_new, v_new, stream=None, pool=None) -> None:
        """Write the new token's K and V rows (device bf16 [batch][Hkv][D])
        at position ctx - 1 of every sequence (``paged_attn_append_kv``)."""
        binding.paged_attn_append_kv(self.pool if pool is None else pool, k_new, v_new, self.bt,
                                     self.bt_stride, self.ctx, self.batch, stream)

    def decode_append(self, k_new, v_new, stream=None, out=None, pool=None, q=None) -> None:
        """``append`` and ``decode`` in one launch, in the same launch
        configuration as ``decode`` (work list, cascade, groups)."""
        pool = self.pool if pool is None else pool
        q = self.q if q is None else q
        n = 0 if self.items is None else int(self.items.numel())
        items = self.items if n else None
        if self.prefix_len or self.group_len:
            g = self.group_len > 0
            binding.paged_attn_decode_cascade_append(
                pool, q, k_new, v_new, self.bt, self.bt_stride, self.ctx, self.batch, self.hq,
                self.w.scale, self.max_ctx, self.partition_size, self.prefix_len,
                self.prefix_partition_size, self.group_start if g else None,
                self.num_groups if g else 0, self.max_group_size if g else 0, self.group_len, items,
                n, self.part_o, self.part_lse, stream)
            return
        binding.paged_attn_decode_append(pool, q, k_new, v_new, self.bt, self.bt_stride, self.ctx,
                                         self.batch, self.hq, self.w.scale, self.max_ctx,
                                         self.partition_size, items, n,
                                         self.out if out is None else out, self.part_o,
                                         self.part_lse, stream)

    def reduce(self, stream=None, out=None) -> None:
        if self.group_len:
            binding.paged_attn_reduce_cascade_groups(
                self.part_o, self.part_lse, self.ctx, self.batch, self.hq, self.d,
                self.partition_size, self.prefix_len, self.prefix_partition_size, self.group_len,
                self.num_parts, self.out if out is None else out, stream)
            return
        if self.prefix_len:
            binding.paged_attn_reduce_cascade(
                self.part_o, self.part_lse, self.ctx, self.batch, self.hq, self.d,
                self.partition_size, self.prefix_len, self.prefix_partition_size, self.num_parts,
                self.out if out is None else out, stream)
            return
        binding.paged_attn_reduce(self.part_o, self.part_lse, self.ctx, self.batch, self.hq, self.d,
                                  self.partition_size, self.num_parts,
                                  self.out if out is None else out, stream)

    def tile_spans(self) -> np.ndarray:
        """Token spans whose K/V tiles one decode step of this batch reads,
        each distinct tile once, as int32 [n][3] (sequence, first token, end
        token): the shared-prefix partitions through sequence 0's table, each
        group's shared tokens through its first sequence's table, then the
        per-sequence partitions, longest first (ties in sequence order).  For
        ``binding.pa_gather_tiles``, the step's data movement alone."""
        ctx = self.w.context_lens.astype(np.int64)
        spans = []
        L, M = self.prefix_len, self.group_len
        if L:
            pps = self.prefix_partition_size
            spans += [(0, s, min(L, s + pps)) for s in range(0, L, pps)]
        if M:
            starts = self.group_start.cpu().numpy()
            spans += [(int(s0), L, L + M) for s0, s1 in zip(starts[:-1], starts[1:]) if s1 > s0]
        first = L + M
        S = self.partition_size if self.partition_size > 0 else max(1, self.max_ctx - first)
        tail = []
        for b in range(self.batch):
            for s in range(first, int(ctx[b]), S):
                e = min(int(ctx[b]), s + S)
                tail.append((e - s, b, s, e))
        tail.sort(key=lambda x: -x[0])          # stable: ties keep (sequence, partition) order
        spans += [(b, s, e) for _, b, s, e in tail]
        return np.asarray(spans, dtype=np.int32).reshape(-1, 3)

    def gather_tiles(self, spans, num_spans, sink, stream=None, pool=None,
                     tiles_in_flight: int = 2) -> None:
        """Read the tiles of ``spans`` (device int32 [n][3]) with no arithmetic."""
        binding.pa_gather_tiles(self.pool if pool is None else pool, self.bt, self.bt_stride,
                                self.batch, spans, num_spans, sink, stream, tiles_in_flight)

    @property
    def needs_reduce(self) -> bool:
        return bool(self.prefix_len or self.group_len) or self.num_parts > 1

    def run(self, stream=None) -> None:
        """One decode step: split-KV (or cascade) decode, then the merge."""
        self.decode(stream)
        if self.needs_reduce:
            self.reduce(stream)

    def out_bits(self) -> np.ndarray:
        return self.out.cpu().numpy().view(np.uint16)

    def partials(self):
        """Split-KV partials as numpy (o [B][Hq][P][D], lse [B][Hq][P])."""
        o = self.part_o.view(self.batch, self.hq, self.num_parts, self.d).cpu().numpy()
        l = self.part_lse.view(self.batch, self.hq, self.num_parts).cpu().numpy()
        return o, l

    def close(self) -> None:
        self.pool.close()
