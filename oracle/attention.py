"""CPU oracle for batched paged decode attention.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
does.  It shares no code with the HIP path: it imports nothing from the
package and decodes bf16 itself.

What it computes.  The paper keeps each stage's prompt context resident on
the engines of its pool and lets successive calls of a stage, such as the
retries of the SQL error fixer against one schema, share that context (paper
section 1, motivating example; section 2, "Cortex Benefits").  On the GPU that
context is a paged KV cache: each sequence reaches its tokens through a block
table, and shared prompt blocks are referenced from many tables.  The decode
step of an LLM stage attends one new query row per head to the sequence's
whole cached context.  The paper gives no formula; this is textbook scaled
dot-product softmax attention over the gathered context:

    s_t   = scale * <q_h, K_g[t]>            t = 0 .. n-1,  g = floor(h / G)
    w_t   = exp(s_t - max s) / sum_u exp(s_u - max s)
    out_h = sum_t w_t V_g[t]
    lse_h = max s + ln sum_t exp(s_t - max s)

in float64, where G = Hq / Hkv (contiguous groups of query heads share a KV
head) and n = ctx includes the token being decoded.  Paging, online softmax
and split-KV are only faster routes to this same value.

Readings where the sources are silent (each one is listed in the design notes
of the repository): ctx = 0 gives a zero output and lse = -inf; table entries
past ceil(n / block_size) and rows past n are never read; the query-to-KV head
map is contiguous (h // G).
"""

from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact bf16 -> float64: the 16 bits are the top half of a float32."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def gather_sequence(k_pool: np.ndarray, v_pool: np.ndarray, table_row: np.ndarray, n: int,
                    block_size: int = 16):
    """Contiguous K and V of one sequence, float64 [Hkv][n][D].

    Token t lives in physical block table_row[t // block_size], row
    t % block_size; only the first ceil(n / block_size) table entries are used.
    """
    nkv, d = k_pool.shape[1], k_pool.shape[3]
    if n <= 0:
        z = np.zeros((nkv, 0, d))
        return z, z.copy()
    nb = (n + block_size - 1) // block_size
    ids = np.asarray(table_row[:nb], dtype=np.int64)
    k = k_pool[ids].transpose(1, 0, 2, 3).reshape(nkv, nb * block_size, d)[:, :n]
    v = v_pool[ids].transpose(1, 0, 2, 3).reshape(nkv, nb * block_size, d)[:, :n]
    return bf16_to_f64(k), bf16_to_f64(v)


def softmax_attention(q_rows: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float):
    """Textbook attention of query rows [R][D] over one context K, V [n][D].

    Returns (out [R][D], lse [R], weights [R][n]) in float64.
    """
    r, d = q_rows.shape
    n = k.shape[0]
    if n == 0:
        return np.zeros((r, d)), np.full(r, -np.inf), np.zeros((r, 0))
    s = scale * (q_rows @ k.T)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(axis=1, keepdims=True)
    w = e / z
    out = w @ v
    lse = (m + np.log(z))[:, 0]
    return out, lse, w


def kv_head_for(h: int, num_q_heads: int, num_kv_heads: int) -> int:
    """KV head serving query head h: contiguous groups of G = Hq / Hkv heads."""
    return h // (num_q_heads // num_kv_heads)


def _rows_of(g: int, hq: int, nkv: int):
    return [h for h in range(hq) if kv_head_for(h, hq, nkv) == g]


def paged_decode(q: np.ndarray, k_pool: np.ndarray, v_pool: np.ndarray,
                 block_tables: np.ndarray, context_lens: np.ndarray, scale: float,
                 block_size: int = 16, seqs=None, return_weights: bool = False):
    """Decode attention for every (or each listed) sequence of a batch.

    q: uint16 bf16 bits [B][Hq][D]; pools: uint16 [NB][Hkv][block_size][D].
    Returns out float64 [len(seqs)][Hq][D] and lse [len(seqs)][Hq]; with
    ``return_weights`` also a list of per-sequence weights [Hq][n].
    """
    B, hq, d = q.shape
    nkv = k_pool.shape[1]
    if hq % nkv:
        raise ValueError("query heads must be a multiple of KV heads")
    seqs = range(B) if seqs is None else list(seqs)
    outs, lses, ws = [], [], []
    for b in seqs:
        n = int(context_lens[b])
        K, V = gather_sequence(k_pool, v_pool, block_tables[b], n, block_size)
        qb = bf16_to_f64(q[b])
        out_b = np.zeros((hq, d)); lse_b = np.zeros(hq); w_b = np.zeros((hq, max(n, 0)))
        for g in range(nkv):
            rows = _rows_of(g, hq, nkv)
            o, l, w = softmax_attention(qb[rows], K[g], V[g], scale)
            out_b[rows], lse_b[rows], w_b[rows] = o, l, w
        outs.append(out_b); lses.append(lse_b); ws.append(w_b)
    out = np.stack(outs) if outs else np.zeros((0, hq, d))
    lse = np.stack(lses) if lses else np.zeros((0, hq))
    if return_weights:
        return out, lse, ws
    return out, lse


def decode_workload(w, seqs=None, return_weights: bool = False):
    """``paged_decode`` over a generated workload object."""
    return paged_decode(w.q, w.k_pool, w.v_pool, w.block_tables, w.context_lens, w.scale,
                        w.block_size, seqs=seqs, return_weights=return_weights)


# ---------------------------------------------------------------------------
# split-KV: per-partition partial results and their log-sum-exp merge
# ---------------------------------------------------------------------------

def split_partials(q, k_pool, v_pool, block_tables, context_lens, scale, partition_size,
                   block_size: int = 16, seqs=None):
    """Attention restricted to each partition [p*S, min((p+1)*S, n)).

    Returns o float64 [len(seqs)][Hq][P_max][D] (normalised within the
    partition) and lse [len(seqs)][Hq][P_max]; partitions at or past the end
    of a sequence hold o = 0, lse = -inf.
    """
    B, hq, d = q.shape
    nkv = k_pool.shape[1]
    seqs = range(B) if seqs is None else list(seqs)
    p_max = max(1, -(-int(np.max(context_lens[list(seqs)], initial=0)) // partition_size))
    o = np.zeros((len(seqs), hq, p_max, d))
    lse = np.full((len(seqs), hq, p_max), -np.inf)
    for i, b in enumerate(seqs):
        n = int(context_lens[b])
        K, V = gather_sequence(k_pool, v_pool, block_tables[b], n, block_size)
        qb = bf16_to_f64(q[b])
        for p in range(-(-n // partition_size)):
            lo, hi = p * partition_size, min(n, (p + 1) * partition_size)
            for g in range(nkv):
                rows = _rows_of(g, hq, nkv)
                op, lp, _ = softmax_attention(qb[rows], K[g, lo:hi], V[g, lo:hi], scale)
                o[i, rows, p], lse[i, rows, p] = op, lp
    return o, lse


def merge_partials(o: np.ndarray, lse: np.ndarray):
    """Combine partition results: weights exp(lse_p - max lse), renormalised.

    o [..., P][D], lse [..., P]; partitions with lse = -inf carry no weight and
    an all-empty row merges to zero with lse = -inf.
    """
    m = np.max(lse, axis=-1, keepdims=True)
    safe_m = np.where(np.isfinite(m), m, 0.0)
    wts = np.where(np.isfinite(lse), np.exp(lse - safe_m), 0.0)
    tot = wts.sum(axis=-1, keepdims=True)
    num = (wts[..., None] * o).sum(axis=-2)
    out = np.where(tot > 0, num / np.where(tot > 0, tot, 1.0), 0.0)
    lse_all = np.where(tot[..., 0] > 0, safe_m[..., 0] + np.log(np.where(tot[..., 0] > 0, tot[..., 0], 1.0)),
                       -np.inf)
    return out, lse_all
