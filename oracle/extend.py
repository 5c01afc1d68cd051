"""CPU oracle for paged extend (chunked prefill) attention.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
does.  It shares no code with the HIP path.

What it computes.  A retry of the SQL error fixer sends new prompt tokens
(the failed query and its error) that must attend to the stage's resident
context -- the shared schema prompt and the first attempt -- and, causally,
to each other (paper section 1, motivating example; section 2, "Cortex
Benefits").  With the chunk's K/V already appended to the paged cache, the L_b
new tokens of sequence b sit at positions n_b - L_b .. n_b - 1 (n_b =
context_lens[b]); the query of the chunk's i-th token, at position
p = n_b - L_b + i, attends to tokens 0 .. p:

    out[q_start[b] + i][h] = softmax_{t <= p}(scale * <q[q_start[b] + i][h], K_g[t]>) V_g[t]

with g = floor(h / G).  Queries and outputs are packed over the batch:
row q_start[b] + i of q[total][Hq][D] is token i of sequence b's chunk.
"""

from __future__ import annotations

import numpy as np

from .attention import bf16_to_f64, gather_sequence, softmax_attention


def extend_attention(q: np.ndarray, q_start: np.ndarray, k_pool: np.ndarray, v_pool: np.ndarray,
                     block_tables: np.ndarray, context_lens: np.ndarray, scale: float,
                     block_size: int = 16):
    """Returns out float64 [total][Hq][D] and lse [total][Hq].

    q: uint16 bf16 bits [total][Hq][D]; q_start int [B+1] (q_start[0] = 0,
    nondecreasing); chunk b has L_b = q_start[b+1] - q_start[b] <= context_lens[b].
    """
    total, hq, d = q.shape
    nkv = k_pool.shape[1]
    group = hq // nkv
    out = np.zeros((total, hq, d))
    lse = np.zeros((total, hq))
    for b in range(len(q_start) - 1):
        lo, hi = int(q_start[b]), int(q_start[b + 1])
        n = int(context_lens[b])
        L = hi - lo
        if L > n:
            raise ValueError("a chunk cannot be longer than its context")
        K, V = gather_sequence(k_pool, v_pool, block_tables[b], n, block_size)
        for i in range(L):
            p = n - L + i
            qi = bf16_to_f64(q[lo + i])
            for g in range(nkv):
                rows = list(range(g * group, (g + 1) * group))
                o, l, _ = softmax_attention(qi[rows], K[g][: p + 1], V[g][: p + 1], scale)
                out[lo + i, rows], lse[lo + i, rows] = o, l
    return out, lse
