"""CPU oracle for appending a decode step's K/V to a paged KV cache.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
does.  It shares no code with the HIP path.

What it computes.  The paper keeps each stage's context resident in the cache
of its engines across the calls of the stage (paper section 2, "Cortex
Benefits"; section 3, "Agentic State"); every decode step adds the key and
value rows of the token just produced to that resident context before the
step's attention reads it.  In a paged cache the token with index t of
sequence b lives in row t mod 16 of physical block block_tables[b][t // 16],
so the append is the plain assignment

    K_pool[block_tables[b][t // 16], g, t mod 16, :] = k_new[b, g, :]
    V_pool[...same slot...]                           = v_new[b, g, :]

for every KV head g, with t = ctx_b - 1 (ctx_b counts the new token).  A
sequence with ctx_b = 0 appends nothing.  Nothing else in the pools changes.
"""

from __future__ import annotations

import numpy as np

BLOCK_SIZE = 16


def append_kv(k_pool: np.ndarray, v_pool: np.ndarray, block_tables: np.ndarray,
              context_lens: np.ndarray, k_new: np.ndarray, v_new: np.ndarray):
    """Return copies of the pools with each sequence's new token written.

    k_pool, v_pool: uint16 [NB][Hkv][16][D]; block_tables int32 [B][W];
    context_lens int [B] (new lengths, the new token included);
    k_new, v_new: uint16 [B][Hkv][D].
    """
    k = k_pool.copy()
    v = v_pool.copy()
    for b, n in enumerate(np.asarray(context_lens)):
        n = int(n)
        if n <= 0:
            continue
        t = n - 1
        phys = int(block_tables[b, t // BLOCK_SIZE])
        k[phys, :, t % BLOCK_SIZE, :] = k_new[b]
        v[phys, :, t % BLOCK_SIZE, :] = v_new[b]
    return k, v
