"""Pure-Python brute force for tiny decode-attention inputs.

TEST INFRASTRUCTURE ONLY (see ``oracle.attention``).  It pins the numpy
oracle: it works on the *un-paged* logical tensors (or on a pool through its
own per-token gather loop), decodes bf16 with ``struct``, and sums with
``math.fsum``, so it shares no arithmetic with the oracle beyond the
definition of softmax attention itself:

    out_h = sum_t exp(s_t - m) V[t] / sum_t exp(s_t - m),  s_t = scale <q_h, K[t]>

with the same contiguous head map g = floor(h / G).
"""

from __future__ import annotations

import math
import struct


def bf16_bits_to_float(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def _decode_rows(rows):
    return [[bf16_bits_to_float(x) for x in row] for row in rows]


def attend(q_row, keys, values, scale):
    """One query row against lists of key and value rows (Python floats)."""
    n = len(keys)
    d = len(q_row)
    if n == 0:
        return [0.0] * d, -math.inf
    s = [scale * math.fsum(q_row[i] * k[i] for i in range(d)) for k in keys]
    m = max(s)
    e = [math.exp(x - m) for x in s]
    z = math.fsum(e)
    out = [math.fsum(e[t] * values[t][i] for t in range(n)) / z for i in range(d)]
    return out, m + math.log(z)


def decode_logical(q_bits, k_seqs, v_seqs, scale):
    """q_bits [B][Hq][D]; k_seqs[b] = [Hkv][n_b][D] bits.  Returns out, lse lists."""
    B = len(q_bits)
    outs, lses = [], []
    for b in range(B):
        hq = len(q_bits[b])
        hkv = len(k_seqs[b])
        group = hq // hkv
        keys = [_decode_rows(k_seqs[b][g]) for g in range(hkv)]
        vals = [_decode_rows(v_seqs[b][g]) for g in range(hkv)]
        ob, lb = [], []
        for h in range(hq):
            g = h // group
            o, l = attend([bf16_bits_to_float(x) for x in q_bits[b][h]], keys[g], vals[g], scale)
            ob.append(o); lb.append(l)
        outs.append(ob); lses.append(lb)
    return outs, lses


def gather_paged(pool, table_row, n, block_size=16):
    """Per-token gather: token t -> pool[table_row[t // bs]][g][t % bs]."""
    hkv = len(pool[0])
    seq = [[] for _ in range(hkv)]
    for t in range(n):
        blk = int(table_row[t // block_size])
        for g in range(hkv):
            seq[g].append(list(pool[blk][g][t % block_size]))
    return seq


def decode_paged(q_bits, k_pool, v_pool, block_tables, context_lens, scale, block_size=16,
                 seqs=None):
    """Brute force straight from the pool, through its own gather loop."""
    seqs = range(len(q_bits)) if seqs is None else seqs
    ks, vs, qs = [], [], []
    for b in seqs:
        n = int(context_lens[b])
        ks.append(gather_paged(k_pool, block_tables[b], n, block_size))
        vs.append(gather_paged(v_pool, block_tables[b], n, block_size))
        qs.append(q_bits[b])
    return decode_logical(qs, ks, vs, scale)
