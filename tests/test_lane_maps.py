"""Host simulation of the LDS staging layouts of the matrix-core bodies
(csrc/mfma_body.h: k_arow, k_stage, v_stage, v_tr), restated here.

* The transposing read (ds_read_b64_tr_b16) is modelled as measured on
  gfx950 with an in-bounds probe: within each group of 16 lanes, lane i
  receives element i % 4 of the 8-byte chunks addressed by lanes 4k + i // 4
  of its group, k = 0..3.
* Staged V tiles written through v_stage and read through v_tr must hand
  lane (q, n) V[token q + 4k][dim 16j + n], the B operand of output column n
  of PV instruction j.
* The staged K layout must give the A operand (row k_arow(n), chunk 4s + q)
  and keep writers and readers on 16 distinct 16-byte positions per
  instruction and row group.
"""
import numpy as np


def k_arow(n):
    return 4 * (n & 3) + (n >> 2)


def k_stage(r, c):
    return r * 256 + ((c ^ k_arow(r)) << 4)


def v_swz(r):
    return (r ^ (r >> 2)) & 7


def v_stage(r, c):
    return r * 256 + ((((c >> 1) ^ v_swz(r)) << 5) | ((c & 1) << 4))


def v_tr(q, n):
    r = q + 4 * (n >> 2)
    return r * 256 + (v_swz(r) << 5) + ((n & 3) << 3)


def bank_conflict_degree(addrs, width, lanes):
    """Worst number of distinct 4-byte words per bank (32 banks) over groups of
    `lanes` consecutive lanes, each lane accessing `width` bytes."""
    worst = 0
    for g in range(0, len(addrs), lanes):
        words = {}
        for a in addrs[g:g + lanes]:
            for w in range(width // 4):
                words.setdefault((a // 4 + w) % 32, set()).add(a // 4 + w)
        worst = max(worst, max(len(v) for v in words.values()))
    return worst


def stage(tile, place):
    """Write a [16][128] tile of shorts as 16-byte chunks through place(row, chunk)."""
    lds = np.full(2048, -1, dtype=np.int64)
    for r in range(16):
        for c in range(16):
            b = place(r, c)
            assert b % 16 == 0 and 0 <= b and b + 16 <= 4096
            assert (lds[b // 2:b // 2 + 8] == -1).all(), "two chunks on one slot"
            lds[b // 2:b // 2 + 8] = tile[r, 8 * c:8 * c + 8]
    assert (lds >= 0).all()
    return lds


def tr_read(lds, addr):
    """ds_read_b64_tr_b16 on 64 lanes with byte addresses addr[lane]."""
    out = np.zeros((64, 4), dtype=np.int64)
    for lane in range(64):
        g, i = lane >> 4, lane & 15
        for k in range(4):
            a = addr[16 * g + 4 * k + i // 4]
            assert a % 8 == 0 and 0 <= a and a + 8 <= 4096
            out[lane, k] = lds[a // 2 + i % 4]
    return out


def test_v_tr_reads_give_the_pv_b_operand():
    v = np.arange(16 * 128).reshape(16, 128)
    lds = stage(v, v_stage)
    for j in range(8):
        got = tr_read(lds, [v_tr(lane >> 4, lane & 15) ^ (j << 5) for lane in range(64)])
        for lane in range(64):
            q, n = lane >> 4, lane & 15
            assert list(got[lane]) == [v[q + 4 * k, 16 * j + n] for k in range(4)]


def test_v_tr_reads_are_free_of_bank_conflicts():
    """Each 16-lane group of a transposing read reaches 32 distinct banks
    (the former window position r & 7 put a group's four rows on the same
    eight banks: 4-way conflicts)."""
    for j in range(8):
        addrs = [v_tr(lane >> 4, lane & 15) ^ (j << 5) for lane in range(64)]
        assert bank_conflict_degree(addrs, 8, 16) == 1
    old = [(q + 4 * (n >> 2)) * 256 + (((q + 4 * (n >> 2)) & 7) << 5) + ((n & 3) << 3)
           for q in range(4) for n in range(16)]
    assert bank_conflict_degree(old, 8, 16) == 4


def test_k_reads_are_free_of_bank_conflicts_per_8_lanes():
    for s in range(4):
        addrs = [k_stage(k_arow(lane & 15), 4 * s + (lane >> 4)) for lane in range(64)]
        assert bank_conflict_degree(addrs, 16, 8) == 1


def test_k_stage_gives_the_a_operand_without_conflicts():
    kt = np.arange(16 * 128).reshape(16, 128)
    lds = stage(kt, k_stage)
    for s in range(4):
        for lane in range(64):
            q, n = lane >> 4, lane & 15
            b = k_stage(k_arow(n), 4 * s + q)
            assert list(lds[b // 2:b // 2 + 8]) == list(kt[k_arow(n), 8 * (4 * s + q):8 * (4 * s + q) + 8])
        # readers of one row group (16 lanes) hit 16 distinct 16-byte positions
        for q in range(4):
            pos = {(k_stage(k_arow(n), 4 * s + q) >> 4) & 15 for n in range(16)}
            assert len(pos) == 16
    # writers: 16 lanes write the 16 chunks of one row, distinct positions
    for r in range(16):
        assert len({(k_stage(r, c) >> 4) & 15 for c in range(16)}) == 16
    assert all(k_arow(k_arow(n)) == n for n in range(16))
