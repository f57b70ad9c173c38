"""The leaf-id line schedule of the fast kernels, restated on the CPU.

Leaf ids leave as whole 128-byte lines of the output: row r's lines begin at
trees congruent to -(b + r T) mod 32 (b: the output's offset within a line,
in ints), and after every fourth tree the rows whose line just ended hand
their last 32 ids to the wave, which stores them. Lines that end with a chunk
leave at the start of the next chunk; with leaf records read from global
memory (TT mode 2) the ids are taken one chunk late and every pass moves with
them. This restatement of the kernel's slot arithmetic checks that, for every
chunk size, line offset, tree count and tree split, each (row, tree) id is
written exactly once, from the slot that holds that tree at that moment.
"""
import numpy as np
import pytest


def phases(T, b):
    """Byte k lists the residues r mod 8 whose lines begin at trees 4k mod 32."""
    ph = 0
    for rho in range(8):
        phi = (32 - (b + T * rho) % 32) % 32
        ph |= 1 << (8 * (phi // 4) + rho)
    return ph


def run_schedule(T, b, n_rows, TC, split_groups=None, lag=False):
    n_groups = (T + 31) // 32
    CPF = 32 // TC
    n_chunks = n_groups * CPF
    parts = [(0, n_chunks)] if not split_groups else [(g * CPF, min((g + split_groups) * CPF, n_chunks)) for g in range(0, n_groups, split_groups)]
    ph = phases(T, b)
    out = np.full((n_rows, T), -1, np.int64)
    cnt = np.zeros((n_rows, T), np.int64)
    def pas(slots, r0w, rho, t_end, c, lo):
        for lane in range(64):
            i, k = lane >> 3, lane & 7
            slot = (c + 4 * k) & 31
            row = r0w + rho + 8 * i
            t0 = t_end - 31 + 4 * k
            if row < n_rows and t0 >= lo and t0 < T:
                for q in range(4):
                    tree = slots[row - r0w][(slot + q) & 31]
                    assert tree == t0 + q, (tree, t0 + q, lag, TC)
                    out[row, t0 + q] = tree
                    cnt[row, t0 + q] += 1
    def passes_at(slots, r0w, cc, t_end, lo):
        m = (ph >> (8 * (cc >> 2))) & 0xff
        for rho in range(8):
            if m >> rho & 1: pas(slots, r0w, rho, t_end, cc, lo)
    def leaves(slots, r0w, QP, tb, t_begin):
        for g in range(TC):
            t = tb + g
            assert (QP * TC + g) == t % 32
            for l in range(64):
                slots[l][t % 32] = t
                if t % 2 == 0: slots[l][t % 32 + 1] = None
            if ((QP * TC + g) & 3) == 3 and g < TC - 1:
                passes_at(slots, r0w, (QP * TC + g + 1) & 31, t, t_begin)
    L = 1 if lag else 0
    for (cb, ce) in parts:
        t_begin = cb * TC
        for r0w in range(0, n_rows, 64):
            slots = [[None] * 32 for _ in range(64)]
            for c in range(cb, ce):
                Q = (c - cb) % CPF
                t0 = c * TC
                kQE = (Q + CPF - L) % CPF
                if ((kQE * TC) & 3) == 0 and t0 - L * TC > t_begin:
                    passes_at(slots, r0w, (kQE * TC) & 31, t0 - L * TC - 1, t_begin)
                if lag:
                    if t0 > t_begin: leaves(slots, r0w, (Q + CPF - 1) % CPF, t0 - TC, t_begin)
                else:
                    leaves(slots, r0w, Q, t0, t_begin)
            t_pad = ce * TC
            if lag:
                t_last = t_pad - TC
                kC = ((CPF - 1) * TC) & 31
                if (kC & 3) == 0 and t_last > t_begin:
                    passes_at(slots, r0w, kC, t_last - 1, t_begin)
                leaves(slots, r0w, CPF - 1, t_last, t_begin)
            for k in range(0, 8):
                m = (ph >> (8 * k)) & 0xff
                for rho in range(8):
                    if m >> rho & 1: pas(slots, r0w, rho, t_pad - 1, 0, max(t_begin, t_pad - 32 + 4 * k))
    assert (cnt == 1).all(), (T, b, TC, lag, np.argwhere(cnt != 1)[:5])
    assert (out == np.arange(T)[None, :]).all()



@pytest.mark.parametrize("lag", [False, True])
@pytest.mark.parametrize("T", [4, 28, 36, 64, 100, 500])
def test_every_id_written_once(lag, T):
    for b in range(0, 32, 4):
        for TC in ([1, 2, 4, 8] if lag else [1, 2, 4, 8, 16, 32]):
            for split in (None, 1, 2):
                run_schedule(T, b, 70, TC, split, lag)
