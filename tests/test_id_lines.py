"""The leaf-id line schedule of the fast kernels, restated on the CPU.

Leaf ids leave as whole 128-byte lines of the output: row r's lines begin at
trees congruent to -(b + r T) mod 32 (b: the output's offset within a line,
in ints), and after every fourth tree the rows whose line just ended hand
their last 32 ids to the wave, which stores them. Lines that end with a chunk
leave at the start of the next chunk; with leaf records read from global
memory (TT mode 2) the ids are taken one chunk late and every pass moves with
them. With chunks of 8 trees the lines that end at a chunk's fourth tree also
leave at the start of the next chunk, while the ids of its last four trees
wait outside their slots, and when each of the two trees ends the lines of a
single residue both lines are staged together. This restatement of the kernel's slot arithmetic checks that, for every
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
    # chunks of 8 trees: the ids of trees 4..7 of a chunk wait outside the
    # slots until the next chunk begins, and so do the lines that end at the
    # chunk's fourth tree
    defer = TC == 8
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
    def mask(cc):
        return (ph >> (8 * (cc >> 2))) & 0xff
    def passes_at(slots, r0w, cc, t_end, lo):
        m = mask(cc)
        for rho in range(8):
            if m >> rho & 1: pas(slots, r0w, rho, t_end, cc, lo)
    def put_pending(slots, pend, QX):
        for l in range(64):
            for g in range(4):
                slots[l][QX * 8 + 4 + g] = pend[l][g]
    def deferred(slots, pend, r0w, QX, tb, lo):
        passes_at(slots, r0w, (QX * 8 + 4) & 31, tb + 3, lo)
        put_pending(slots, pend, QX)
    def leaves(slots, pend, r0w, QP, tb, t_begin):
        for g in range(TC):
            t = tb + g
            assert (QP * TC + g) == t % 32
            for l in range(64):
                if defer and g >= 4:
                    pend[l][g - 4] = t
                else:
                    slots[l][t % 32] = t
            if not defer and ((QP * TC + g) & 3) == 3 and g < TC - 1:
                passes_at(slots, r0w, (QP * TC + g + 1) & 31, t, t_begin)
    L = 1 if lag else 0
    for (cb, ce) in parts:
        t_begin = cb * TC
        for r0w in range(0, n_rows, 64):
            slots = [[None] * 32 for _ in range(64)]
            pend = [[None] * 4 for _ in range(64)]
            for c in range(cb, ce):
                Q = (c - cb) % CPF
                t0 = c * TC
                kQE = (Q + CPF - L) % CPF
                if t0 - L * TC > t_begin:
                    cC = (kQE * TC) & 31
                    m_end = mask(cC) if ((kQE * TC) & 3) == 0 else 0
                    if defer:
                        QX = (Q + 2 * CPF - 1 - L) % CPF
                        cI = (QX * 8 + 4) & 31
                        tb = t0 - (1 + L) * TC
                        m_in = mask(cI)
                        if bin(m_in).count("1") == 1 and bin(m_end).count("1") == 1:
                            # both lines staged at once: the first from the
                            # slots as they stand, the second with the
                            # pending ids in their slots
                            pas(slots, r0w, (m_in & -m_in).bit_length() - 1, tb + 3, cI, t_begin)
                            after = [row[:] for row in slots]
                            put_pending(after, pend, QX)
                            pas(after, r0w, (m_end & -m_end).bit_length() - 1, tb + TC - 1, cC, t_begin)
                            put_pending(slots, pend, QX)
                        else:
                            deferred(slots, pend, r0w, QX, tb, t_begin)
                            for rho in range(8):
                                if m_end >> rho & 1: pas(slots, r0w, rho, t0 - L * TC - 1, cC, t_begin)
                    else:
                        for rho in range(8):
                            if m_end >> rho & 1: pas(slots, r0w, rho, t0 - L * TC - 1, cC, t_begin)
                if lag:
                    if t0 > t_begin: leaves(slots, pend, r0w, (Q + CPF - 1) % CPF, t0 - TC, t_begin)
                else:
                    leaves(slots, pend, r0w, Q, t0, t_begin)
            t_pad = ce * TC
            if defer and not lag:
                deferred(slots, pend, r0w, CPF - 1, t_pad - TC, t_begin)
            if lag:
                t_last = t_pad - TC
                if defer and t_last - TC >= t_begin:
                    deferred(slots, pend, r0w, (2 * CPF - 2) % CPF, t_last - TC, t_begin)
                kC = ((CPF - 1) * TC) & 31
                if (kC & 3) == 0 and t_last > t_begin:
                    passes_at(slots, r0w, kC, t_last - 1, t_begin)
                leaves(slots, pend, r0w, CPF - 1, t_last, t_begin)
                if defer:
                    deferred(slots, pend, r0w, CPF - 1, t_last, t_begin)
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
