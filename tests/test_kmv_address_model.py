"""Host model of the fused kernel's buffer-load addresses (CPU only).

The fused kernel (paper_1806_06144_amd/csrc/kmv.hip) reads queries, centres
and weights with raw buffer loads: address = descriptor base + voffset +
soffset, where the descriptor's range check sees voffset only (a load whose
voffset is at or past the descriptor's extent returns zero and touches no
memory; soffset is added unchecked). This module restates the kernel's
offset arithmetic in numpy, lane by lane, and asserts that every load that
is not dropped by the range check lies inside the buffer the caller owns:

* queries Q: nq rows of length d at stride ldq (the caller's rows end at
  d, the last row at (nq - 1) ldq + d floats),
* centres C: nc rows likewise,
* weights W: round_up(nc, 256) rows of ldw floats plus a 16-byte tail.

It covers the ragged cases n mod 32 and n_z mod 64 in 1..63 that the
vector body sees in its last centre tile and its last query tile. A second
model with the row offsets of the second centre block and of the later
query rows in soffset (as the kernel once had them) must fail, which shows
the model can see the fault it guards against.
"""

import numpy as np
import pytest

KBM, KBN, KTILE, KRDC, KRP = 64, 256, 32, 16, 4
KOOB = 0x40000000
TAIL = 16


def batch_chunks(d):
    nchunk = -(-d // KRDC)
    return 8 if nchunk % 8 == 0 or nchunk % 8 > 4 else 4


class Violation(AssertionError):
    pass


def _check(what, voff, soff, nbytes, extent, lo, hi, row_len=None, ld=None):
    """Loads of `nbytes` at voff + soff (bytes, relative to the descriptor
    base, which sits at byte `lo` of the buffer) that pass the range check
    must lie in [0, hi) of the buffer and, for row data, within one row's
    first row_len floats."""
    voff = np.asarray(voff, dtype=np.int64)
    soff = np.asarray(soff, dtype=np.int64)
    voff, soff = np.broadcast_arrays(voff, soff)
    taken = voff < extent
    addr = lo + voff[taken] + soff[taken]
    if addr.size == 0:
        return
    if addr.min() < 0 or (addr + nbytes).max() > hi:
        bad = addr[(addr < 0) | (addr + nbytes > hi)]
        raise Violation(f"{what}: load at byte {int(bad[0])} outside [0, {hi})")
    if row_len is not None:
        col = addr % (ld * 4)
        if (col + nbytes).max() > row_len * 4:
            raise Violation(f"{what}: load past the end of a row")


def model_w16(ldw, lt16, w_lo, w_alloc):
    """Weight loads of the 16-wide contraction for one tile: wave w takes
    centre quarter w >> 1; lane l reads lt16 contiguous floats of row
    64 cq + 4 st + l/16, starting at column lt16 (l % 16), as 16-byte loads
    and 4-byte ones for the rest; row offsets of the k-step in soffset."""
    lane = np.arange(64)
    ldw4 = ldw * 4
    wext = KBN * ldw * 4 + TAIL
    voff0 = ((lane >> 4) * ldw + lt16 * (lane & 15)) * 4
    for wave in range(8):
        cq = wave >> 1
        for st in range(16):
            soff = (64 * cq + 4 * st) * ldw4
            a = 0
            while a < lt16:
                nbytes = 16 if a + 4 <= lt16 else 4
                voff = voff0 + 4 * a
                _check("weight16", voff, soff, nbytes, wext, w_lo, w_alloc)
                col = (voff % ldw4) + nbytes
                if col.max() > ldw4:
                    raise Violation("weight16: load past the end of a weight row")
                a += 4 if nbytes == 16 else 1


def model_vec(nq, nc, d, ldw, lt, ltw, wl, wj, cps, soffset_rows=False, t0=0, lt16=0):
    """All loads of one vector-body launch (every query tile and split)."""
    ldq = ldc = d
    krb = batch_chunks(d)
    krf = KRDC * krb
    kqpr = krf // 4
    krowstep = 512 // kqpr
    nchunk = -(-d // KRDC)
    nbt = -(-nchunk // krb)
    tq = -(-nq // KBM)
    nsplit = -(-nc // cps)
    tid = np.arange(512)
    lane = tid & 63
    q_alloc = ((nq - 1) * ldq + d) * 4
    c_alloc = ((nc - 1) * ldc + d) * 4
    w_rows = -(-nc // KBN) * KBN
    w_alloc = (w_rows * ldw) * 4 + TAIL
    # queries
    qst_row, qst_qq = tid // kqpr, tid % kqpr
    qst_col = 4 * qst_qq
    qst_voff = qst_row * ldq * 4 + 16 * qst_qq
    qst_step = krowstep * ldq * 4
    for qt in range(tq):
        q0 = qt * KBM
        q_rows = min(KBM, nq - q0)
        ext = ((q_rows - 1) * ldq + d) * 4
        for bi in range(nbt + 1):            # + the batch after the last (invalid)
            f0 = bi * krf
            valid = bi < nbt
            for part in range(krb // KRP):
                for i in range(2):
                    ok = valid & (f0 + qst_col < d)
                    if soffset_rows:
                        voff = np.where(ok, qst_voff, KOOB)
                        soff = f0 * 4 + (2 * part + i) * qst_step
                    else:
                        voff = np.where(ok, qst_voff + (2 * part + i) * qst_step, KOOB)
                        soff = f0 * 4
                    _check("query", voff, soff, 16, ext, q0 * ldq * 4, q_alloc, d, ldq)
    # centres and weights, per split and tile
    q4 = lane >> 4
    for sp in range(nsplit):
        cb = sp * cps
        ce = min(nc, cb + cps)
        ntile = -(-(ce - cb) // KBN)
        for t in range(ntile):
            c0 = cb + t * KBN
            ext = ((ce - c0 - 1) * ldc + d) * 4
            for wave in range(8):
                c_voff = ((wave * 32 + (lane & 15)) * ldc + 4 * q4) * 4
                c_blk = 16 * ldc * 4
                for ch in range(nchunk + KRP):   # + the ring's look-ahead past the tile
                    f0 = ch * KRDC
                    ok = (ch < nchunk) & (f0 + 4 * q4 < d)
                    for cbk in range(2):
                        if soffset_rows:
                            voff = np.where(ok, c_voff, KOOB)
                            soff = f0 * 4 + cbk * c_blk
                        else:
                            voff = np.where(ok, c_voff + cbk * c_blk, KOOB)
                            soff = f0 * 4
                        _check("centre", voff, soff, 16, ext, c0 * ldc * 4, c_alloc, d, ldc)
                if lt16:
                    if wave == 0:
                        model_w16(ldw, lt16, c0 * ldw * 4, w_alloc)
                    continue
                # weights of this wave's contraction role
                gl, gj = wave % wl, wave // wl
                lb = gl * ltw * KTILE
                lvalid = lt * KTILE
                if not (wave < wl * wj and lb < lvalid):
                    continue
                w_col = lb + ltw * (lane & 31)
                ldw4 = ldw * 4
                w_voff = np.where(w_col < lvalid, ((lane >> 5) << 2) * ldw4 + w_col * 4, KOOB)
                nbytes = 16 if ltw >= 3 else 4 * ltw
                wext = KBN * ldw * 4 + TAIL
                for jt in range(gj, 8, wj):
                    for v in range(16):
                        soff = (jt * 32 + ((v >> 2) << 3) + (v & 3)) * ldw4
                        _check("weight", w_voff, soff, nbytes, wext,
                               (c0 * ldw + t0 * KTILE) * 4, w_alloc)


def layouts(lt):
    out = []
    for wl, wj in [(8, 1), (4, 2), (2, 4), (1, 8)]:
        ltw = -(-lt // wl)
        if ltw <= 4:
            out.append((ltw, wl, wj))
    return out


CASES = []
for nz_mod in range(1, 64, 7):            # ragged last query tile
    CASES.append((64 + nz_mod, 300 + nz_mod % 32 + 32, 36, 10))
for n_mod in range(1, 64, 5):             # ragged last centre tile (n mod 32)
    CASES.append((70, 512 + n_mod, 20, 33))
CASES += [(65, 257, 440, 144), (127, 1023, 2048 // 8, 1000 // 4), (1, 1, 4, 1), (3, 33, 196, 160)]


@pytest.mark.parametrize("nq,nc,d,l", CASES)
def test_vector_body_loads_stay_inside_the_callers_buffers(nq, nc, d, l):
    ldw = -(-l // KTILE) * KTILE
    lt = ldw // KTILE
    nct = -(-nc // KBN)
    for ltw, wl, wj in layouts(lt):
        for P in sorted({1, min(2, nct), nct}):
            cps = -(-nct // P) * KBN
            model_vec(nq, nc, d, ldw, lt, ltw, wl, wj, cps)
    lt16 = -(-l // 16)
    if lt16 <= 10:
        for P in sorted({1, nct}):
            cps = -(-nct // P) * KBN
            model_vec(nq, nc, d, ldw, lt, -(-lt // 2), 2, 4, cps, lt16=lt16)


def test_model_sees_rows_in_soffset():
    """With the second centre block and the later query rows in soffset the
    model reports loads past the caller's rows (ragged n and n_z)."""
    with pytest.raises(Violation):
        model_vec(64 + 5, 512 + 7, 36, 32, 1, 1, 8, 1, 512, soffset_rows=True)
    # the same case with the row offsets in voffset is clean
    model_vec(64 + 5, 512 + 7, 36, 32, 1, 1, 8, 1, 512)


def test_label_blocks_beyond_1024_stay_inside():
    """l > 1024 runs one pass per block of 32 label tiles with W offset by
    the block's first column."""
    l = 1100
    ldw = -(-l // KTILE) * KTILE
    lt_total = ldw // KTILE
    t0 = 32
    lt = lt_total - t0
    for ltw, wl, wj in layouts(lt):
        model_vec(70, 300, 8, ldw, lt, ltw, wl, wj, 512, t0=t0)


@pytest.mark.parametrize("l", [1, 5, 10, 16, 17, 33, 48, 70, 100, 129, 144, 150, 160])
def test_weight_loads_of_the_16_wide_contraction(l):
    """Every weight load of the 16-wide contraction (l <= 160) lies in the
    padded tile of weight rows and inside one row."""
    ldw = -(-l // KTILE) * KTILE
    lt16 = -(-l // 16)
    assert 16 * lt16 <= ldw
    nc = 700
    w_rows = -(-nc // KBN) * KBN
    w_alloc = w_rows * ldw * 4 + TAIL
    for c0 in range(0, nc, KBN):
        model_w16(ldw, lt16, c0 * ldw * 4, w_alloc)
