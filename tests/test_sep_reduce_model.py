"""CPU model of sep_rows_cols_kernel (the single-pass row and column sums of
dG * G for the separable log-gain gradients, C <= 256): every (row, column)
element is read exactly once, the row sums and the per-block column partials
are the plain sums, and the blocks cover every row."""
import numpy as np
import pytest


def sep_rows_cols_model(dG, G, rows_per_block, U=4):
    """Lane l of wave w holds columns (l mod SEG)*KPL + [0, KPL) of row
    rb + (u*4 + w)*RPW + l // SEG in step u of the iteration at rb (U steps
    per iteration, the block's four waves interleaved); a row past the block
    is loaded as the block's last row and adds nothing."""
    P, C = dG.shape
    SEG = min(C, 64)
    RPW = 64 // SEG
    KPL = C // SEG
    nblk = -(-P // rows_per_block)
    seen = np.zeros((P, C), int)
    dgt = np.full(P, np.nan)
    part = np.zeros((C, nblk))                            # column-major, as stored
    for blk in range(nblk):
        r0, r1 = blk * rows_per_block, min((blk + 1) * rows_per_block, P)
        assert r1 > r0
        red = np.zeros((4, C))
        for wave in range(4):
            cs = np.zeros((64, KPL))
            for rb in range(r0, r1, U * 4 * RPW):
                for u in range(U):
                    rs = np.zeros(64)
                    for lane in range(64):
                        r = rb + (u * 4 + wave) * RPW + lane // SEG
                        rl = min(r, r1 - 1)               # the load's row, always in range
                        assert r0 <= rl < r1
                        for k in range(KPL):
                            c = (lane % SEG) * KPL + k
                            assert 0 <= c < C
                            if r >= r1:
                                continue
                            p = dG[r, c] * G[r, c]
                            seen[r, c] += 1
                            cs[lane, k] += p
                            rs[lane] += p
                    for lane in range(0, 64, SEG):          # segmented reduction
                        r = rb + (u * 4 + wave) * RPW + lane // SEG
                        if r < r1:
                            dgt[r] = rs[lane:lane + SEG].sum()
            for lane in range(SEG):                      # rows of the wave, then waves
                for k in range(KPL):
                    red[wave, lane * KPL + k] = cs[lane::SEG, k].sum()
        part[:, blk] = red.sum(axis=0)
    return dgt, part.T, seen


@pytest.mark.parametrize("C", [1, 2, 16, 32, 64, 128, 256])
@pytest.mark.parametrize("P,rpb", [(1, 64), (5, 64), (200, 64), (1024, 64), (1000, 96)])
def test_single_pass_sums(C, P, rpb):
    rng = np.random.default_rng(C * 1000 + P)
    dG = rng.standard_normal((P, C))
    G = rng.uniform(0.5, 1.5, (P, C))
    dgt, part, seen = sep_rows_cols_model(dG, G, rpb)
    assert np.all(seen == 1)
    np.testing.assert_allclose(dgt, (dG * G).sum(axis=1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(part.sum(axis=0), (dG * G).sum(axis=0), rtol=1e-12, atol=1e-12)


def rows_per_block(P, C):
    """The backward layout's rule: about 2048 row blocks, at least one step of
    the kernel's rows (256 / min(C, 64))."""
    return max(-(-P // 2048), 256 // min(C, 64))


@pytest.mark.parametrize("C", [1, 8, 64, 128, 256])
@pytest.mark.parametrize("P", [3, 100, 4096, 9000])
def test_layout_rule_blocks(C, P):
    rpb = rows_per_block(P, C)
    assert rpb >= 256 // min(C, 64)
    assert -(-P // rpb) <= 2048
    rng = np.random.default_rng(P + C)
    dG = rng.standard_normal((P, C))
    G = rng.uniform(0.5, 1.5, (P, C))
    dgt, part, seen = sep_rows_cols_model(dG, G, rpb)
    assert np.all(seen == 1)
    np.testing.assert_allclose(dgt, (dG * G).sum(axis=1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(part.sum(axis=0), (dG * G).sum(axis=0), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- fused sums
def sep_tile_sums_model(p, tau_count, run, chunk, nchunks, A, HB, cbits, rowpart, colpart,
                        writes):
    """sep_tile_sums on one middle tile: p[k][tau] = dG*G of the element with
    tile index t = e | k << 5 | (tau >> 5) << 10 (e = tau mod 32), i.e. f =
    ((t >> 5) << A) | (run << 5) | e.  Models the LDS round trip (with the
    pad of one word per 32; each word written once, conflict-free banks), the
    per-thread row and column sums and the group sum."""
    R = 5
    qb = cbits - R
    q = run & ((1 << qb) - 1)
    M = HB + R
    pad = lambda t: t + (t >> 5)
    lds = np.full(pad((1 << M) - 1) + 1, np.nan)
    lw = np.zeros(lds.size, int)
    taus = np.arange(tau_count)
    base = (taus & 31) | ((taus >> 5) << 10)
    for k in range(32):
        a = pad(base + (k << R))
        lds[a] = p[k]
        np.add.at(lw, a, 1)
        for w in range(0, tau_count, 64):                 # 32 distinct banks per half-wave
            for h in (0, 32):
                seg = a[w + h:w + h + 32]
                if seg.size:
                    assert len(set(seg % 32)) == seg.size
    assert lw.sum() == 1 << M and lw.max() == 1
    rblock = (((chunk << qb) | q) << (A - cbits)) | (run >> qb)
    for tau in range(tau_count):                          # row hi = tau
        rs = sum(lds[pad((tau << R) + e)] for e in range(32))
        idx = (rblock << HB) + tau
        assert 0 <= idx < rowpart.size
        rowpart[idx] = rs
        writes["row"][idx] += 1
    ng = tau_count // 32
    red = np.zeros((ng, 32))
    for tau in range(tau_count):
        g, e = tau >> 5, tau & 31
        red[g, e] = sum(lds[pad((((g << 5) + i) << R) + e)] for i in range(32))
    np_ = nchunks << (A - cbits)
    for e in range(32):
        c = (q << R) | e
        idx = c * np_ + ((chunk << (A - cbits)) | (run >> qb))
        assert 0 <= idx < colpart.size
        colpart[idx] = red[:, e].sum()
        writes["col"][idx] += 1


def sep_fused_final_model(rowpart, colpart, P, C, nq, HB, rlbits):
    """sep_fused_final_kernel: storage index i = rl * 2^HB + hi -> token
    hi * 2^rlbits + rl; columns summed over their partials."""
    dgt = np.full(P, np.nan)
    hit = np.zeros(P, int)
    for i in range(P):
        n = ((i & ((1 << HB) - 1)) << rlbits) | (i >> HB)
        dgt[n] = sum(rowpart[j * P + i] for j in range(nq))
        hit[n] += 1
    assert np.all(hit == 1)
    return dgt, colpart.reshape(C, -1).sum(axis=1)


@pytest.mark.parametrize("A,HB,cbits,B,nchunks", [(14, 9, 7, 4, 1), (12, 6, 6, 8, 4),
                                                    (13, 8, 7, 2, 2), (11, 7, 11, 3, 3),
                                                    (12, 7, 5, 1, 1)])
def test_fused_separable_sums(A, HB, cbits, B, nchunks):
    """Over every (chunk, run) tile the fused partial sums, then the final
    kernel's fixed-order sums, give dg_t = row sums and dg_c = column sums of
    dG * G; every partial is written exactly once, inside its buffer."""
    R = 5
    K = A + HB
    C, P = 1 << cbits, 1 << (K - cbits)
    rng = np.random.default_rng(K + cbits)
    dGG = rng.standard_normal((nchunks, 1 << K))          # per-chunk p over the flat index f
    tau_count = 1 << (HB + R - 5)
    rowpart = np.full(nchunks * (1 << (K - R)), np.nan)
    colpart = np.full(C * (nchunks << (A - cbits)), np.nan)
    writes = {"row": np.zeros(rowpart.size, int), "col": np.zeros(colpart.size, int)}
    tau = np.arange(tau_count)
    for chunk in range(nchunks):
        for run in range(1 << (A - R)):
            p = np.empty((32, tau_count))
            for k in range(32):
                t = (tau & 31) | (k << 5) | ((tau >> 5) << 10)
                f = ((t >> R) << A) | (run << R) | (t & 31)
                p[k] = dGG[chunk, f]
            sep_tile_sums_model(p, tau_count, run, chunk, nchunks, A, HB, cbits, rowpart,
                                colpart, writes)
    assert np.all(writes["row"] == 1) and np.all(writes["col"] == 1)
    nq = nchunks << (cbits - R)
    dgt, dgc = sep_fused_final_model(rowpart, colpart, P, C, nq, HB, A - cbits)
    tot = dGG.sum(axis=0).reshape(P, C)
    np.testing.assert_allclose(dgt, tot.sum(axis=1), rtol=1e-12, atol=1e-10)
    np.testing.assert_allclose(dgc, tot.sum(axis=0), rtol=1e-12, atol=1e-10)


def sep_tile_sums_single_model(d, gt, gc, tau_count, run, chunk, nchunks, A, HB, cbits,
                               rowpart, colpart, writes):
    """sep_tile_sums_single on one 2^(HB+5)-element tile: d[k][tau] = dG (no
    gain); the exp tables hold exp(g_c) of the tile's 32 channels and exp(g_t)
    of the token of each row hi = tau."""
    R = 5
    qb = cbits - R
    q, rl = run & ((1 << qb) - 1), run >> qb
    taus = np.arange(tau_count)
    egc = np.exp(gc[(q << R) | np.arange(32)])
    egt = np.exp(gt[(taus << (A - cbits)) | rl])
    tile = np.empty((tau_count, 32))                      # [hi][e]
    for k in range(32):
        hi = k | ((taus >> 5) << 5)
        tile[hi, taus & 31] = d[k]
    rblock = (((chunk << qb) | q) << (A - cbits)) | rl
    idx = (rblock << HB) + taus
    rowpart[idx] = (tile * egc[None, :]).sum(axis=1) * egt
    np.add.at(writes["row"], idx, 1)
    np_ = nchunks << (A - cbits)
    for e in range(32):
        c = (q << R) | e
        idx = c * np_ + ((chunk << (A - cbits)) | rl)
        colpart[idx] = (tile[:, e] * egt).sum() * egc[e]
        writes["col"][idx] += 1


@pytest.mark.parametrize("A,HB,cbits,nchunks", [(12, 10, 7, 2), (13, 10, 8, 1), (11, 10, 5, 3)])
def test_fused_separable_sums_single_form(A, HB, cbits, nchunks):
    """The one-slice form with the separable exp factors applied to the row
    and column sums gives the same gradients as sums of dG * exp(g_t + g_c)."""
    R = 5
    K = A + HB
    C, P = 1 << cbits, 1 << (K - cbits)
    rng = np.random.default_rng(K + cbits + nchunks)
    dG = rng.standard_normal((nchunks, 1 << K))
    gt = 0.3 * rng.standard_normal(P)
    gc = 0.3 * rng.standard_normal(C)
    tau_count = 1 << HB
    rowpart = np.full(nchunks * (1 << (K - R)), np.nan)
    colpart = np.full(C * (nchunks << (A - cbits)), np.nan)
    writes = {"row": np.zeros(rowpart.size, int), "col": np.zeros(colpart.size, int)}
    tau = np.arange(tau_count)
    kk = np.arange(32)[:, None]
    t = (tau[None, :] & 31) | (kk << 5) | ((tau[None, :] >> 5) << 10)
    for chunk in range(nchunks):
        for run in range(1 << (A - R)):
            d = dG[chunk, ((t >> R) << A) | (run << R) | (t & 31)]
            sep_tile_sums_single_model(d, gt, gc, tau_count, run, chunk, nchunks, A, HB, cbits,
                                       rowpart, colpart, writes)
    assert np.all(writes["row"] == 1) and np.all(writes["col"] == 1)
    dgt, dgc = sep_fused_final_model(rowpart, colpart, P, C, nchunks << (cbits - R), HB,
                                     A - cbits)
    G = np.exp(gt[:, None] + gc[None, :])
    tot = dG.sum(axis=0).reshape(P, C) * G
    np.testing.assert_allclose(dgt, tot.sum(axis=1), rtol=1e-10, atol=1e-9)
    np.testing.assert_allclose(dgc, tot.sum(axis=0), rtol=1e-10, atol=1e-9)
