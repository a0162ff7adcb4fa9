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
