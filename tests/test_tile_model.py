"""CPU model of the HIP kernels' tile index maps (no GPU).

Re-states, in numpy, the index arithmetic of csrc/whtmix_kernels.hip (layouts,
LDS padding, bit groups, workspace run map, gain map, block decoding) and the
plan table of csrc/whtmix_plan.h, then checks for every plan shape:

* every global load/store and every LDS access stays inside its buffer;
* each kernel reads and writes every element of its tile exactly once, and
  the tiles of a launch partition the buffer;
* executing the modelled schedule (butterflies, exchanges, gain) on data
  reproduces the CPU oracle -- i.e. the bit-group plan transforms every bit
  of the flattened index exactly once in each direction.

The model is test code only; nothing in the product path uses it.
"""
import numpy as np
import pytest

from oracle import oracle as oracle_mod

VB, V = 5, 32


def pad(t):
    return t + (t >> 5)


def layout_base(S, tau):
    return (tau & ((1 << S) - 1)) | ((tau >> S) << (S + VB))


def layout_index(S, tau):
    """[P, 32] tile indices of every thread's registers in layout S (a window
    start), or in the vector-first layout ("v", VW, M): register k holds
    t = (k mod 2^VW) | (tau << VW) | ((k >> VW) << (M - 5 + VW))."""
    k = np.arange(V)[None, :]
    if isinstance(S, tuple):
        _, vw, M = S
        return (k & ((1 << vw) - 1)) | (tau[:, None] << vw) | ((k >> vw) << (M - VB + vw))
    return layout_base(S, tau)[:, None] | (k << S)


class Groups:
    def __init__(self, M, WT):
        self.M, self.WT = M, WT
        self.TOP = M - VB
        self.JT = WT - self.TOP if WT > self.TOP else 0
        self.NBOT = (self.TOP - WT + VB - 1) // VB if self.TOP > WT else 0
        self.SL = WT + VB * (self.NBOT - 1) if self.NBOT > 0 else self.TOP

    def S(self, i):
        return self.WT + VB * i

    def NB(self, i):
        return min(VB, self.TOP - self.S(i))


class VGroups:
    """Bit groups of an outer tile whose first layout is vector-first
    (csrc/whtmix_tile.h VGroups): the first group is t bits [0, VW) and
    [M - 5 + VW, M) straight from 16-byte loads; the windows then cover
    [VW, M - 5 + VW) from the bottom."""

    def __init__(self, M, vw):
        self.M, self.WT, self.vw = M, vw, vw
        self.TOP = ("v", vw, M)
        self.JT = 0
        self.top_hi = M - VB + vw
        self.NBOT = (M - VB + VB - 1) // VB
        self.SL = vw + VB * (self.NBOT - 1)
        assert self.SL + VB <= M, "last window past the tile"

    def S(self, i):
        return self.vw + VB * i

    def NB(self, i):
        return min(VB, self.top_hi - self.S(i))


def clampi(v, lo, hi):
    return max(lo, min(hi, v))


def module_split(K):
    """The block's split (csrc/whtmix_plan.h module_split): tiles <= 2^15."""
    if K >= 16:
        A = clampi((K + 6) // 2, 11, 15)
        HB = K - A
        R = clampi(5, 11 - HB, 15 - HB)
        return A, HB, R
    return 11, K - 11, 22 - K


def three_pass_split(K):
    """The mixer's split: 2^16 outer tiles (two register sets) from K = 26."""
    if K < 26:
        return module_split(K)
    HB = K - 16
    return 16, HB, clampi(5, 11 - HB, 15 - HB)


def butterflies(v, j0, j1):
    for j in range(j0, j1):
        h = 1 << j
        for k in range(V):
            if not k & h:
                a, b = v[:, k].copy(), v[:, k | h].copy()
                v[:, k], v[:, k | h] = a + b, a - b


class Tile:
    """One workgroup: P threads x 32 registers, plus an LDS array."""

    def __init__(self, M, WT, vw=0):
        self.g = VGroups(M, vw) if vw else Groups(M, WT)
        self.P = 1 << (M - VB)
        self.tau = np.arange(self.P)
        self.lds = np.full(pad(1 << M), np.nan)
        self.lds_touched = np.zeros(pad(1 << M), bool)

    def idx(self, S):
        return layout_index(S, self.tau)

    def exchange(self, v, SA, SB):
        ia, ib = pad(self.idx(SA)), pad(self.idx(SB))
        assert ia.max() < self.lds.size and ib.max() < self.lds.size
        assert len(np.unique(ia)) == ia.size and len(np.unique(ib)) == ib.size
        self.lds[:] = np.nan
        self.lds[ia] = v
        self.lds_touched[ia] = True
        out = self.lds[ib]
        assert not np.isnan(out).any(), "read an LDS word no thread wrote"
        return out

    def forward_groups(self, v, SPREV):
        g = self.g
        for i in range(g.NBOT):
            v = self.exchange(v, SPREV, g.S(i))
            butterflies(v, 0, g.NB(i))
            SPREV = g.S(i)
        return v

    def inverse_groups(self, v):
        g = self.g
        for i in range(g.NBOT - 1, -1, -1):
            butterflies(v, 0, g.NB(i))
            snext = g.TOP if i == 0 else g.S(i - 1)
            v = self.exchange(v, g.S(i), snext)
        return v


def contig_map(t, **_):
    return t


def run_map(t, HB, R):
    return ((t >> R) << (HB + R)) | (t & ((1 << R) - 1))


def gain_map(t, A, R):
    return ((t >> R) << A) | (t & ((1 << R) - 1))


class Access:
    """Records every element offset read or written in a buffer."""

    def __init__(self, size):
        self.size = size
        self.count = np.zeros(size, np.int64)

    def at(self, offs):
        if offs.size == 0:
            return offs
        assert offs.min() >= 0 and offs.max() < self.size, "out of bounds"
        np.add.at(self.count, offs.reshape(-1), 1)
        return offs


def tile_valid(nvalid, hi, A):
    start = hi << A
    return 0 if nvalid <= start else min(nvalid - start, 1 << A)


def outer_sets(A, vw=0):
    """Register sets of an outer tile: (tile, offset of the set's t) -- one
    2^A tile, or for A = 16 two 2^15 sub-tiles at t and t + 2^15.  vw: the
    vector-first layout for 2^vw-element global accesses (0: the top window)."""
    if A <= 15:
        return [(Tile(A, 0, vw), 0)]
    return [(Tile(15, 0, vw), 0), (Tile(15, 0, vw), 1 << 15)]


def outer_vw(A, elt_bytes, nvalid, widths={2: 3, 4: 0}):
    """csrc/whtmix_tile.h vec_width / use_vec: the vector width of an outer
    pass (log2 of the elements per 16-byte access), or 0 for per-element
    accesses.  The kernels use it for bf16 only; `widths` lets the model
    exercise the layout's float32 form (VW = 2) too."""
    vw = widths[elt_bytes]
    M = min(A, 15)
    if vw == 0 or (nvalid * elt_bytes) % 16 != 0 or vw + VB * ((M - VB + VB - 1) // VB) > M:
        return 0
    return vw


def cross(v0, v1):
    return v0 + v1, v0 - v1


def model_outer_fwd_block(src, nvalid, b, hi, split, acc=None, vw=0):
    """One outer_fwd block (outer_fwd_tile / outer_fwd_tile2): returns the
    workspace offsets (relative to the slice) and values of its tile."""
    A, HB, R = split
    valid = tile_valid(nvalid, hi, A)
    sets = outer_sets(A, vw)
    vals = []
    for T, t0 in sets:
        t = T.idx(T.g.TOP) + t0
        v = np.zeros(t.shape)
        m = t < valid
        o = b * nvalid + (hi << A) + t[m]
        v[m] = src[acc.at(o) if acc is not None else o]
        vals.append(v)
    if len(sets) == 2:
        vals = list(cross(*vals))
    offs, out = [], []
    for (T, t0), v in zip(sets, vals):
        butterflies(v, 0, VB)
        v = T.forward_groups(v, T.g.TOP)
        offs.append((hi << R) + run_map(T.idx(T.g.SL) + t0, HB, R))
        out.append(v)
    return offs, out


def model_outer_inv_block(ws_slice, nvalid, b, hi, split, acc=None, base=0, vw=0):
    """One outer_inv block: returns (y offsets, values) of its valid elements."""
    A, HB, R = split
    valid = tile_valid(nvalid, hi, A)
    sets = outer_sets(A, vw)
    vals = []
    for T, t0 in sets:
        o = base + (hi << R) + run_map(T.idx(T.g.SL) + t0, HB, R)
        v = ws_slice[acc.at(o) if acc is not None else o].copy()
        v = T.inverse_groups(v)
        butterflies(v, 0, VB)
        vals.append(v)
    if len(sets) == 2:
        vals = list(cross(*vals))
    offs, out = [], []
    for (T, t0), v in zip(sets, vals):
        t = T.idx(T.g.TOP) + t0
        m = t < valid
        offs.append(b * nvalid + (hi << A) + t[m])
        out.append(v[m])
    return offs, out


KMIDDLE_MIN_WAVES = 4096


def middle_slices_per_group(B, run_bits, thread_bits):
    """Slices per forward middle workgroup (the library's rule)."""
    waves = 1 << (thread_bits - 6) if thread_bits > 6 else 1
    nb = 1
    while B % (2 * nb) == 0 and (B // (2 * nb)) * (1 << run_bits) * waves >= KMIDDLE_MIN_WAVES:
        nb *= 2
    return nb


def simulate_three_pass(x, g, K, split, vw=0, nb=None):
    """Model of outer_fwd_kernel, middle_kernel, outer_inv_kernel.  x holds
    N <= 2^K / C real tokens per slice (zero padding of the token axis).
    vw: the outer passes' vector-first layout (0: per-element accesses).
    nb: slices per middle workgroup (default: the library's rule)."""
    B = x.shape[0]
    L = 1 << K
    nvalid = x.shape[1] * x.shape[2]
    A, HB, R = split
    xs = x.reshape(B * nvalid)
    ws = np.full(B * L, np.nan)
    y = np.full(B * nvalid, np.nan)
    gf = g.reshape(L)
    acc = {k: Access(B * L) for k in ("ws_w1", "ws_r2", "ws_w2")}
    acc_x, acc_y, acc_r3 = Access(B * nvalid), Access(B * nvalid), Access(B * L)
    acc_g = Access(L)
    # outer forward: block = b * 2^HB + hi
    for blk in range(B << HB):
        b, hi = blk >> HB, blk & ((1 << HB) - 1)
        offs, vals = model_outer_fwd_block(xs, nvalid, b, hi, split, acc_x, vw)
        for o, v in zip(offs, vals):
            ws[acc["ws_w1"].at(b * L + o)] = v
    # middle: the run's gain read once, then the group's nb slices in turn;
    # nb = 1: logical tile = run * B + b with the XCD renumbering of blocks,
    # nb > 1: block = group * 2^(A-R) + run
    M = HB + R
    if nb is None:
        nb = middle_slices_per_group(B, A - R, M - VB)
    assert B % nb == 0
    nblk = (B // nb) << (A - R)
    for blk in range(nblk):
        if nb == 1:
            logical = (blk & 7) * (nblk >> 3) + (blk >> 3) if nblk % 8 == 0 else blk
            run, b0 = logical // B, logical % B
        else:
            run, b0 = blk & ((1 << (A - R)) - 1), (blk >> (A - R)) * nb
        T = Tile(M, R)
        gv = gf[acc_g.at((run << R) + gain_map(T.idx(T.g.SL), A, R))]
        for b in range(b0, b0 + nb):
            base = b * (1 << (A + HB)) + (run << M)
            v = ws[acc["ws_r2"].at(base + T.idx(T.g.TOP))].copy()
            butterflies(v, T.g.JT, VB)
            v = T.forward_groups(v, T.g.TOP)
            v = v * (gv * (1.0 / L))
            if T.g.NBOT > 0:
                v = T.inverse_groups(v)
            butterflies(v, T.g.JT, VB)
            ws[acc["ws_w2"].at(base + T.idx(T.g.TOP))] = v
    # outer inverse
    for blk in range(B << HB):
        b, hi = blk >> HB, blk & ((1 << HB) - 1)
        if tile_valid(nvalid, hi, A) == 0:
            continue
        offs, vals = model_outer_inv_block(ws, nvalid, b, hi, split, acc_r3, base=b * L, vw=vw)
        for o, v in zip(offs, vals):
            y[acc_y.at(o)] = v
    for k, a in acc.items():
        assert np.all(a.count == 1), f"{k}: elements not touched exactly once"
    assert np.all(acc_x.count == 1) and np.all(acc_y.count == 1)
    assert np.all(acc_r3.count <= 1)
    assert np.all(acc_g.count == B // nb), "each gain element read once per slice group"
    return y.reshape(x.shape)


def simulate_fused(x, g, K):
    B = x.shape[0]
    L = 1 << K
    nvalid = x.shape[1] * x.shape[2]
    xs = x.reshape(B * nvalid)
    y = np.full(B * nvalid, np.nan)
    acc_x, acc_y, acc_g = Access(B * nvalid), Access(B * nvalid), Access(L)
    for b in range(B):
        T = Tile(K, 0)
        t = T.idx(T.g.TOP)
        m = t < nvalid
        v = np.zeros(t.shape)
        v[m] = xs[acc_x.at(b * nvalid + t[m])]
        butterflies(v, T.g.JT, VB)
        v = T.forward_groups(v, T.g.TOP)
        v = v * (g.reshape(L)[acc_g.at(T.idx(T.g.SL))] * (1.0 / L))
        if T.g.NBOT > 0:
            v = T.inverse_groups(v)
        butterflies(v, T.g.JT, VB)
        y[acc_y.at(b * nvalid + t[m])] = v[m]
    assert np.all(acc_x.count == 1) and np.all(acc_y.count == 1)
    assert np.all(acc_g.count == B)
    return y.reshape(x.shape)


def simulate_fused_pair(x, g):
    """fused_pair_kernel: a 2^16 slice in one workgroup of two 2^15 register
    sets (tile bit 15 = the set), each through the 2^15 schedule; the set
    butterfly right after the load and right before the store."""
    K = 16
    B = x.shape[0]
    L = 1 << K
    nvalid = x.shape[1] * x.shape[2]
    xs = x.reshape(B * nvalid)
    y = np.full(B * nvalid, np.nan)
    acc_x, acc_y, acc_g = Access(B * nvalid), Access(B * nvalid), Access(L)
    for b in range(B):
        sets = outer_sets(16)
        vals = []
        for T, t0 in sets:
            t = T.idx(T.g.TOP) + t0
            m = t < nvalid
            v = np.zeros(t.shape)
            v[m] = xs[acc_x.at(b * nvalid + t[m])]
            vals.append(v)
        vals = list(cross(*vals))
        for i, (T, t0) in enumerate(sets):
            butterflies(vals[i], 0, VB)
            vals[i] = T.forward_groups(vals[i], T.g.TOP)
        for i, (T, t0) in enumerate(sets):
            vals[i] = vals[i] * (g.reshape(L)[acc_g.at(T.idx(T.g.SL) + t0)] * (1.0 / L))
            vals[i] = T.inverse_groups(vals[i])
            butterflies(vals[i], 0, VB)
        vals = list(cross(*vals))
        for (T, t0), v in zip(sets, vals):
            t = T.idx(T.g.TOP) + t0
            m = t < nvalid
            y[acc_y.at(b * nvalid + t[m])] = v[m]
    assert np.all(acc_x.count == 1) and np.all(acc_y.count == 1)
    assert np.all(acc_g.count == B)
    return y.reshape(x.shape)


@pytest.fixture(scope="module")
def orc():
    return oracle_mod.Oracle()


@pytest.mark.parametrize("N,C", [(1024, 64), (1000, 64), (300, 128), (65536, 1)])
def test_fused_pair_schedule(N, C, orc):
    """2^16 slices in one workgroup, padded token counts included."""
    rng = np.random.default_rng(N + C)
    P = 1 << (N - 1).bit_length()
    assert P * C == 1 << 16
    x = rng.standard_normal((2, N, C))
    g = rng.uniform(0.5, 1.5, (P, C))
    y = simulate_fused_pair(x, g)
    ref = orc.whtmix(x, g)
    assert np.max(np.abs(y - ref)) < 1e-11 * np.max(np.abs(ref))


@pytest.mark.parametrize("K", [11, 12, 13, 14, 15])
def test_fused_schedule(K, orc):
    rng = np.random.default_rng(K)
    N, C = 1 << (K - K // 2), 1 << (K // 2)
    x = rng.standard_normal((2, N, C))
    g = rng.uniform(0.5, 1.5, (N, C))
    y = simulate_fused(x, g, K)
    ref = orc.whtmix(x, g)
    assert np.max(np.abs(y - ref)) < 1e-11 * np.max(np.abs(ref))


@pytest.mark.parametrize("K", list(range(12, 19)))
def test_three_pass_schedule(K, orc):
    """Executed schedule for the forced (12..15) and automatic (16..18) splits;
    B = 3 also exercises a middle grid that is not a multiple of 8."""
    rng = np.random.default_rng(100 + K)
    N, C = 1 << (K - 6), 64
    for B in (3, 8):
        x = rng.standard_normal((B, N, C))
        g = rng.uniform(0.5, 1.5, (N, C))
        y = simulate_three_pass(x, g, K, three_pass_split(K))
        ref = orc.whtmix(x, g)
        assert np.max(np.abs(y - ref)) < 1e-11 * np.max(np.abs(ref)), (K, B)


@pytest.mark.parametrize("nb", [2, 4, 8])
def test_middle_slice_groups(nb, orc):
    """The middle pass over groups of nb slices gives the one-slice result,
    with each gain element read once per group."""
    rng = np.random.default_rng(7 + nb)
    K, B = 17, 8
    N, C = 1 << 11, 64
    x = rng.standard_normal((B, N, C))
    g = rng.uniform(0.5, 1.5, (N, C))
    y = simulate_three_pass(x, g, K, three_pass_split(K), nb=nb)
    y1 = simulate_three_pass(x, g, K, three_pass_split(K), nb=1)
    assert np.array_equal(y, y1)
    ref = orc.whtmix(x, g)
    assert np.max(np.abs(y - ref)) < 1e-11 * np.max(np.abs(ref))


def test_middle_slices_per_group_rule():
    """Groups only where the grid keeps >= 4096 waves: the 2^23-element
    slices of the four-slice stereo workload get 4; the other workloads 1."""
    def nb(B, K):
        A, HB, R = three_pass_split(K)
        return middle_slices_per_group(B, A - R, HB + R - VB)
    assert nb(4, 23) == 4 and nb(2, 23) == 2 and nb(8, 23) == 8 and nb(16, 23) == 16
    assert nb(1, 23) == 1 and nb(3, 23) == 1 and nb(6, 23) == 2
    assert nb(2, 21) == 1 and nb(32, 18) == 1 and nb(1, 26) == 1
    assert nb(32, 20) == 4 and nb(4, 26) == 4
    for B in range(1, 70):
        for K in range(12, 31):
            n = nb(B, K)
            assert B % n == 0 and n & (n - 1) == 0


@pytest.mark.parametrize("K", list(range(12, 31)))
def test_three_pass_maps_in_bounds(K):
    """Index-only check for every split up to N*C = 2^30: one representative
    block per kernel at the first, last and a middle block index, for B = 3."""
    A, HB, R = three_pass_split(K)
    L = 1 << K
    B = 3
    Mm = HB + R
    assert 11 <= A <= 16 and 11 <= Mm <= 15 and 0 <= R <= A and HB >= 1
    if K >= 26:   # 2^16 outer tiles: one more carried bit than the block's split
        assert A == 16 and R == module_split(K)[2] + 1
    To = Tile(min(A, 15), 0)
    Tm = Tile(Mm, R)
    # groups transform every tile bit in [WT, M) exactly once
    for T in (To, Tm):
        g = T.g
        bits = list(range(g.TOP + g.JT, g.M))
        for i in range(g.NBOT):
            bits += list(range(g.S(i), g.S(i) + g.NB(i)))
        assert sorted(bits) == list(range(g.WT, g.M)), (K, T.g.M)
        if g.NBOT:
            assert g.S(g.NBOT - 1) + VB <= g.M
    # the outer passes' last layout keeps 32 consecutive lanes on consecutive
    # elements (coalesced workspace runs)
    assert To.g.SL == 5
    sets = [0] if A <= 15 else [0, 1 << 15]
    for blk in (0, (B << HB) // 2, (B << HB) - 1):
        b, hi = blk >> HB, blk & ((1 << HB) - 1)
        o = np.concatenate([b * L + (hi << A) + To.idx(To.g.TOP) + t0 for t0 in sets])
        assert o.min() >= 0 and o.max() < B * L
        assert len(np.unique(o)) == o.size == 1 << A
        w = np.concatenate([b * L + (hi << R) + run_map(To.idx(To.g.SL) + t0, HB, R)
                            for t0 in sets])
        assert w.min() >= 0 and w.max() < B * L
        assert len(np.unique(w)) == w.size
        # the buffer extent of the block's workspace resource covers every offset
        assert (w - b * L - (hi << R)).max() < run_map((1 << A) - 1, HB, R) + 1
    nblk = B << (A - R)
    for blk in (0, nblk // 2, nblk - 1):
        logical = (blk & 7) * (nblk >> 3) + (blk >> 3) if nblk % 8 == 0 else blk
        run, b = logical // B, logical % B
        base = b * (1 << (A + HB)) + (run << Mm)
        t = Tm.idx(Tm.g.TOP)
        assert base + t.min() >= 0 and base + t.max() < B * L
        goff = (run << R) + gain_map(Tm.idx(Tm.g.SL), A, R)
        assert goff.min() >= 0 and goff.max() < L
    assert pad((1 << 15) - 1) < 160 * 1024 // 4   # LDS fits in 160 KiB


@pytest.mark.parametrize("K,split,vw", [(18, (16, 2, 9), 0), (20, (16, 4, 7), 3),
                                        (17, (16, 1, 10), 2), (17, (16, 1, 10), 3)])
@pytest.mark.parametrize("N_frac", [1.0, 0.93, 0.8, 0.55])
def test_pair_outer_tiles(K, split, N_frac, vw, orc):
    """2^16 outer tiles (two 2^15 register sets and a butterfly between them),
    executed on small slices by forcing A = 16.  With padding (N > P/2, so the
    padded size stays P) the straddling tile's second set is partly valid or
    wholly padding, and later tiles are all padding."""
    rng = np.random.default_rng(K + int(10 * N_frac))
    C = 64
    P = 1 << (K - 6)
    N = max(1, int(P * N_frac))
    x = rng.standard_normal((2, N, C))
    g = rng.uniform(0.5, 1.5, (P, C))
    y = simulate_three_pass(x, g, K, split, vw)
    ref = orc.whtmix(x, g)
    assert np.max(np.abs(y - ref)) < 1e-11 * np.max(np.abs(ref))
    dy = rng.standard_normal((2, N, C))
    dx_ref, dg_ref = orc.whtmix_grad(x, dy, g)
    dg, dx = simulate_grad_three_pass(x, dy, g, K, split, vw)
    assert np.max(np.abs(dg - dg_ref.reshape(-1))) < 1e-11 * np.max(np.abs(dg_ref))
    assert np.max(np.abs(dx - dx_ref)) < 1e-11 * np.max(np.abs(dx_ref))


def bank_conflicts(addr, banks):
    """Worst number of lanes of one wave (64 lanes; with 32 banks served in
    two halves of 32) that hit the same bank in one LDS access."""
    worst = 1
    for w0 in range(0, addr.shape[0], 64):
        for k in range(addr.shape[1]):
            a = addr[w0:w0 + 64, k]
            halves = [a[:32], a[32:]] if banks == 32 else [a]
            for h in halves:
                _, cnt = np.unique(h % banks, return_counts=True)
                worst = max(worst, int(cnt.max()))
    return worst


@pytest.mark.parametrize("M,vw", [(12, 2), (13, 2), (14, 2), (15, 2), (13, 3), (14, 3), (15, 3)])
def test_vector_first_layouts(M, vw):
    """The vector-first layout: each thread's 2^vw registers of one access
    are consecutive elements (one 16-byte load or store); the layouts of the
    outer pass cover the tile once each; every LDS write and read of their
    exchanges is free of bank conflicts (32 banks, a wave served by halves:
    the model the existing window layouts are built for)."""
    T = Tile(M, 0, vw)
    g = T.g
    first = T.idx(g.TOP)
    assert sorted(first.reshape(-1)) == list(range(1 << M))
    step = 1 << vw
    for j in range(V // step):
        blk = first[:, j * step:(j + 1) * step]
        assert np.all(blk == blk[:, :1] + np.arange(step)), "a 16-byte access is contiguous"
        assert np.all(blk[:, 0] % step == 0)
    layouts = [g.TOP] + [g.S(i) for i in range(g.NBOT)]
    for L in layouts:
        idx = T.idx(L)
        assert sorted(idx.reshape(-1)) == list(range(1 << M))
        assert bank_conflicts(pad(idx), 32) == 1, L
    bits = list(range(vw)) + list(range(g.top_hi, M))
    for i in range(g.NBOT):
        bits += list(range(g.S(i), g.S(i) + g.NB(i)))
    assert sorted(bits) == list(range(M)), "every tile bit transformed once"
    assert g.SL == layouts[-1] and g.SL >= 6   # 64 lanes on 64 consecutive elements


@pytest.mark.parametrize("K,vw", [(18, 2), (19, 2), (20, 3)])
def test_vector_first_schedules(K, vw, orc):
    """Executed forward and backward schedules with vector-first outer
    passes reproduce the oracle (power-of-two and padded token counts)."""
    split = three_pass_split(K)
    rng = np.random.default_rng(K * 10 + vw)
    C = 64
    P = 1 << (K - 6)
    if outer_vw(split[0], 2 if vw == 3 else 4, P * C, {2: 3, 4: 2}) != vw:
        pytest.skip("outer tile too small for this width")
    for N in (P, P - P // 8 + 3):
        x = rng.standard_normal((2, N, C))
        g = rng.uniform(0.5, 1.5, (P, C))
        ref = orc.whtmix(x, g)
        y = simulate_three_pass(x, g, K, split, vw)
        assert np.max(np.abs(y - ref)) < 1e-11 * np.max(np.abs(ref))
        dy = rng.standard_normal((2, N, C))
        dx_ref, dg_ref = orc.whtmix_grad(x, dy, g)
        dg, dx = simulate_grad_three_pass(x, dy, g, K, split, vw)
        assert np.max(np.abs(dg - dg_ref.reshape(-1))) < 1e-11 * np.max(np.abs(dg_ref))
        assert np.max(np.abs(dx - dx_ref)) < 1e-11 * np.max(np.abs(dx_ref))


def test_vector_width_rule():
    """Vector accesses need 16-byte aligned slices and a tile whose last
    window fits (bf16 from 2^13 elements; the float32 form from 2^12)."""
    assert outer_vw(12, 2, 4096) == 0 and outer_vw(13, 2, 8192) == 3
    assert outer_vw(14, 2, 1000 * 16) == 3 and outer_vw(14, 2, 1001 * 4) == 0
    assert outer_vw(16, 2, 1 << 26) == 3 and outer_vw(14, 4, 1 << 14) == 0
    f32 = {2: 3, 4: 2}
    assert outer_vw(11, 4, 4096, f32) == 0 and outer_vw(12, 4, 4096, f32) == 2
    assert outer_vw(14, 4, 4 * 1001, f32) == 2 and outer_vw(14, 4, 1001, f32) == 0


@pytest.mark.parametrize("N,C", [(1000, 2), (33, 64), (100, 64), (130, 128), (257, 64)])
def test_padded_schedules(N, C, orc):
    """Token counts that are not powers of two: the padded slice of
    P = 2^ceil(log2 N) rows, with the tiles straddling or beyond row N masked."""
    rng = np.random.default_rng(N + C)
    P = 1 << (N - 1).bit_length()
    K = (P * C).bit_length() - 1
    x = rng.standard_normal((3, N, C))
    g = rng.uniform(0.5, 1.5, (P, C))
    ref = orc.whtmix(x, g)
    if K <= 15:
        y = simulate_fused(x, g, K)
        assert np.max(np.abs(y - ref)) < 1e-11 * np.max(np.abs(ref))
    if K >= 12:
        y = simulate_three_pass(x, g, K, three_pass_split(K))
        assert np.max(np.abs(y - ref)) < 1e-11 * np.max(np.abs(ref))


def model_outer_fwd(x, K, split, vw=0):
    """outer_fwd_kernel over a batch: the low-bit transforms in the run layout."""
    B = x.shape[0]
    L = 1 << K
    nvalid = x.shape[1] * x.shape[2]
    A, HB, R = split
    xs = x.reshape(B * nvalid)
    ws = np.full(B * L, np.nan)
    for blk in range(B << HB):
        b, hi = blk >> HB, blk & ((1 << HB) - 1)
        offs, vals = model_outer_fwd_block(xs, nvalid, b, hi, split, vw=vw)
        for o, v in zip(offs, vals):
            ws[b * L + o] = v
    assert not np.isnan(ws).any()
    return ws


def chunking(B, want):
    nch = min(B, want)
    per = -(-B // nch)
    return -(-B // per), per


def grad_chunking(B, K, split):
    """Chunks of the three-pass gradient kernels: about 512 workgroups over
    the chunks and runs, one slice per chunk for 2^15-element middle tiles."""
    A, HB, R = split
    runs = 1 << (A - R)
    return chunking(B, B if HB + R == 15 else -(-512 // runs))


def simulate_grad_three_pass(x, dy, g, K, split, vw=0):
    """Model of the fused three-pass gradients: outer_fwd2 of x and dy, then
    grad_mix_middle_kernel over (chunk, run) blocks (product sum, then dY's
    gain and inverse in place), the chunk sum, and outer_inv of dY's
    workspace.  Returns (dG, dX)."""
    B = x.shape[0]
    L = 1 << K
    nvalid = x.shape[1] * x.shape[2]
    A, HB, R = split
    M = HB + R
    wsx, wsd = model_outer_fwd(x, K, split, vw), model_outer_fwd(dy, K, split, vw)
    gf = g.reshape(L)
    runs = 1 << (A - R)
    nch, per = grad_chunking(B, K, split)
    out = Access(nch * L)
    ws_w = Access(B * L)
    part = np.full(nch * L, np.nan)
    for blk in range(nch << (A - R)):
        run, chunk = blk & (runs - 1), blk >> (A - R)
        T = Tile(M, R)
        acc = np.zeros((T.P, V))
        goff = (run << R) + gain_map(T.idx(T.g.SL), A, R)
        for b in range(chunk * per, min(chunk * per + per, B)):
            off = (b << (A + HB)) + (run << M)
            vx = wsx[off + T.idx(T.g.TOP)].copy()
            vd = wsd[off + T.idx(T.g.TOP)].copy()
            butterflies(vx, T.g.JT, VB)
            butterflies(vd, T.g.JT, VB)
            vx = T.forward_groups(vx, T.g.TOP)
            vd = T.forward_groups(vd, T.g.TOP)
            acc += vx * vd
            vd = vd * (gf[goff] * (1.0 / L))
            if T.g.NBOT > 0:
                vd = T.inverse_groups(vd)
            butterflies(vd, T.g.JT, VB)
            wsd[ws_w.at(off + T.idx(T.g.TOP))] = vd
        o = out.at((chunk << (A + HB)) + (run << R) + gain_map(T.idx(T.g.SL), A, R))
        part[o] = acc / L
    assert np.all(out.count == 1)
    assert np.all(ws_w.count == 1), "dY's workspace rewritten exactly once"
    dx = np.full(B * nvalid, np.nan)
    acc_y = Access(B * nvalid)
    for blk in range(B << HB):
        b, hi = blk >> HB, blk & ((1 << HB) - 1)
        if tile_valid(nvalid, hi, A) == 0:
            continue
        offs, vals = model_outer_inv_block(wsd, nvalid, b, hi, split, base=b * L, vw=vw)
        for o, v in zip(offs, vals):
            dx[acc_y.at(o)] = v
    assert np.all(acc_y.count == 1)
    return part.reshape(nch, L).sum(axis=0), dx.reshape(x.shape)


def simulate_grad_fused(x, dy, K):
    B = x.shape[0]
    L = 1 << K
    nvalid = x.shape[1] * x.shape[2]
    nch, per = chunking(B, 1024)
    part = np.full(nch * L, np.nan)
    out = Access(nch * L)
    xs, ds = x.reshape(-1), dy.reshape(-1)
    for chunk in range(nch):
        T = Tile(K, 0)
        acc = np.zeros((T.P, V))
        for b in range(chunk * per, min(chunk * per + per, B)):
            t = T.idx(T.g.TOP)
            m = t < nvalid
            vx, vd = np.zeros(t.shape), np.zeros(t.shape)
            vx[m] = xs[b * nvalid + t[m]]
            vd[m] = ds[b * nvalid + t[m]]
            butterflies(vx, T.g.JT, VB)
            butterflies(vd, T.g.JT, VB)
            vx = T.forward_groups(vx, T.g.TOP)
            vd = T.forward_groups(vd, T.g.TOP)
            acc += vx * vd
        part[out.at((chunk << K) + T.idx(T.g.SL))] = acc / L
    assert np.all(out.count == 1)
    return part.reshape(nch, L).sum(axis=0)


@pytest.mark.parametrize("B,N,C", [(3, 64, 64), (5, 1000, 16), (2, 4096, 8), (40, 128, 128),
                                   (2, 300, 64), (7, 2048, 32), (3, 512, 2)])
def test_grad_schedules(B, N, C, orc):
    """The backward schedules reproduce the oracle's gain gradient, and the
    fused three-pass schedule also its dX."""
    rng = np.random.default_rng(B * N + C)
    P = 1 << (N - 1).bit_length()
    K = (P * C).bit_length() - 1
    x = rng.standard_normal((B, N, C))
    dy = rng.standard_normal((B, N, C))
    g = rng.uniform(0.5, 1.5, (P, C))
    dx_ref, ref = orc.whtmix_grad(x, dy, g)
    ref = ref.reshape(-1)
    if K <= 15:
        got = simulate_grad_fused(x, dy, K)
        _, ref1 = orc.whtmix_grad(x, dy, np.ones((P, C)))
        ref1 = ref1.reshape(-1)
        assert np.max(np.abs(got - ref1)) < 1e-11 * np.max(np.abs(ref1))
    if K >= 12:
        got, dx = simulate_grad_three_pass(x, dy, g, K, three_pass_split(K))
        assert np.max(np.abs(got - ref)) < 1e-11 * np.max(np.abs(ref))
        assert np.max(np.abs(dx - dx_ref)) < 1e-11 * np.max(np.abs(dx_ref))


@pytest.mark.parametrize("K", list(range(12, 31)))
@pytest.mark.parametrize("B", [1, 2, 3, 4, 7, 32, 1000])
def test_grad_chunking(K, B):
    """Chunks cover the batch exactly once; 2^15-element middle tiles get one
    slice per chunk (the only form their 1024-thread kernel has)."""
    split = three_pass_split(K) if K >= 16 else (11, K - 11, 22 - K)
    nch, per = grad_chunking(B, K, split)
    covered = [b for c in range(nch) for b in range(c * per, min(c * per + per, B))]
    assert covered == list(range(B))
    assert all(c * per < B for c in range(nch)), "no empty chunk"
    if split[1] + split[2] == 15:
        assert per == 1


def test_middle_renumbering_is_a_permutation():
    for nblk in (8, 16, 24, 4096, 3 * 8):
        seen = sorted((blk & 7) * (nblk >> 3) + (blk >> 3) for blk in range(nblk))
        assert seen == list(range(nblk))


def test_middle_groups_share_a_gain_on_one_xcd():
    """Blocks are dealt round-robin over the 8 XCDs.  With slice groups the
    middle blocks of one run (one per group) are 2^(A-R) apart, a multiple
    of 8 for every automatic split, so they read the run's gain through one
    L2; with one slice per block the renumbering puts a run's B blocks on
    one XCD when B divides the per-XCD share."""
    for K in range(16, 31):
        A, HB, R = three_pass_split(K)
        assert (1 << (A - R)) % 8 == 0, K
        for B in (1, 2, 4, 32):
            nblk = B << (A - R)
            xcd = {}
            for blk in range(nblk):
                logical = (blk & 7) * (nblk >> 3) + (blk >> 3)
                xcd.setdefault(logical // B, set()).add(blk % 8)
            assert all(len(v) == 1 for v in xcd.values()), (K, B)


def outer_block(blk, nblk, R):
    if R >= 5:
        return blk
    g = 1 << (5 - R)
    if nblk % (8 * g):
        return blk
    return (blk & ~(8 * g - 1)) | ((blk & 7) * g) | ((blk >> 3) & (g - 1))


@pytest.mark.parametrize("R", [0, 1, 2, 3, 4, 5, 6])
def test_outer_renumbering(R):
    """A permutation of the outer grid; with R < 5 the 2^(5-R) blocks that
    share a 128-byte workspace line sit on one XCD (same block index mod 8)."""
    for nblk in (2048, 4096, 8 * (1 << max(0, 5 - R)) * 3, 24, 7):
        m = [outer_block(b, nblk, R) for b in range(nblk)]
        assert sorted(m) == list(range(nblk))
        if R < 5 and nblk % (8 << (5 - R)) == 0:
            g = 1 << (5 - R)
            inv = {v: b for b, v in enumerate(m)}
            for hi0 in range(0, nblk, g):
                assert len({inv[hi0 + j] % 8 for j in range(g)}) == 1
