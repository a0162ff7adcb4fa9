"""CPU model of the fused block kernels' index arithmetic (no GPU).

The block with its projections (section III-B, eqs. (1)-(4)) runs its MFMA
prologue and epilogue inside the mixer's kernels.  This file re-derives, in
numpy, every index the HIP code computes -- the weight repacking, the lane
layout of the 16x16 matrix-core operands and results, the layout-4 fragments
of the prologue, the exchange schedules through LDS and the epilogue layout,
stores and masks -- and checks that the composition reproduces the oracle's
block on small tiles.  A wrong index here would be a wrong or out-of-bounds
access on the GPU, so these run before any GPU parity test.

The matrix-core lane layouts used (v_mfma_f32_16x16x16_bf16 and
v_mfma_f32_16x16x4_f32) are the documented CDNA ones: lane l supplies row
l%16 of A and column l%16 of B with k = 4*(l//16) + r (bf16, element r) or
k = l//16 (fp32), and receives D[4*(l//16) + r][l%16] in element r.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle.oracle import Oracle
from paper_2607_25234_amd.workloads import round_to_bf16

VB = 5


def pad(t):
    return t + (t >> 5)


# ------------------------------------------------------------------ matrix core
def mfma_bf16(a, b, acc):
    """a, b: [64, 4] lane operands; acc: [64, 4].  16x16x16."""
    A = np.zeros((16, 16))
    B = np.zeros((16, 16))
    for lane in range(64):
        for r in range(4):
            A[lane % 16, 4 * (lane // 16) + r] = a[lane, r]
            B[4 * (lane // 16) + r, lane % 16] = b[lane, r]
    D = A @ B
    out = acc.copy()
    for lane in range(64):
        for r in range(4):
            out[lane, r] += D[4 * (lane // 16) + r, lane % 16]
    return out


def mfma_f32(a, b, acc):
    """a, b: [64] lane operands; acc: [64, 4].  16x16x4."""
    A = np.zeros((16, 4))
    B = np.zeros((4, 16))
    for lane in range(64):
        A[lane % 16, lane // 16] = a[lane]
        B[lane // 16, lane % 16] = b[lane]
    D = A @ B
    out = acc.copy()
    for lane in range(64):
        for r in range(4):
            out[lane, r] += D[4 * (lane // 16) + r, lane % 16]
    return out


# ------------------------------------------------------------------ packing
def k_in_bf16(C, kk, q, r):
    return 32 * (kk >> 1) + 8 * q + 4 * (kk & 1) + r if C >= 32 else 4 * q + r


def k_in_f32(s, q):
    return 16 * (s >> 2) + 4 * q + (s & 3)


def oc_bf16(C, nb, m):
    return 32 * (nb >> 1) + 8 * (m >> 2) + 4 * (nb & 1) + (m & 3) if C >= 32 else m


def pack(w_in, w_out, bf):
    C = w_in.shape[0]
    p_in = np.empty(C * C)
    p_out = np.empty(C * C)
    src_in = np.full(C * C, -1)
    src_out = np.full(C * C, -1)
    for idx in range(C * C):
        e, lane, rest = idx & 3, (idx >> 2) & 63, idx >> 8
        j, q = lane & 15, lane >> 4
        if bf:
            ks = C // 16
            kk, nb = rest % ks, rest // ks
            si = k_in_bf16(C, kk, q, e) * C + 16 * nb + j
            so = (q * (C // 4) + 4 * kk + e) * C + oc_bf16(C, nb, j)
        else:
            npc = C // 16
            p, nb = rest % npc, rest // npc
            s = 4 * p + e
            si = k_in_f32(s, q) * C + 16 * nb + j
            so = (q * (C // 4) + s) * C + 16 * nb + j
        assert 0 <= si < C * C and 0 <= so < C * C
        src_in[idx], src_out[idx] = si, so
        p_in[idx] = w_in.reshape(-1)[si]
        p_out[idx] = w_out.reshape(-1)[so]
    # each packed array is a permutation of the weights
    assert sorted(src_in) == list(range(C * C))
    assert sorted(src_out) == list(range(C * C))
    return p_in, p_out


def mfma_bf16_x32(a, b, acc):
    """16x16x32 (gfx950): a, b [64, 8]; lane 16 g + i supplies row i of A
    (column i of B) with k = 8 g + e; the result layout is the 16x16x16 one."""
    A = a.reshape(4, 16, 8).transpose(1, 0, 2).reshape(16, 32)
    B = b.reshape(4, 16, 8).transpose(0, 2, 1).reshape(32, 16)
    D = A @ B
    return acc + D.reshape(4, 4, 16).transpose(0, 2, 1).reshape(64, 4)


def pack_x32(w_in, w_out):
    """bf16, C >= 32: operands of the 16x16x32 instruction.  Packed index
    ((nb * C/32 + kk) * 64 + 16 g + j) * 8 + e holds W_in[32 kk + 8 g + e][16 nb + j]
    and W_out[(C/4) g + 8 kk + e][oc_bf16(nb, j)]."""
    C = w_in.shape[0]
    idx = np.arange(C * C)
    e, lane, rest = idx & 7, (idx >> 3) & 63, idx >> 9
    j, g = lane & 15, lane >> 4
    kk, nb = rest % (C // 32), rest // (C // 32)
    si = (32 * kk + 8 * g + e) * C + 16 * nb + j
    so = ((C // 4) * g + 8 * kk + e) * C + np.array([oc_bf16(C, int(n), int(m))
                                                      for n, m in zip(nb, j)])
    assert sorted(si) == list(range(C * C)) and sorted(so) == list(range(C * C))
    return w_in.reshape(-1)[si], w_out.reshape(-1)[so]


def x32(C, bf):
    """The fused kernels' bf16 products take the 16x16x32 instruction from C = 32."""
    return bf and C >= 32


def pack_fused(w_in, w_out, bf):
    """Packed weights of the fused kernels."""
    return pack_x32(w_in, w_out) if x32(w_in.shape[0], bf) else pack(w_in, w_out, bf)


# ------------------------------------------------------------------ layouts
class Std:
    def __init__(self, S):
        self.S = S

    def reg(self, j):
        return self.S + j

    def base(self, tau):
        S = self.S
        return (tau & ((1 << S) - 1)) | ((tau >> S) << (S + VB))


class Epi:
    def __init__(self, M, CB):
        self.M, self.CB = M, CB

    def reg(self, j):
        CB, M = self.CB, self.M
        return j if j < CB - 2 else M - 7 + CB + (j - (CB - 2))

    def base(self, tau):
        CB = self.CB
        return ((tau & 15) << CB) | (((tau >> 4) & 3) << (CB - 2)) | ((tau >> 6) << (CB + 4))


def reg_offset(L, k):
    t = 0
    for j in range(VB):
        if k & (1 << j):
            t |= 1 << L.reg(j)
    return t


def flat_index(L, M):
    """[NT, 32] tile index of every (thread, register) of layout L."""
    NT = 1 << (M - VB)
    tau = np.arange(NT)
    t = np.array([[L.base(int(u)) | reg_offset(L, k) for k in range(32)] for u in tau])
    assert sorted(t.reshape(-1)) == list(range(1 << M)), "layout is not a bijection"
    return t


class Tracker:
    """Runs register butterflies and LDS exchanges on a [NT, 32] register
    file, records which tile bits each butterfly step transforms, checks LDS
    bounds and measures bank conflicts of every LDS access."""

    def __init__(self, M, v, layout):
        self.M = M
        self.v = v
        self.layout = layout
        self.done = []
        self.conflicts = []

    def butterflies(self, mask):
        for j in range(VB):
            if not mask & (1 << j):
                continue
            self.done.append(self.layout.reg(j))
            for k in range(32):
                if not k & (1 << j):
                    a = self.v[:, k].copy()
                    b = self.v[:, k | (1 << j)].copy()
                    self.v[:, k] = a + b
                    self.v[:, k | (1 << j)] = a - b

    def _addresses(self, L):
        NT = 1 << (self.M - VB)
        return np.array([[pad(L.base(u)) + pad(reg_offset(L, k)) for k in range(32)]
                         for u in range(NT)])

    def _conflict(self, addr):
        worst = 1
        NT = addr.shape[0]
        for w in range(0, NT, 64):
            for k in range(32):
                banks = addr[w:w + 64, k] % 64
                worst = max(worst, np.bincount(banks, minlength=64).max())
        return worst

    def relayout(self, LB):
        size = pad(1 << self.M)
        lds = np.full(size, np.nan)
        wa = self._addresses(self.layout)
        assert wa.max() < size and wa.min() >= 0
        assert len(np.unique(wa)) == wa.size, "two registers write one LDS word"
        lds[wa] = self.v
        ra = self._addresses(LB)
        assert ra.max() < size
        self.v = lds[ra]
        assert not np.isnan(self.v).any(), "read of an LDS word nobody wrote"
        self.conflicts.append((self._conflict(wa), self._conflict(ra)))
        self.layout = LB


class Low4Hi9:
    """2^15 tiles: registers hold t bits 0-3 and 9; threads bits 4-8, 10-14."""

    def reg(self, j):
        return j if j < 4 else 9

    def base(self, tau):
        return ((tau & 31) << 4) | ((tau >> 5) << 10)


def forward_from_prologue(tr, M):
    tr.butterflies(31)
    if M <= 14:
        tr.relayout(Std(0))
        tr.butterflies(15)
        tr.relayout(Std(M - 5))
        tr.butterflies(31 & ~((1 << (14 - M)) - 1))
    else:
        tr.relayout(Low4Hi9())
        tr.butterflies(31)
        tr.relayout(Std(10))
        tr.butterflies(31)


def inverse_to_epilogue(tr, M, CB):
    ln = M - 3 - CB
    tr.butterflies((1 << (CB - 2)) - 1)
    if ln <= VB:
        tr.relayout(Std(CB - 2))
        tr.butterflies((1 << ln) - 1)
    else:
        tr.relayout(Std(CB - 2))
        tr.butterflies(31)
        tr.relayout(Std(CB + 3))
        tr.butterflies((1 << (ln - VB)) - 1)
    tr.relayout(Epi(M, CB))
    tr.butterflies(31)


def to_registers(flat, L, M):
    return flat[flat_index(L, M)]


def from_registers(v, L, M):
    out = np.empty(1 << M)
    out[flat_index(L, M)] = v
    return out


def wht_bits(flat, M):
    """Unnormalised Sylvester transform over all M bits."""
    y = flat.copy()
    h = 1
    while h < (1 << M):
        y = y.reshape(-1, 2, h)
        y = np.stack([y[:, 0] + y[:, 1], y[:, 0] - y[:, 1]], axis=1).reshape(-1)
        h *= 2
    return y


# ------------------------------------------------------------------ prologue
def prologue_token(CB, rb, m, w):
    return (m & 3) | (rb << 2) | ((m >> 2) << (9 - CB)) | (w << (11 - CB))


def model_prologue(xtile, valid, p_in, CB, M, bf):
    """Registers [NT, 32] of layout 4 holding Z = X W_in of the tile."""
    C = 1 << CB
    NT = 1 << (M - VB)
    NRB = 1 << (7 - CB)
    NNB = C // 16
    flat = xtile.reshape(-1)
    v = np.zeros((NT, 32))
    for w in range(NT // 64):
        lanes = np.arange(64)
        i, q = lanes & 15, lanes >> 4

        def row_of(rb):
            tok = prologue_token(CB, rb, i, w)
            rows = np.zeros((64, C))
            ok = tok * C < valid
            rows[ok] = flat.reshape(-1, C)[tok[ok]]
            return rows

        rows = [row_of(rb) for rb in range(NRB)]
        for nb in range(NNB):
            for rb in range(NRB):
                acc = np.zeros((64, 4))
                if x32(C, bf):       # step kk: channels 32 kk + 8 q + [0, 8)
                    for kk in range(C // 32):
                        cols = 32 * kk + 8 * q[:, None] + np.arange(8)[None, :]
                        a = rows[rb][lanes[:, None], cols]
                        idx = ((nb * (C // 32) + kk) * 64 + lanes[:, None]) * 8 + \
                            np.arange(8)[None, :]
                        acc = mfma_bf16_x32(a, p_in[idx], acc)
                elif bf:
                    for kk in range(C // 16):
                        a = np.array([[rows[rb][l, k_in_bf16(C, kk, q[l], r)] for r in range(4)]
                                      for l in range(64)])
                        b = np.array([[p_in[((nb * (C // 16) + kk) * 64 + l) * 4 + r]
                                       for r in range(4)] for l in range(64)])
                        acc = mfma_bf16(a, b, acc)
                else:
                    for p in range(C // 16):
                        bvec = np.array([[p_in[((nb * (C // 16) + p) * 64 + l) * 4 + e]
                                          for e in range(4)] for l in range(64)])
                        for e in range(4):
                            s = 4 * p + e
                            a = np.array([rows[rb][l, k_in_f32(s, q[l])] for l in range(64)])
                            acc = mfma_f32(a, bvec[:, e], acc)
                for r in range(4):
                    v[w * 64:(w + 1) * 64, nb | (r << (CB - 4)) | (rb << (CB - 2))] = acc[:, r]
    return v


# ------------------------------------------------------------------ epilogue
def split_bf16(z):
    hi = round_to_bf16(np.asarray(z, dtype=np.float32).copy()).astype(np.float64)
    lo = round_to_bf16(np.asarray(z - hi, dtype=np.float32).copy()).astype(np.float64)
    return hi, lo


def model_epilogue(v, p_out, CB, M, valid, bf):
    """Stores of Y = Z' W_out from epilogue-layout registers; returns the
    tile's output (NaN where nothing was stored) and the byte offsets used."""
    C = 1 << CB
    NT = 1 << (M - VB)
    NRB = 1 << (7 - CB)
    NNB = C // 16
    esz = 2 if bf else 4
    out = np.full((1 << M), np.nan)
    written = np.zeros(1 << M, dtype=int)
    rb_bytes = (1 << (M - 7)) * C * esz
    for w in range(NT // 64):
        lanes = np.arange(64)
        j, q = lanes & 15, lanes >> 4
        row = (j | (w << 4)) * C * esz
        vw = v[w * 64:(w + 1) * 64]
        for rb in range(NRB):
            accs = []
            for nb in range(NNB):
                acc = np.zeros((64, 4))
                if x32(C, bf):       # step kk: channels q C/4 + 8 kk + [0, 8)
                    for kk in range(C // 32):
                        z = np.stack([vw[:, (8 * kk + e) | (rb << (CB - 2))] for e in range(8)],
                                     axis=1)
                        hi, lo = split_bf16(z)
                        idx = ((nb * (C // 32) + kk) * 64 + lanes[:, None]) * 8 + \
                            np.arange(8)[None, :]
                        a = p_out[idx]
                        acc = mfma_bf16_x32(a, hi, acc)
                        acc = mfma_bf16_x32(a, lo, acc)
                elif bf:
                    for kk in range(C // 16):
                        z = np.stack([vw[:, (4 * kk + e) | (rb << (CB - 2))] for e in range(4)],
                                     axis=1)
                        hi, lo = split_bf16(z)
                        a = np.array([[p_out[((nb * (C // 16) + kk) * 64 + l) * 4 + r]
                                       for r in range(4)] for l in range(64)])
                        acc = mfma_bf16(a, hi, acc)
                        acc = mfma_bf16(a, lo, acc)
                else:
                    for p in range(C // 16):
                        avec = np.array([[p_out[((nb * (C // 16) + p) * 64 + l) * 4 + e]
                                          for e in range(4)] for l in range(64)])
                        for e in range(4):
                            s = 4 * p + e
                            acc = mfma_f32(avec[:, e], vw[:, s | (rb << (CB - 2))], acc)
                accs.append(acc)

            def store(byte_off, vals):
                for l in range(64):
                    for u, val in enumerate(vals[l]):
                        off = byte_off[l] + u * esz
                        assert off % esz == 0
                        t = off // esz
                        if off + esz <= valid * esz:     # buffer range check
                            out[t] = val
                            written[t] += 1

            if bf and C >= 32:
                for n in range(NNB // 2):
                    vals = np.concatenate([accs[2 * n], accs[2 * n + 1]], axis=1)
                    store(row + 16 * q + rb * rb_bytes + 64 * n, vals)
            elif bf:
                store(row + 8 * q + rb * rb_bytes, accs[0])
            else:
                for nb in range(NNB):
                    store(row + 16 * q + rb * rb_bytes + 64 * nb, accs[nb])
    assert written.max() <= 1, "an element stored twice"
    assert (written[:valid] == 1).all(), "an element of the tile not stored"
    return out


# ------------------------------------------------------------------ tests
CASES = [(cb, M, bf) for bf in (True, False) for cb in (4, 5, 6, 7) for M in (11, 12, 13, 14, 15)]


def _weights(rng, C):
    return rng.standard_normal((C, C)) / np.sqrt(C), rng.standard_normal((C, C)) / np.sqrt(C)


@pytest.mark.parametrize("CB,bf", [(cb, bf) for bf in (True, False) for cb in (4, 5, 6, 7)])
def test_packing_is_a_permutation(CB, bf):
    rng = np.random.default_rng(CB)
    w_in, w_out = _weights(rng, 1 << CB)
    pack(w_in, w_out, bf)
    pack_fused(w_in, w_out, bf)


@pytest.mark.parametrize("CB,M,bf", [c for c in CASES if c[1] in (11, 14)])
def test_prologue_fragments_are_layout_4(CB, M, bf):
    """The MFMA result registers, read as layout 4, are Z = X W_in."""
    rng = np.random.default_rng(100 * CB + M)
    C = 1 << CB
    w_in, w_out = _weights(rng, C)
    p_in, _ = pack_fused(w_in, w_out, bf)
    rows = (1 << M) // C
    x = rng.standard_normal((rows, C))
    valid = (rows - 3) * C          # a ragged tile: the last 3 rows are padding
    v = model_prologue(x, valid, p_in, CB, M, bf)
    z = from_registers(v, Std(4), M).reshape(rows, C)
    ref = x.copy()
    ref[valid // C:] = 0.0
    ref = ref @ w_in
    np.testing.assert_allclose(z, ref, atol=1e-12)


@pytest.mark.parametrize("CB,M", [(cb, M) for cb in (4, 5, 6, 7) for M in (11, 12, 13, 14, 15)])
def test_schedules_cover_every_bit_once(CB, M):
    """Prologue schedule + epilogue schedule: every tile bit is transformed
    exactly once in each direction, every exchange is an in-bounds bijection
    through LDS, and the result equals the full transform."""
    rng = np.random.default_rng(7 * M + CB)
    flat = rng.standard_normal(1 << M)
    tr = Tracker(M, to_registers(flat, Std(4), M), Std(4))
    forward_from_prologue(tr, M)
    assert sorted(tr.done) == list(range(M))
    assert isinstance(tr.layout, Std) and tr.layout.S == M - 5
    np.testing.assert_allclose(from_registers(tr.v, tr.layout, M), wht_bits(flat, M), atol=1e-9)
    tr2 = Tracker(M, to_registers(flat, Std(M - 5), M), Std(M - 5))
    inverse_to_epilogue(tr2, M, CB)
    assert sorted(tr2.done) == list(range(M))
    np.testing.assert_allclose(from_registers(tr2.v, Epi(M, CB), M), wht_bits(flat, M),
                               atol=1e-9)
    # standard layouts stay conflict-free; the epilogue layout at most 2-way
    for (wr, rd), L in zip(tr.conflicts + tr2.conflicts, [None] * 99):
        assert wr <= 2 and rd <= 2


@pytest.mark.parametrize("CB,M,bf", [c for c in CASES if c[1] in (11, 13, 15)])
def test_epilogue_stores_y(CB, M, bf):
    """Epilogue-layout registers of Z' give Y = Z' W_out, each valid element
    stored once, nothing stored past the valid rows."""
    rng = np.random.default_rng(31 * CB + M)
    C = 1 << CB
    w_in, w_out = _weights(rng, C)
    _, p_out = pack_fused(w_in, w_out, bf)
    rows = (1 << M) // C
    z = rng.standard_normal((rows, C))
    valid = (rows - 5) * C
    v = to_registers(z.reshape(-1), Epi(M, CB), M)
    y = model_epilogue(v, p_out, CB, M, valid, bf)
    assert np.isnan(y[valid:]).all()
    ref = (z @ w_out).reshape(-1)[:valid]
    tol = 1e-5 if bf else 1e-12      # the two-term bf16 split of Z'
    np.testing.assert_allclose(y[:valid], ref, atol=tol * np.abs(ref).max())


def _block_tile_model(x, w_in, g, w_out, CB, bf):
    """One slice through the FUSED kernel's steps (M = K)."""
    C = 1 << CB
    N = x.shape[0]
    P = 1 << (N - 1).bit_length()
    M = (P * C).bit_length() - 1
    p_in, p_out = pack_fused(w_in, w_out, bf)
    xt = np.zeros((P, C))
    xt[:N] = x
    v = model_prologue(xt, N * C, p_in, CB, M, bf)
    tr = Tracker(M, v, Std(4))
    forward_from_prologue(tr, M)
    gv = to_registers(g.reshape(-1), Std(M - 5), M)
    tr.v = tr.v * gv / (1 << M)
    inverse_to_epilogue(tr, M, CB)
    y = model_epilogue(tr.v, p_out, CB, M, N * C, bf)
    return y[:N * C].reshape(N, C)


@pytest.fixture(scope="module")
def oracle():
    return Oracle()


@pytest.mark.parametrize("N,CB,bf", [(32, 6, True), (100, 5, False), (16, 7, False),
                                     (200, 4, True)])
def test_fused_model_matches_oracle(oracle, N, CB, bf):
    rng = np.random.default_rng(N + CB)
    C = 1 << CB
    P = 1 << (N - 1).bit_length()
    x = rng.standard_normal((N, C))
    w_in, w_out = _weights(rng, C)
    if bf:
        x = round_to_bf16(x.astype(np.float32)).astype(np.float64)
        w_in = round_to_bf16(w_in.astype(np.float32)).astype(np.float64)
        w_out = round_to_bf16(w_out.astype(np.float32)).astype(np.float64)
    g = rng.uniform(0.5, 1.5, (P, C))
    y = _block_tile_model(x, w_in, g, w_out, CB, bf)
    ref = oracle.whtmix_module(x, w_in, g, w_out)
    tol = 1e-5 if bf else 1e-12
    np.testing.assert_allclose(y, ref, atol=tol * np.abs(ref).max())


# ------------------------------------------------------------------ C = 256: 2^16 pair tiles
# A bf16 block with C = 256 runs its outer passes on tiles of 256 tokens x 256
# channels (t = token * 256 + channel), 1024 threads of two register sets of
# 32.  Forward: set = t bit 15 (token bit 7), each set in layout 4 of its 2^15
# elements straight from the MFMA results.  Inverse: set = t bit 5 (channel bit
# 5); within a set t' drops that bit and the set's elements are laid out like
# a C = 128 tile, so the epilogue layout is Epi(15, 7).
PC, PCB, PM = 256, 8, 15


def mfma_bf16_fast(a, b, acc):
    """mfma_bf16 with array reshapes (same lane layout)."""
    A = a.reshape(4, 16, 4).transpose(1, 0, 2).reshape(16, 16)
    B = b.reshape(4, 16, 4).transpose(0, 2, 1).reshape(16, 16)
    D = A @ B
    return acc + D.reshape(4, 4, 16).transpose(0, 2, 1).reshape(64, 4)


def pair_token(m, w):
    """Token of MFMA row m = 4q + r in wave w: r0 -> token bit 0, q -> bits
    1-2, the wave -> bits 3-6, r1 -> bit 7 (the register set)."""
    return (m & 1) | (((m >> 2) & 3) << 1) | (w << 3) | (((m >> 1) & 1) << 7)


def model_prologue_pair(xtile, valid, p_in):
    """[2, 1024, 32] registers of Z = X W_in: set s, register nb | r0 << 4.
    Step kk of lane group q is one 16-byte load: channels 32 kk + 8 q + [0, 8)."""
    v = np.zeros((2, 1024, 32))
    lanes = np.arange(64)
    i, q = lanes & 15, lanes >> 4
    ks = PC // 32
    for w in range(16):
        tok = pair_token(i, w)
        rows = np.zeros((64, PC))
        ok = tok * PC < valid
        rows[ok] = xtile[tok[ok]]
        for nb in range(16):
            acc = np.zeros((64, 4))
            for kk in range(ks):
                cols = 32 * kk + 8 * q[:, None] + np.arange(8)[None, :]
                a = rows[lanes[:, None], cols]
                idx = ((nb * ks + kk) * 64 + lanes[:, None]) * 8 + np.arange(8)[None, :]
                acc = mfma_bf16_x32(a, p_in[idx], acc)
            for r in range(4):
                v[r >> 1, w * 64:(w + 1) * 64, nb | ((r & 1) << 4)] = acc[:, r]
    return v


def cross(v0, v1):
    return v0 + v1, v0 - v1


def expand5(tp):
    """Set-local index t' -> tile index with bit 5 clear."""
    return (tp & 31) | ((tp >> 5) << 6)


def model_epilogue_pair(v0, v1, p_out, valid):
    """Y = Z' W_out from the two sets' Epi(15, 7) registers; lane (j, q) of
    wave w holds channels 64 q + 32 s + k' of token j | w << 4."""
    out = np.full(1 << 16, np.nan)
    written = np.zeros(1 << 16, dtype=int)
    lanes = np.arange(64)
    j, q = lanes & 15, lanes >> 4
    ks = PC // 32
    for w in range(16):
        vw = np.concatenate([v0[w * 64:(w + 1) * 64], v1[w * 64:(w + 1) * 64]], axis=1)
        row = (j | (w << 4)) * PC * 2
        accs = []
        for nb in range(16):
            acc = np.zeros((64, 4))
            for kk in range(ks):     # channels 64 q + 8 kk + [0, 8)
                hi, lo = split_bf16(vw[:, 8 * kk:8 * kk + 8])
                idx = ((nb * ks + kk) * 64 + lanes[:, None]) * 8 + np.arange(8)[None, :]
                a = p_out[idx]
                acc = mfma_bf16_x32(a, hi, acc)
                acc = mfma_bf16_x32(a, lo, acc)
            accs.append(acc)
        for n in range(8):
            vals = np.concatenate([accs[2 * n], accs[2 * n + 1]], axis=1)
            off = row + 16 * q + 64 * n
            for l in range(64):
                for u in range(8):
                    t = (off[l] + 2 * u) // 2
                    if 2 * t + 2 <= valid * 2:
                        out[t] = vals[l, u]
                        written[t] += 1
    assert written.max() <= 1, "an element stored twice"
    assert (written[:valid] == 1).all(), "an element of the tile not stored"
    return out


def test_fast_mfma_model_is_the_lane_model():
    rng = np.random.default_rng(3)
    a, b, c = rng.standard_normal((64, 4)), rng.standard_normal((64, 4)), rng.standard_normal((64, 4))
    np.testing.assert_allclose(mfma_bf16_fast(a, b, c), mfma_bf16(a, b, c), atol=1e-12)
    # the 16x16x32 form is two 16x16x16 products over k = 8 g + [0, 4) and 8 g + [4, 8)
    a8, b8 = rng.standard_normal((64, 8)), rng.standard_normal((64, 8))
    two = mfma_bf16(a8[:, 4:], b8[:, 4:], mfma_bf16(a8[:, :4], b8[:, :4], c))
    np.testing.assert_allclose(mfma_bf16_x32(a8, b8, c), two, atol=1e-12)


def test_pair_prologue_fragments_are_layout_4():
    """C = 256: the MFMA results of each set, read as layout 4 of that set's
    2^15 elements, are Z = X W_in (ragged tile: the last 37 tokens padding)."""
    rng = np.random.default_rng(256)
    w_in, w_out = _weights(rng, PC)
    w_in = round_to_bf16(w_in.astype(np.float32)).astype(np.float64)
    p_in, _ = pack_x32(w_in, w_out)
    x = round_to_bf16(rng.standard_normal((256, PC)).astype(np.float32)).astype(np.float64)
    valid = (256 - 37) * PC
    v = model_prologue_pair(x, valid, p_in)
    ref = x.copy()
    ref[valid // PC:] = 0.0
    ref = (ref @ w_in).reshape(-1)
    for s in range(2):
        z = from_registers(v[s], Std(4), PM)
        np.testing.assert_allclose(z, ref[s << PM:(s + 1) << PM], atol=1e-12)


def test_pair_schedules_cover_every_bit_once():
    """Forward: cross butterfly (bit 15), then each set from layout 4 to the
    store layout 10; inverse: each set (t bit 5) from layout 10 to the
    epilogue layout, then the cross butterfly.  Both give the transform over
    all 16 bits; every exchange stays in bounds, at most 2-way bank
    conflicts."""
    rng = np.random.default_rng(16)
    flat = rng.standard_normal(1 << 16)
    full = wht_bits(flat, 16)
    v = [to_registers(flat[s << PM:(s + 1) << PM], Std(4), PM) for s in range(2)]
    v0, v1 = cross(v[0], v[1])
    trs = [Tracker(PM, v0, Std(4)), Tracker(PM, v1, Std(4))]
    for tr in trs:
        forward_from_prologue(tr, PM)
        assert sorted(tr.done) == list(range(PM))
        assert isinstance(tr.layout, Std) and tr.layout.S == 10
        assert all(wr <= 2 and rd <= 2 for wr, rd in tr.conflicts)
    for s in range(2):
        np.testing.assert_allclose(from_registers(trs[s].v, Std(10), PM),
                                   full[s << PM:(s + 1) << PM], atol=1e-9)
    tp = np.arange(1 << PM)
    sets = [flat[expand5(tp) | (s << 5)] for s in range(2)]
    trs = [Tracker(PM, to_registers(sets[s], Std(10), PM), Std(10)) for s in range(2)]
    for tr in trs:
        inverse_to_epilogue(tr, PM, 7)
        assert sorted(tr.done) == list(range(PM))
        assert all(wr <= 2 and rd <= 2 for wr, rd in tr.conflicts)
    e0, e1 = cross(trs[0].v, trs[1].v)
    for s, e in enumerate((e0, e1)):
        np.testing.assert_allclose(from_registers(e, Epi(PM, 7), PM),
                                   full[expand5(tp) | (s << 5)], atol=1e-9)


def test_pair_epilogue_stores_y():
    """Epilogue registers of Z' (both sets) give Y = Z' W_out; each valid
    element stored once, nothing past the valid rows."""
    rng = np.random.default_rng(257)
    w_in, w_out = _weights(rng, PC)
    w_out = round_to_bf16(w_out.astype(np.float32)).astype(np.float64)
    _, p_out = pack_x32(w_in, w_out)
    z = rng.standard_normal((256, PC))
    valid = (256 - 11) * PC
    flat = z.reshape(-1)
    tp = np.arange(1 << PM)
    v = [to_registers(flat[expand5(tp) | (s << 5)], Epi(PM, 7), PM) for s in range(2)]
    y = model_epilogue_pair(v[0], v[1], p_out, valid)
    assert np.isnan(y[valid:]).all()
    ref = (z @ w_out).reshape(-1)[:valid]
    np.testing.assert_allclose(y[:valid], ref, atol=1e-5 * np.abs(ref).max())


# ------------------------------------------------------------------ UNFUSED MFMA projection
def model_project(inp, w, bf_w, in_bf, CB):
    """project_mfma_kernel: column slices of NCOL, 64-row blocks, 16 rows per
    wave, weights in the prologue's packed order."""
    C = 1 << CB
    s = 2 if bf_w else 4
    NCOL = min(min(C, 128), max(16, 65536 // (C * s)))
    NB = NCOL // 16
    KS = C // 16 if bf_w else C // 4
    packed, _ = pack(w, w, bf_w)
    rows = inp.shape[0]
    out = np.full((rows, C), np.nan)
    lanes = np.arange(64)
    i, q = lanes & 15, lanes >> 4
    for sl in range(C // NCOL):
        wsl = packed[sl * NCOL * C:(sl + 1) * NCOL * C]
        for blk in range((rows + 63) // 64):
            for wv in range(4):
                r0 = blk * 64 + wv * 16
                ok = r0 + i < rows
                A = np.zeros((64, C))
                A[ok] = inp[(r0 + i)[ok]]
                acc = [np.zeros((64, 4)) for _ in range(NB)]

                def wfrag(idx0):
                    return np.array([[wsl[(idx0 * 64 + l) * 4 + r] for r in range(4)]
                                     for l in range(64)])
                if bf_w:
                    for p in range(C // 32):
                        cols = 32 * p + 8 * q[:, None] + np.arange(8)[None, :]
                        piece = A[lanes[:, None], cols]
                        parts = [piece[:, :4], piece[:, 4:]]
                        for nb in range(NB):
                            for h in range(2):
                                b = wfrag(nb * KS + 2 * p + h)
                                if in_bf:
                                    acc[nb] = mfma_bf16(parts[h], b, acc[nb])
                                else:
                                    hi, lo = split_bf16(parts[h])
                                    acc[nb] = mfma_bf16(hi, b, acc[nb])
                                    acc[nb] = mfma_bf16(lo, b, acc[nb])
                else:
                    for p in range(C // 16):
                        cols = 16 * p + 4 * q[:, None] + np.arange(4)[None, :]
                        a = A[lanes[:, None], cols]
                        for nb in range(NB):
                            b = wfrag(nb * (C // 16) + p)
                            for e in range(4):
                                acc[nb] = mfma_f32(a[:, e], b[:, e], acc[nb])
                for r in range(4):
                    row = r0 + 4 * q + r
                    for nb in range(NB):
                        m = row < rows
                        out[row[m], (sl * NCOL + i + 16 * nb)[m]] = acc[nb][m, r]
    return out


@pytest.mark.parametrize("CB,bf_w,in_bf", [(8, True, True), (8, True, False), (8, False, False),
                                           (9, True, True), (9, False, False), (5, True, True),
                                           (5, True, False), (6, False, False), (7, True, False),
                                           (7, True, True)])
def test_unfused_projection_model(CB, bf_w, in_bf):
    rng = np.random.default_rng(CB * 10 + bf_w + 2 * in_bf)
    C = 1 << CB
    rows = 83                    # a ragged last block
    x = rng.standard_normal((rows, C))
    w = rng.standard_normal((C, C)) / np.sqrt(C)
    if bf_w:
        w = round_to_bf16(w.astype(np.float32)).astype(np.float64)
    if in_bf:
        x = round_to_bf16(x.astype(np.float32)).astype(np.float64)
    else:
        x = x.astype(np.float32).astype(np.float64)
    y = model_project(x, w, bf_w, in_bf, CB)
    assert not np.isnan(y).any(), "an output element never stored"
    ref = x @ w
    tol = 1e-5 if (bf_w and not in_bf) else 1e-12
    np.testing.assert_allclose(y, ref, atol=tol * np.abs(ref).max())


def test_transposed_packing_is_the_packing_of_the_transpose():
    """pack_b_kernel with trans reads W[col][k]: the packing of W^T."""
    rng = np.random.default_rng(5)
    for C in (32, 128):
        w = rng.standard_normal((C, C))
        for bf in (True, False):
            a, _ = pack(w.T.copy(), w, bf)
            # the kernel's transposed read, written out independently
            b = np.empty(C * C)
            for idx in range(C * C):
                e, lane, rest = idx & 3, (idx >> 2) & 63, idx >> 8
                j, q = lane & 15, lane >> 4
                if bf:
                    ks = C // 16
                    k, col = k_in_bf16(C, rest % ks, q, e), 16 * (rest // ks) + j
                else:
                    npc = C // 16
                    k, col = k_in_f32(4 * (rest % npc) + e, q), 16 * (rest // npc) + j
                b[idx] = w[col, k]
            assert np.array_equal(a, b)


def wgrad_plan(rows, cb):
    """csrc/whtmix_module.h wgrad_plan."""
    if rows == 0:
        return 0, 4
    C = 1 << cb
    T = min(C, 128)
    blocks = (C // T) ** 2 if C >= 16 else 1
    chunks = max(1, 512 // blocks)
    chunks = min(chunks, (rows + 63) // 64)
    rpc = -(-rows // chunks)
    rpc = max(4, (rpc + 3) // 4 * 4)
    return -(-rows // rpc), rpc


def bf16_rne(v):
    """Round float32 values to bf16 (round to nearest even), as float32."""
    u = np.asarray(v, np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32)


def model_wgrad(a, b, cb, kinds=("f32", "f32")):
    """wgrad_mfma_kernel: per (chunk, T x T block), LDS blocks of RB rows (32
    for float32 x float32 at T = 128, else 64), waves
    owning TQ x TQ quadrants of 16 x 16 tiles; in a step the lanes (i, q)
    take, for k-slot e, row kb + q + 4e (16x16x32 bf16 instruction, 32 rows)
    or row kb + q (float32 instruction, 4 rows) of column i.  kinds: the dtypes of
    a and b; a float against a bf16 operand is split into three bf16 terms."""
    if kinds == ("f32", "bf16"):   # run as (b, a), the sum transposed at the end
        return model_wgrad(b, a, cb, ("bf16", "f32")).T
    rows, C = a.shape
    chunks, rpc = wgrad_plan(rows, cb)
    T = min(C, 128)
    TQ = T // 32 if T >= 32 else 1
    f32 = kinds == ("f32", "f32")
    RB = 32 if f32 and T == 128 else 64
    part = np.full((chunks, C, C), np.nan)
    lanes = np.arange(64)
    i, q = lanes & 15, lanes >> 4

    def parts(v, kind):
        if f32 or kind == "bf16":
            return [v]
        v32 = v.astype(np.float32)
        hi = bf16_rne(v32)
        r1 = v32 - hi
        mid = bf16_rne(r1)
        return [t.astype(np.float64) for t in (hi, mid, bf16_rne(r1 - mid))]

    nside = C // T
    for ch in range(chunks):
        r_end = min(rows, ch * rpc + rpc)
        for blk in range(nside * nside):
            c0, d0 = (blk // nside) * T, (blk % nside) * T
            for w in range(4 if T >= 32 else 1):
                tr0, tc0 = ((w >> 1) * TQ, (w & 1) * TQ) if T >= 32 else (0, 0)
                acc = {(x, y): np.zeros((64, 4)) for x in range(TQ) for y in range(TQ)}
                for r0 in range(ch * rpc, r_end, RB):
                    step = 4 if f32 else 32
                    for kb in range(0, RB, step):
                        slots = [kb + q] if f32 else [kb + q + 4 * e for e in range(8)]
                        for x in range(TQ):
                            for y in range(TQ):
                                sa, sb = [], []
                                for rr in slots:
                                    row = r0 + rr
                                    ok = row < r_end
                                    rw = np.where(ok, row, 0)
                                    sa.append(np.where(ok, a[rw, c0 + 16 * (tr0 + x) + i], 0.0))
                                    sb.append(np.where(ok, b[rw, d0 + 16 * (tc0 + y) + i], 0.0))
                                av, bv = np.stack(sa, 1), np.stack(sb, 1)   # [64 lanes, k]
                                for pa in parts(av, kinds[0]):
                                    for pb in parts(bv, kinds[1]):
                                        acc[x, y] = mfma_k(pa, pb, acc[x, y])
                for (x, y), v in acc.items():
                    for r in range(4):
                        part[ch, c0 + 16 * (tr0 + x) + 4 * q + r, d0 + 16 * (tc0 + y) + i] = v[:, r]
    assert not np.isnan(part).any()
    # fixed-order sum: groups of 16 consecutive chunks, then the groups
    groups = [part[g:g + 16].sum(axis=0) for g in range(0, chunks, 16)]
    return np.sum(groups, axis=0)


def mfma_k(av, bv, acc):
    """One 16x16xK MFMA: lane 16q + i holds k-slots of row i (a) / column i
    (b); the result lane 16q + j holds rows 4q + r of column j."""
    K = av.shape[1]
    A = np.zeros((16, 4 * K))
    Bm = np.zeros((4 * K, 16))
    for lane in range(64):
        ii, qq = lane & 15, lane >> 4
        A[ii, qq * K:(qq + 1) * K] = av[lane]
        Bm[qq * K:(qq + 1) * K, ii] = bv[lane]
    D = A @ Bm
    out = acc.copy()
    for lane in range(64):
        j, qq = lane & 15, lane >> 4
        out[lane] += D[4 * qq:4 * qq + 4, j]
    return out


@pytest.mark.parametrize("rows,cb", [(130, 4), (77, 5), (300, 7), (1000, 7), (4, 6), (1100, 4),
                                     (70, 8)])
@pytest.mark.parametrize("kinds", [("f32", "f32"), ("f32", "bf16"), ("bf16", "f32"),
                                   ("bf16", "bf16")])
def test_weight_gradient_model(rows, cb, kinds):
    """The modelled kernel's index maps reproduce A^T B: exactly for float32 x
    float32 and bf16 x bf16, within the hi/lo split's residual otherwise."""
    rng = np.random.default_rng(rows + cb)
    C = 1 << cb
    a = rng.standard_normal((rows, C)).astype(np.float32).astype(np.float64)
    b = rng.standard_normal((rows, C)).astype(np.float32).astype(np.float64)
    if kinds[0] == "bf16":
        a = bf16_rne(a).astype(np.float64)
    if kinds[1] == "bf16":
        b = bf16_rne(b).astype(np.float64)
    ref = a.T @ b
    got = model_wgrad(a, b, cb, kinds)
    tol = 1e-10 if kinds[0] == kinds[1] else 2.0 ** -26
    assert np.max(np.abs(got - ref)) <= tol * np.max(np.abs(a).sum(0)[:, None] * np.abs(b).max(0))
    chunks, rpc = wgrad_plan(rows, cb)
    assert chunks * rpc >= rows and (chunks - 1) * rpc < rows and rpc % 4 == 0
