"""Checks that pin the CPU oracle to facts fixed outside the oracle itself.

Each ``pin_*`` function takes an ``oracle.oracle.Oracle`` and raises
AssertionError when the oracle disagrees with the paper or with mathematics
that does not depend on the oracle's code:

* a library Sylvester construction (``scipy.linalg.hadamard``) and the closed
  form (-1)^popcount(i & j) of the matrix entries (section III-B);
* dense matrix products of the mixer's definition;
* the dyadic (XOR) convolution form of the mixer, by brute force;
* hand-worked examples under ``tests/golden/``;
* invariants: unit gain is the identity (the zero-initialised log gain of
  section III-B), energy preservation of orthonormal transforms, one-hot gains
  selecting a single Walsh basis image, linearity, self-adjointness, batch
  independence;
* the paper's separable form (eq. (2) then eq. (3)) equals the joint gain
  form with a rank-one G;
* zero padding of the token axis (section III-B) against dense products of
  explicitly padded matrices;
* the backward pass (dX, dG and the separable log-gain gradients) against
  dense products and against finite differences of the forward mixer;
* the full block of eqs. (1)-(4) (projections W_in, W_out around the mixer)
  against dense products, and its gradients against an explicit dense
  operator and finite differences.

The same functions run against the real oracle (``test_oracle_pins.py``) and
against deliberately broken copies of it (``test_oracle_mutants.py``), which
shows that a plausible mistake anywhere in the oracle fails at least one pin.
"""
from __future__ import annotations

import json
import os

import numpy as np
import scipy.linalg

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

SHAPES_SMALL = [(1, 1), (2, 1), (1, 2), (2, 2), (4, 8), (8, 4), (16, 16),
                (2, 64), (64, 2), (32, 8), (1, 32), (128, 1)]


def _rel(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = max(np.max(np.abs(b)), 1e-300)
    return float(np.max(np.abs(a - b)) / den) if a.size else 0.0


def _popcount(v: int) -> int:
    return bin(v).count("1")


def _walsh(n: int, k: int) -> np.ndarray:
    """Row k of the orthonormal Sylvester matrix, by the closed form."""
    return np.array([(-1.0) ** _popcount(k & i) for i in range(n)]) / np.sqrt(n)


def _hadamard_orth(n: int) -> np.ndarray:
    return scipy.linalg.hadamard(n).astype(np.float64) / np.sqrt(n)


# --------------------------------------------------------------------------
def pin_sylvester_closed_form(o) -> None:
    """scipy's Sylvester construction has entries (-1)^popcount(i & j): the
    natural (Hadamard) ordering that section III-B names."""
    for n in [1, 2, 4, 8, 16, 64]:
        H = scipy.linalg.hadamard(n)
        ref = np.array([[(-1) ** _popcount(i & j) for j in range(n)]
                        for i in range(n)])
        assert np.array_equal(H, ref), n


def pin_butterfly_matches_dense(o) -> None:
    """The oracle's butterfly equals the dense +/-1 Sylvester product."""
    rng = np.random.default_rng(100)
    for k in range(0, 10):
        n = 1 << k
        v = rng.standard_normal(n)
        got = o.fwht(v)
        ref = scipy.linalg.hadamard(n).astype(np.float64) @ v
        assert _rel(got, ref) < 1e-13, (n, _rel(got, ref))


def pin_dense_product(o) -> None:
    """Y = H_N (G o (H_N X H_C)) H_C with explicit orthonormal matrices."""
    rng = np.random.default_rng(101)
    for (N, C) in SHAPES_SMALL + [(64, 64), (256, 16)]:
        x = rng.standard_normal((N, C))
        g = rng.uniform(0.5, 1.5, (N, C))
        Hn, Hc = _hadamard_orth(N), _hadamard_orth(C)
        ref = Hn @ (g * (Hn @ x @ Hc)) @ Hc
        got = o.whtmix(x, g)
        assert got.shape == (N, C)
        assert _rel(got, ref) < 1e-12, ((N, C), _rel(got, ref))


def pin_dyadic_convolution(o) -> None:
    """Brute force: Y[n,c] = sum_{m,d} K[n^m, c^d] X[m,d] with
    K[i,j] = (1/(N C)) sum_{k,l} G[k,l] (-1)^(popcount(i&k) + popcount(j&l)).
    (Expanding the definition entry-wise and using
    (-1)^popcount(n&k) (-1)^popcount(m&k) = (-1)^popcount((n^m)&k).)"""
    rng = np.random.default_rng(102)
    for (N, C) in [(1, 1), (2, 1), (1, 4), (4, 2), (2, 8), (8, 8), (16, 4)]:
        x = rng.standard_normal((N, C))
        g = rng.uniform(-1.0, 2.0, (N, C))
        K = np.zeros((N, C))
        for i in range(N):
            for j in range(C):
                s = 0.0
                for k in range(N):
                    for l in range(C):
                        sgn = -1.0 if (_popcount(i & k) + _popcount(j & l)) & 1 else 1.0
                        s += sgn * g[k, l]
                K[i, j] = s / (N * C)
        ref = np.zeros((N, C))
        for n in range(N):
            for c in range(C):
                s = 0.0
                for m in range(N):
                    for d in range(C):
                        s += K[n ^ m, c ^ d] * x[m, d]
                ref[n, c] = s
        got = o.whtmix(x, g)
        assert _rel(got, ref) < 1e-12, ((N, C), _rel(got, ref))


def pin_golden_hand_examples(o) -> None:
    """Hand-worked values (tests/golden/hand_examples.json)."""
    with open(os.path.join(GOLDEN, "hand_examples.json")) as f:
        data = json.load(f)
    for case in data["cases"]:
        got = o.whtmix(np.array(case["x"]), np.array(case["g"]))
        ref = np.array(case["y"])
        assert np.allclose(got, ref, rtol=0, atol=1e-13), (case["name"], got, ref)


def pin_unit_gain_identity(o) -> None:
    """Zero log gain = unit gain (section III-B): G = 1 returns X, because H is
    orthonormal and involutory."""
    rng = np.random.default_rng(103)
    for (N, C) in SHAPES_SMALL + [(1024, 64), (4096, 2)]:
        x = rng.standard_normal((2, N, C))
        got = o.whtmix(x, np.ones((N, C)))
        assert _rel(got, x) < 1e-13, ((N, C), _rel(got, x))


def pin_energy(o) -> None:
    """Orthonormal transforms preserve energy (section III-B, magnitude
    preserving): a +/-1 gain keeps ||Y|| = ||X||; any gain keeps
    min|G| ||X|| <= ||Y|| <= max|G| ||X||."""
    rng = np.random.default_rng(104)
    for (N, C) in [(8, 4), (64, 32), (256, 8), (2, 1)]:
        x = rng.standard_normal((N, C))
        s = rng.choice([-1.0, 1.0], size=(N, C))
        y = o.whtmix(x, s)
        assert abs(np.linalg.norm(y) / np.linalg.norm(x) - 1) < 1e-13
        g = rng.uniform(0.25, 3.0, (N, C))
        y = o.whtmix(x, g)
        nx, ny = np.linalg.norm(x), np.linalg.norm(y)
        assert g.min() * nx * (1 - 1e-12) <= ny <= g.max() * nx * (1 + 1e-12)


def pin_one_hot_gain(o) -> None:
    """A gain that keeps only frequency (k, j) projects X onto the single Walsh
    basis image B = h_k h_j^T: Y = <X, B> B.  X = B is kept whole by that gain
    and removed by any other one-hot gain."""
    rng = np.random.default_rng(105)
    for (N, C) in [(8, 4), (4, 16), (16, 2), (1, 8), (32, 1)]:
        x = rng.standard_normal((N, C))
        for (k, j) in [(0, 0), (N - 1, C - 1), (N // 2, C // 3), (1 % N, 0)]:
            B = np.outer(_walsh(N, k), _walsh(C, j))
            g = np.zeros((N, C))
            g[k, j] = 1.0
            got = o.whtmix(x, g)
            ref = np.sum(x * B) * B
            assert _rel(got, ref) < 1e-12, ((N, C, k, j), _rel(got, ref))
            kept = o.whtmix(B, g)
            assert _rel(kept, B) < 1e-12
            k2, j2 = (k + 1) % N, (j + 1) % C
            if (k2, j2) != (k, j):
                g2 = np.zeros((N, C))
                g2[k2, j2] = 1.0
                assert np.max(np.abs(o.whtmix(B, g2))) < 1e-13


def pin_separable_form(o) -> None:
    """The paper's eq. (2) then eq. (3) with log gains equals, with dense
    matrices, H_N D_t H_N X H_C D_c H_C, and equals the joint form with the
    rank-one gain exp(g_t) exp(g_c)^T."""
    rng = np.random.default_rng(106)
    for (N, C) in [(8, 4), (2, 32), (64, 8), (1, 4), (4, 1)]:
        x = rng.standard_normal((3, N, C))
        gt = rng.normal(0, 0.5, N)
        gc = rng.normal(0, 0.5, C)
        Hn, Hc = _hadamard_orth(N), _hadamard_orth(C)
        Dt, Dc = np.diag(np.exp(gt)), np.diag(np.exp(gc))
        ref = np.stack([Hn @ Dt @ Hn @ xb @ Hc @ Dc @ Hc for xb in x])
        got = o.whtmix_separable(x, gt, gc)
        assert _rel(got, ref) < 1e-12, ((N, C), _rel(got, ref))
        joint = o.whtmix(x, np.outer(np.exp(gt), np.exp(gc)))
        assert _rel(joint, ref) < 1e-12, ((N, C), _rel(joint, ref))


def pin_flat_1d_equivalence(o) -> None:
    """H_N kron H_C = H_{N C} in Sylvester order, so the mixer is also
    (1/(N C)) H (g o H x) on the flattened row-major slice of length N C.
    (Checked with the dense 1-D matrix; this is the fact the GPU's bit-group
    passes rely on.)"""
    rng = np.random.default_rng(107)
    for (N, C) in [(4, 8), (16, 4), (2, 2), (8, 32)]:
        x = rng.standard_normal((N, C))
        g = rng.uniform(0.5, 1.5, (N, C))
        H = scipy.linalg.hadamard(N * C).astype(np.float64)
        ref = (H @ (g.reshape(-1) * (H @ x.reshape(-1)))) / (N * C)
        got = o.whtmix(x, g).reshape(-1)
        assert _rel(got, ref) < 1e-12, ((N, C), _rel(got, ref))


def pin_structure(o) -> None:
    """Linearity in X, linearity in G, self-adjointness <f(X1),X2> = <X1,f(X2)>
    (H and diag(G) are symmetric), and batch independence / equivariance."""
    rng = np.random.default_rng(108)
    N, C = 16, 8
    g = rng.uniform(-1, 2, (N, C))
    x1, x2 = rng.standard_normal((2, N, C))
    a, b = 1.7, -0.3
    f = lambda x, gg=g: o.whtmix(x, gg)
    assert _rel(f(a * x1 + b * x2), a * f(x1) + b * f(x2)) < 1e-12
    assert _rel(o.whtmix(x1, 2.5 * g), 2.5 * f(x1)) < 1e-12
    lhs, rhs = np.sum(f(x1) * x2), np.sum(x1 * f(x2))
    assert abs(lhs - rhs) < 1e-12 * max(1.0, abs(lhs))
    xb = rng.standard_normal((5, N, C))
    yb = o.whtmix(xb, g)
    for i in range(5):
        assert np.array_equal(yb[i], o.whtmix(xb[i], g)), i
    perm = [3, 0, 4, 1, 2]
    assert np.array_equal(o.whtmix(xb[perm], g), yb[perm])


def _pad_rows(x, P):
    return np.concatenate([x, np.zeros((P - x.shape[0],) + x.shape[1:])], axis=0)


def pin_padding_dense(o) -> None:
    """Section III-B zero-pads the token axis to the next power of two before
    H_N: with dense matrices, Y = first N rows of
    H_P (G o (H_P [X; 0] H_C)) H_C, and likewise for the separable form."""
    rng = np.random.default_rng(109)
    for (N, C) in [(3, 4), (5, 2), (6, 8), (7, 1), (9, 4), (12, 16), (100, 2), (33, 32)]:
        P = 1 << (N - 1).bit_length()
        x = rng.standard_normal((2, N, C))
        g = rng.uniform(0.5, 1.5, (P, C))
        Hp, Hc = _hadamard_orth(P), _hadamard_orth(C)
        ref = np.stack([(Hp @ (g * (Hp @ _pad_rows(xb, P) @ Hc)) @ Hc)[:N] for xb in x])
        got = o.whtmix(x, g)
        assert got.shape == x.shape
        assert _rel(got, ref) < 1e-12, ((N, C), _rel(got, ref))
        gt, gc = rng.normal(0, 0.5, P), rng.normal(0, 0.5, C)
        Dt, Dc = np.diag(np.exp(gt)), np.diag(np.exp(gc))
        ref = np.stack([(Hp @ Dt @ Hp @ _pad_rows(xb, P) @ Hc @ Dc @ Hc)[:N] for xb in x])
        got = o.whtmix_separable(x, gt, gc)
        assert _rel(got, ref) < 1e-12, ((N, C), _rel(got, ref))


def pin_padding_unit_gain(o) -> None:
    """Padding rows are zeros, so a unit gain still returns X exactly."""
    rng = np.random.default_rng(110)
    for (N, C) in [(3, 1), (17, 8), (1000, 4), (9216 // 8, 8)]:
        P = 1 << (N - 1).bit_length()
        x = rng.standard_normal((2, N, C))
        assert _rel(o.whtmix(x, np.ones((P, C))), x) < 1e-13, (N, C)
        assert _rel(o.whtmix_separable(x, np.zeros(P), np.zeros(C)), x) < 1e-13, (N, C)


def pin_grad_dense(o) -> None:
    """Backward with dense matrices: dX = first N rows of
    H_P (G o (H_P [dY; 0] H_C)) H_C and dG = sum_b T_x[b] o T_dy[b] with
    T = H_P [.; 0] H_C; separable log gains by the chain rule through exp."""
    rng = np.random.default_rng(111)
    for (N, C, B) in [(4, 8, 3), (3, 4, 2), (16, 2, 1), (1, 8, 2), (6, 1, 2)]:
        P = 1 << (N - 1).bit_length()
        Hp, Hc = _hadamard_orth(P), _hadamard_orth(C)
        x = rng.standard_normal((B, N, C))
        dy = rng.standard_normal((B, N, C))
        g = rng.uniform(0.5, 1.5, (P, C))
        T = lambda a: Hp @ _pad_rows(a, P) @ Hc
        dx_ref = np.stack([(Hp @ (g * T(d)) @ Hc)[:N] for d in dy])
        dg_ref = sum(T(xb) * T(db) for xb, db in zip(x, dy))
        dx, dg = o.whtmix_grad(x, dy, g)
        assert _rel(dx, dx_ref) < 1e-12 and _rel(dg, dg_ref) < 1e-12, (N, C)
        gt, gc = rng.normal(0, 0.4, P), rng.normal(0, 0.4, C)
        G = np.outer(np.exp(gt), np.exp(gc))
        dG = sum(T(xb) * T(db) for xb, db in zip(x, dy))
        dx_ref = np.stack([(Hp @ (G * T(d)) @ Hc)[:N] for d in dy])
        dx, dgt, dgc = o.whtmix_grad_separable(x, dy, gt, gc)
        assert _rel(dx, dx_ref) < 1e-12, (N, C)
        assert _rel(dgt, (dG * G).sum(axis=1)) < 1e-12 and _rel(dgc, (dG * G).sum(axis=0)) < 1e-12


def pin_grad_finite_differences(o) -> None:
    """The loss L = sum_b <Y_b, W_b> is linear in G and in X, so central
    differences of the forward mixer give dG and dX up to rounding; in the
    log gains it is smooth, checked with a small step."""
    rng = np.random.default_rng(112)
    B, N, C = 2, 5, 4
    P = 8
    x = rng.standard_normal((B, N, C))
    w = rng.standard_normal((B, N, C))
    g = rng.uniform(0.5, 1.5, (P, C))
    dx, dg = o.whtmix_grad(x, w, g)
    loss = lambda xx, gg: float(np.sum(o.whtmix(xx, gg) * w))
    for (i, j) in [(0, 0), (3, 2), (7, 3), (5, 1)]:
        e = np.zeros((P, C))
        e[i, j] = 1.0
        fd = (loss(x, g + 0.5 * e) - loss(x, g - 0.5 * e)) / 1.0
        assert abs(fd - dg[i, j]) < 1e-12 * max(1.0, abs(fd)), (i, j)
    for (b, n, c) in [(0, 0, 0), (1, 4, 3), (0, 2, 1)]:
        e = np.zeros((B, N, C))
        e[b, n, c] = 1.0
        fd = (loss(x + 0.5 * e, g) - loss(x - 0.5 * e, g)) / 1.0
        assert abs(fd - dx[b, n, c]) < 1e-12 * max(1.0, abs(fd)), (b, n, c)
    gt, gc = rng.normal(0, 0.3, P), rng.normal(0, 0.3, C)
    _, dgt, dgc = o.whtmix_grad_separable(x, w, gt, gc)
    sloss = lambda a, b_: float(np.sum(o.whtmix_separable(x, a, b_) * w))
    h = 1e-5
    for n in [0, 3, 7]:
        e = np.zeros(P)
        e[n] = h
        fd = (sloss(gt + e, gc) - sloss(gt - e, gc)) / (2 * h)
        assert abs(fd - dgt[n]) < 1e-7 * max(1.0, abs(fd)), n
    for c in [0, 2]:
        e = np.zeros(C)
        e[c] = h
        fd = (sloss(gt, gc + e) - sloss(gt, gc - e)) / (2 * h)
        assert abs(fd - dgc[c]) < 1e-7 * max(1.0, abs(fd)), c


def pin_module_dense(o) -> None:
    """The full block of eqs. (1)-(4) with dense matrices: the projections are
    plain matrix products around the (padded) mixer, Y = M(X W_in) W_out,
    for both gain forms; identity weights reduce it to the mixer."""
    rng = np.random.default_rng(113)
    for (B, N, C) in [(2, 8, 4), (1, 5, 8), (3, 16, 16), (2, 3, 2)]:
        P = 1 << (N - 1).bit_length()
        Hp, Hc = _hadamard_orth(P), _hadamard_orth(C)
        x = rng.standard_normal((B, N, C))
        wi = rng.standard_normal((C, C)) / np.sqrt(C)
        wo = rng.standard_normal((C, C)) / np.sqrt(C)
        g = rng.uniform(0.5, 1.5, (P, C))
        mix = lambda z, G: (Hp @ (G * (Hp @ _pad_rows(z, P) @ Hc)) @ Hc)[:N]
        ref = np.stack([mix(xb @ wi, g) @ wo for xb in x])
        assert _rel(o.whtmix_module(x, wi, g, wo), ref) < 1e-12, (B, N, C)
        gt, gc = rng.normal(0, 0.3, P), rng.normal(0, 0.3, C)
        G = np.outer(np.exp(gt), np.exp(gc))
        ref = np.stack([mix(xb @ wi, G) @ wo for xb in x])
        assert _rel(o.whtmix_module_separable(x, wi, gt, gc, wo), ref) < 1e-12, (B, N, C)
        eye = np.eye(C)
        assert _rel(o.whtmix_module(x, eye, g, eye), o.whtmix(x, g)) < 1e-13


def pin_module_grad(o) -> None:
    """Gradients of the block, eqs. (1)-(4), for L = sum_b <dY_b, Y_b>.
    dense: the mixer is written out as an explicit (N C) x (N C) matrix M built
    from dense Hadamard products, and the chain rule is applied with M^T (no use
    of self-adjointness): dZ' = dY W_out^T, dW_out = sum Z'^T dY, dZ = M^T dZ',
    dX = dZ W_in^T, dW_in = sum X^T dZ.  finite differences: L is linear in
    each of X, W_in, W_out and G, so unit central differences are exact up to
    rounding; in the log gains it is smooth (small step)."""
    rng = np.random.default_rng(114)
    B, N, C = 2, 5, 4
    P = 8
    Hp, Hc = _hadamard_orth(P), _hadamard_orth(C)
    x = rng.standard_normal((B, N, C))
    dy = rng.standard_normal((B, N, C))
    wi = rng.standard_normal((C, C)) / np.sqrt(C)
    wo = rng.standard_normal((C, C)) / np.sqrt(C)
    g = rng.uniform(0.5, 1.5, (P, C))

    def mix(z, G):
        return (Hp @ (G * (Hp @ _pad_rows(z, P) @ Hc)) @ Hc)[:N]

    M = np.stack([mix(e.reshape(N, C), g).reshape(-1) for e in np.eye(N * C)], axis=1)
    dx, dwi, dwo, dg = o.whtmix_module_grad(x, wi, g, wo, dy)
    ref_dwi = np.zeros((C, C))
    ref_dwo = np.zeros((C, C))
    for b in range(B):
        z = x[b] @ wi
        zp = (M @ z.reshape(-1)).reshape(N, C)
        dzp = dy[b] @ wo.T
        ref_dwo += zp.T @ dy[b]
        dz = (M.T @ dzp.reshape(-1)).reshape(N, C)
        assert _rel(dx[b], dz @ wi.T) < 1e-12, b
        ref_dwi += x[b].T @ dz
    assert _rel(dwi, ref_dwi) < 1e-12 and _rel(dwo, ref_dwo) < 1e-12

    loss = lambda xx, a, gg, bb: float(np.sum(o.whtmix_module(xx, a, gg, bb) * dy))
    for (i, j) in [(0, 0), (3, 2), (7, 3)]:
        e = np.zeros((P, C))
        e[i, j] = 1.0
        fd = (loss(x, wi, g + 0.5 * e, wo) - loss(x, wi, g - 0.5 * e, wo))
        assert abs(fd - dg[i, j]) < 1e-11 * max(1.0, abs(fd)), (i, j)
    for (i, j) in [(0, 1), (2, 3), (3, 0)]:
        e = np.zeros((C, C))
        e[i, j] = 1.0
        fd = loss(x, wi + 0.5 * e, g, wo) - loss(x, wi - 0.5 * e, g, wo)
        assert abs(fd - dwi[i, j]) < 1e-11 * max(1.0, abs(fd)), ("w_in", i, j)
        fd = loss(x, wi, g, wo + 0.5 * e) - loss(x, wi, g, wo - 0.5 * e)
        assert abs(fd - dwo[i, j]) < 1e-11 * max(1.0, abs(fd)), ("w_out", i, j)
    for (b, n, c) in [(0, 0, 0), (1, 4, 3)]:
        e = np.zeros((B, N, C))
        e[b, n, c] = 1.0
        fd = loss(x + 0.5 * e, wi, g, wo) - loss(x - 0.5 * e, wi, g, wo)
        assert abs(fd - dx[b, n, c]) < 1e-11 * max(1.0, abs(fd)), (b, n, c)

    gt, gc = rng.normal(0, 0.3, P), rng.normal(0, 0.3, C)
    sdx, sdwi, sdwo, dgt, dgc = o.whtmix_module_grad_separable(x, wi, gt, gc, wo, dy)
    G = np.outer(np.exp(gt), np.exp(gc))
    jdx, jdwi, jdwo, _ = o.whtmix_module_grad(x, wi, G, wo, dy)
    assert _rel(sdx, jdx) < 1e-12 and _rel(sdwi, jdwi) < 1e-12 and _rel(sdwo, jdwo) < 1e-12
    sloss = lambda a, b_: float(np.sum(o.whtmix_module_separable(x, wi, a, b_, wo) * dy))
    h = 1e-5
    for n in [0, 5]:
        e = np.zeros(P)
        e[n] = h
        fd = (sloss(gt + e, gc) - sloss(gt - e, gc)) / (2 * h)
        assert abs(fd - dgt[n]) < 1e-7 * max(1.0, abs(fd)), n
    e = np.zeros(C)
    e[1] = h
    fd = (sloss(gt, gc + e) - sloss(gt, gc - e)) / (2 * h)
    assert abs(fd - dgc[1]) < 1e-7 * max(1.0, abs(fd))


def pin_rejects_bad_shapes(o) -> None:
    """The channel transform needs a power-of-two C (section III-B pads only
    the token axis); a token count must be at least 1."""
    for (N, C) in [(4, 3), (4, 6), (12, 12)]:
        try:
            o.whtmix(np.zeros((N, C)), np.ones((1 << (N - 1).bit_length(), C)))
        except ValueError:
            continue
        raise AssertionError(f"accepted non-power-of-two C {(N, C)}")


ALL_PINS = [
    pin_sylvester_closed_form,
    pin_butterfly_matches_dense,
    pin_dense_product,
    pin_dyadic_convolution,
    pin_golden_hand_examples,
    pin_unit_gain_identity,
    pin_energy,
    pin_one_hot_gain,
    pin_separable_form,
    pin_flat_1d_equivalence,
    pin_structure,
    pin_padding_dense,
    pin_padding_unit_gain,
    pin_grad_dense,
    pin_grad_finite_differences,
    pin_module_dense,
    pin_module_grad,
    pin_rejects_bad_shapes,
]
