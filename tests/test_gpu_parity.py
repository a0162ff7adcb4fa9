"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Both sides receive the same seeded inputs (paper_2607_25234_amd.workloads);
the oracle computes in float64.  The bar is the normwise maximum relative
error max|y - r| / max|r| over the whole output: <= 1e-5 for float32 I/O and
<= 2e-2 for bf16 I/O with float32 arithmetic.
"""
import numpy as np
import pytest

from oracle import oracle as oracle_mod
from paper_2607_25234_amd import whtmix, workloads
from tests.gpu_util import (DERIVED, TOL, case_ids, device, errors, random_cases, run_gpu,
                            run_gpu_separable, say, to_device, to_host)

log_gains = workloads.draw_log_gains

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return device()


@pytest.fixture(scope="module")
def orc():
    return oracle_mod.Oracle()


def check(name, y, ref, dtype):
    """The stated tolerance and the tighter bound the arithmetic allows."""
    err, rms = errors(y, ref)
    say(f"  {name}: normwise-max {err:.3e} rms {rms:.3e} (tol {TOL[dtype]:g}, "
        f"derived {DERIVED[dtype]:.3e})")
    assert y.shape == ref.shape
    assert np.all(np.isfinite(y))
    assert err <= TOL[dtype], (name, err)
    assert err <= DERIVED[dtype], (name, err)
    return err


@pytest.mark.parametrize("name", list(workloads.WORKLOADS))
def test_workload_parity(name, dev, orc):
    """Every workload at full size, in the plan the benchmark runs."""
    w = workloads.WORKLOADS[name]
    say(f"workload {name}: B={w.B} N={w.N} C={w.C} {w.dtype}")
    x, g = workloads.inputs(w)
    y = run_gpu(x, g, w.dtype, dev)
    ref = orc.whtmix(x, g)
    check(name, y, ref, w.dtype)


SHAPES = [
    # (B, N, C) -- K = log2(N*C) from 0 (degenerate) to 20, square and
    # skewed, every plan and every three-pass split shape class
    (1, 1, 1), (3, 1, 1), (2, 2, 1), (1, 1, 2), (2, 4, 8), (1, 16, 1),
    (5, 32, 32), (2, 1, 1024), (1, 1024, 1),
    (3, 64, 32), (1, 2048, 1), (2, 1, 2048), (2, 128, 32), (4, 64, 128),
    (1, 8192, 2), (2, 512, 64), (3, 256, 128),
    (1, 1024, 64), (2, 65536, 1), (1, 1, 65536), (2, 512, 256),
    (1, 4096, 64), (3, 1024, 256), (1, 16384, 64), (2, 4096, 512),
    (1, 8192, 128),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_shapes(shape, dtype, dev, orc):
    B, N, C = shape
    x, g = workloads.draw(B, N, C, dtype, seed=11 + N + 3 * C + B)
    plan = whtmix.plan_describe(B, N, C, dtype)["plan"]
    say(f"shape {shape} {dtype} plan={plan}")
    y = run_gpu(x, g, dtype, dev)
    check(f"{shape}", y, orc.whtmix(x, g), dtype)


# Token counts that are not powers of two (zero padding, section III-B),
# including the paper's stereo joint token counts 9216, 25600 and 50176
# (384x768, 640x1280 and 896x1792 images).
# 139872 x 256 pads to a 2^26 slice: 2^16-element outer tiles, the
# straddling one with its second 2^15 register set wholly padding.  bf16
# slices whose byte size is a multiple of 16 move with 16-byte accesses (the
# straddling tile element by element); 262143 x 4 in bf16 (2 097 144 bytes)
# is not, and takes per-element accesses throughout.
PADDED = [(1, 3, 4), (2, 5, 8), (1, 100, 8), (3, 1000, 16), (2, 130, 128), (2, 9216, 64),
          (1, 25600, 64), (1, 50176, 64), (2, 36864, 64), (1, 139872, 256), (2, 262143, 4),
          # 2^16 in one workgroup: the second register set partly or wholly padding
          (2, 1000, 64), (1, 300, 128), (3, 513, 64)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", PADDED, ids=lambda s: "x".join(map(str, s)))
def test_padded_tokens(shape, dtype, dev, orc):
    B, N, C = shape
    P = whtmix.padded_tokens(N)
    x, _ = workloads.draw(B, N, C, dtype, seed=300 + N)
    _, g = workloads.draw(1, P, C, "f32", seed=301 + N)
    d = whtmix.plan_describe(B, N, C, dtype)
    plan, K = d["plan"], d["log2_slice"]
    say(f"padded {shape} -> P={P} {dtype} plan={plan}")
    ref = orc.whtmix(x, g)
    check(f"{shape}", run_gpu(x, g, dtype, dev), ref, dtype)
    # the other plan of slices one workgroup can hold (2^11..2^16)
    if 12 <= K <= 16:
        other = "three_pass" if plan == "fused" else "fused"
        check(f"{shape} {other}", run_gpu(x, g, dtype, dev, plan=other), ref, dtype)


RANDOM_CASES = random_cases(40, 2607)


@pytest.mark.parametrize("case", RANDOM_CASES, ids=case_ids(RANDOM_CASES))
def test_random_shapes_every_plan(case, dev, orc):
    """Each seeded shape through AUTO and every plan it allows, against the
    oracle: the plans must agree with the definition wherever they apply."""
    B, N, C, dtype = case
    x, _ = workloads.draw(B, N, C, dtype, seed=5000 + 7 * N + C + B)
    P = whtmix.padded_tokens(N)
    _, g = workloads.draw(1, P, C, "f32", seed=5001 + N)
    g = g.reshape(P, C)
    ref = orc.whtmix(x, g)
    plans = ["auto"]
    for p in ("small", "fused", "three_pass", "wave_tiles", "one_launch", "two_pass"):
        try:
            whtmix.plan_describe(B, N, C, dtype, p)
        except whtmix.WhtmixError:
            continue
        plans.append(p)
    for p in plans:
        say(f"random {case} plan={p}")
        check(f"{case} {p}", run_gpu(x, g, dtype, dev, plan=p), ref, dtype)


SEPARABLE_CASES = random_cases(24, 2608)


@pytest.mark.parametrize("case", SEPARABLE_CASES, ids=case_ids(SEPARABLE_CASES))
def test_random_shapes_separable(case, dev, orc):
    """The separable form (eqs. (2)-(3), log-domain gains) on seeded shapes,
    through AUTO, against the oracle's two-stage form."""
    B, N, C, dtype = case
    P = whtmix.padded_tokens(N)
    x, _ = workloads.draw(B, N, C, dtype, seed=6000 + 7 * N + C + B)
    gt, gc = log_gains(P, C, seed=6001 + N)
    say(f"random separable {case}")
    check(f"{case} separable", run_gpu_separable(x, gt, gc, dtype, dev),
          orc.whtmix_separable(x, gt, gc), dtype)


def test_fused_2_16_large_batch(dev, orc):
    """2^16-element slices in batches of 48 and more take one workgroup each."""
    B, N, C = 64, 1000, 64
    assert whtmix.plan_describe(B, N, C)["plan"] == "fused"
    x, g = workloads.draw(B, N, C, "f32", seed=61)
    _, g = workloads.draw(1, 1024, C, "f32", seed=62)
    check("2^16 x 64", run_gpu(x, g, "f32", dev), orc.whtmix(x, g), "f32")


def test_pair_tiles_two_padded_slices(dev, orc):
    """Two bf16 slices of 100000 x 512, padded to 2^26: 2048 outer tiles of
    2^16 over the forward outer pass's 256 persistent workgroups (8 each),
    among them tiles that straddle the last token and tiles wholly in the
    padding; the backward takes x and dy in one such launch."""
    import torch
    B, N, C, dtype = 2, 100000, 512, "bf16"
    d = whtmix.plan_describe(B, N, C, dtype)
    assert (d["plan"], d["log2_slice"]) == ("three_pass", 26)
    P = whtmix.padded_tokens(N)
    x, _ = workloads.draw(B, N, C, dtype, seed=71)
    _, g = workloads.draw(1, P, C, "f32", seed=72)
    g = g.reshape(P, C)
    say(f"pair tiles {(B, N, C)} {dtype}")
    check("forward", run_gpu(x, g, dtype, dev), orc.whtmix(x, g), dtype)
    dy, _ = workloads.draw(B, N, C, dtype, seed=73)
    dx, dg = whtmix.backward(to_device(x, dtype, dev), to_device(dy, dtype, dev),
                             torch.from_numpy(g).to(dev))
    torch.cuda.synchronize(dev)
    dx_ref, dg_ref = orc.whtmix_grad(x, dy, g)
    check("dx", to_host(dx), dx_ref, dtype)
    e, _ = errors(to_host(dg), dg_ref)
    say(f"  dG: normwise-max {e:.3e}")
    assert e <= 1e-5, e


SEPARABLE = [(1, 1, 1), (2, 32, 32), (3, 64, 128), (2, 4096, 64), (1, 9216, 64),
             (2, 16384, 128), (1, 1000, 16), (2, 1000, 64)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SEPARABLE, ids=lambda s: "x".join(map(str, s)))
def test_separable_gains(shape, dtype, dev, orc):
    """The paper's parametrisation: eq. (2) then eq. (3) with log gains."""
    B, N, C = shape
    P = whtmix.padded_tokens(N)
    x, _ = workloads.draw(B, N, C, dtype, seed=400 + N)
    gt, gc = log_gains(P, C, seed=401 + N)
    plan = whtmix.plan_describe(B, N, C, dtype)["plan"]
    say(f"separable {shape} {dtype} plan={plan}")
    check(f"separable {shape}", run_gpu_separable(x, gt, gc, dtype, dev),
          orc.whtmix_separable(x, gt, gc), dtype)


def test_separable_workload(dev, orc):
    """The benchmarked workload shape with the paper's log gains."""
    w = workloads.WORKLOADS[workloads.BENCH_WORKLOAD]
    x, _ = workloads.inputs(w)
    gt, gc = log_gains(w.N, w.C, seed=77)
    check("separable stereo64k_bf16", run_gpu_separable(x, gt, gc, w.dtype, dev),
          orc.whtmix_separable(x, gt, gc), w.dtype)


def test_separable_zero_log_gain_and_joint_equivalence(dev):
    """Zero log gains (the paper's initialisation) give Y = X, and the
    separable entry point matches the joint one with G = exp(g_t) exp(g_c)^T."""
    B, N, C = 2, 4096, 64
    x, _ = workloads.draw(B, N, C, "f32", seed=5)
    y0 = run_gpu_separable(x, np.zeros(N, np.float32), np.zeros(C, np.float32), "f32", dev)
    assert errors(y0, x)[0] < 1e-6
    gt, gc = log_gains(N, C, seed=6)
    G = (np.exp(gt.astype(np.float64))[:, None] * np.exp(gc.astype(np.float64))[None, :])
    yj = run_gpu(x, G.astype(np.float32), "f32", dev)
    ys = run_gpu_separable(x, gt, gc, "f32", dev)
    assert errors(ys, yj)[0] < 2e-6


@pytest.mark.parametrize("K", [12, 13, 14, 15, 16])
def test_three_pass_matches_fused(K, dev, orc):
    """Slices that fit one workgroup, forced through the three-pass plan too."""
    N, C = 1 << (K - 6), 64
    x, g = workloads.draw(3, N, C, "f32", seed=K)
    say(f"K={K}: fused vs three_pass")
    ref = orc.whtmix(x, g)
    y_f = run_gpu(x, g, "f32", dev, plan="fused")
    y_3 = run_gpu(x, g, "f32", dev, plan="three_pass")
    check("fused", y_f, ref, "f32")
    check("three_pass", y_3, ref, "f32")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(2, 32, 16), (2, 64, 64), (2, 4096, 64)])
def test_in_place(shape, dtype, dev, orc):
    import torch
    B, N, C = shape
    x, g = workloads.draw(B, N, C, dtype, seed=5)
    xd = to_device(x, dtype, dev)
    gd = torch.from_numpy(g).to(dev)
    out = whtmix.forward(xd, gd, out=xd)
    torch.cuda.synchronize()
    assert out.data_ptr() == xd.data_ptr()
    check(f"in-place {shape}", to_host(xd), orc.whtmix(x, g), dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 32, 32), (2, 128, 64), (4, 65536, 128)])
def test_unit_gain_is_identity(shape, dtype, dev):
    """G = 1 (the paper's zero-initialised log gain) returns x.  For bf16 the
    float32 result differs from x by rounding errors of the order of
    1e-7 * max|x|; that is far below half a bf16 ulp of all but the smallest
    elements, so nearly every output rounds back to x exactly and none moves
    by more than one bf16 ulp of max|x| * 2^-8."""
    B, N, C = shape
    x, _ = workloads.draw(B, N, C, dtype, seed=21)
    y = run_gpu(x, np.ones((N, C), np.float32), dtype, dev)
    err = errors(y, x)[0]
    if dtype == "bf16":
        exact = float(np.mean(y == x))
        say(f"  bf16 identity: {exact:.5f} bit-exact, normwise-max {err:.2e}")
        assert exact > 0.99
        assert err <= 2.0 ** -8
    else:
        assert err < 1e-6


def test_deterministic_and_batch_independent(dev):
    import torch
    x, g = workloads.draw(4, 4096, 64, "f32", seed=3)
    xd = to_device(x, "f32", dev)
    gd = torch.from_numpy(g).to(dev)
    y1 = to_host(whtmix.forward(xd, gd))
    y2 = to_host(whtmix.forward(xd, gd))
    assert np.array_equal(y1, y2)
    for b in [0, 3]:
        yb = to_host(whtmix.forward(xd[b:b + 1].contiguous(), gd))
        assert np.array_equal(yb[0], y1[b])


@pytest.mark.parametrize("shape,dtype,nb", [
    ((2, 65536, 128), "bf16", 2), ((8, 65536, 128), "bf16", 8), ((32, 16384, 64), "f32", 4),
], ids=["2x2^23", "8x2^23", "32x2^20"])
def test_middle_slice_groups(shape, dtype, nb, dev, orc):
    """Batches whose middle pass runs nb slices per workgroup (the run's gain
    read once for the group): every sampled slice is bit-identical to a
    one-slice call (which takes nb = 1) and matches the oracle."""
    import torch
    from tests.test_tile_model import VB, middle_slices_per_group, three_pass_split
    B, N, C = shape
    K = (N * C).bit_length() - 1
    A, HB, R = three_pass_split(K)
    assert middle_slices_per_group(B, A - R, HB + R - VB) == nb
    assert whtmix.plan_describe(B, N, C, dtype)["plan"] == "three_pass"
    say(f"slice groups: B={B} N={N} C={C} {dtype} nb={nb}")
    x, g = workloads.draw(B, N, C, dtype, seed=41)
    xd = to_device(x, dtype, dev)
    gd = torch.from_numpy(g).to(dev)
    y = whtmix.forward(xd, gd)
    torch.cuda.synchronize(dev)
    for b in (0, nb - 1, B - 1):
        yb = whtmix.forward(xd[b:b + 1].contiguous(), gd)
        assert torch.equal(yb[0], y[b]), b
    yh = to_host(y)
    sample = [0, B - 1]
    check(f"slice groups {shape}", yh[sample], orc.whtmix(x[sample], g), dtype)


def test_bf16_round_to_nearest_even(dev):
    """N = C = 1 reduces the mixer to y = g x: products placed exactly on bf16
    halfway points must round to the even neighbour."""
    import torch
    xs = np.array([1.0, 1.0, -1.0, 2.0, 1.0], np.float32)
    gs = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8, 1 + 2 ** -9, 1 + 2 ** -8 + 2 ** -20],
                  np.float32)
    want = [1.0, 1 + 2 ** -6, -1.0, 2.0, 1 + 2 ** -7]
    for xv, gv, wv in zip(xs, gs, want):
        y = run_gpu(np.array([[[xv]]]), np.array([[gv]]), "bf16", dev)
        assert float(y.reshape(-1)[0]) == wv, (xv, gv, y, wv)
    del torch


def test_device_pointer_checks(dev):
    import torch
    x = torch.zeros(2, 64, 64, device=dev)
    g = torch.ones(64, 64, device=dev)
    y = torch.zeros(2, 64, 64, device=dev)
    s = torch.cuda.current_stream().cuda_stream
    assert whtmix.forward_raw(x.data_ptr() + 4, g.data_ptr(), y.data_ptr(), 1, 64, 64, 0, s) == 4
    assert whtmix.forward_raw(x.data_ptr(), g.data_ptr(), x.data_ptr() + 1024, 1, 64, 64, 0, s) == 1
    assert whtmix.forward_raw(x.data_ptr(), y.data_ptr(), y.data_ptr(), 1, 64, 64, 0, s) == 1
    assert whtmix.forward_raw(x.data_ptr(), g.data_ptr(), y.data_ptr(), 0, 64, 64, 0, s) == 0
    torch.cuda.synchronize()
    assert torch.count_nonzero(y).item() == 0


def test_workspace_growth_and_streams(dev, orc):
    """Growing the per-stream workspace, then shrinking the shape, on two
    streams whose work overlaps."""
    import torch
    cases = [(1, 4096, 64), (2, 16384, 128), (1, 2048, 64)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for i, (B, N, C) in enumerate(cases):
        x, g = workloads.draw(B, N, C, "f32", seed=40 + i)
        x2, g2 = workloads.draw(B, N, C, "f32", seed=50 + i)
        xd, gd = to_device(x, "f32", dev), torch.from_numpy(g).to(dev)
        xd2, gd2 = to_device(x2, "f32", dev), torch.from_numpy(g2).to(dev)
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            y1 = whtmix.forward(xd, gd)
        with torch.cuda.stream(s2):
            y2 = whtmix.forward(xd2, gd2)
        torch.cuda.synchronize()
        check(f"stream1 {(B, N, C)}", to_host(y1), orc.whtmix(x, g), "f32")
        check(f"stream2 {(B, N, C)}", to_host(y2), orc.whtmix(x2, g2), "f32")


@pytest.mark.parametrize("shape", [(1, 1 << 22, 256), (2, 1 << 20, 256)])
def test_large_slices_by_properties(shape, dev):
    """Up to the largest slice (N*C = 2^30), where the float64 oracle would be
    slow: unit gain returns x, a +/-1 gain preserves energy, and a one-hot
    gain at (2^p, 2^q) projects x on the Walsh image s_n s_c / sqrt(N C)
    with s_n = (-1)^(bit p of n), s_c = (-1)^(bit q of c)."""
    import torch
    B, N, C = shape
    say(f"large {shape}")
    gen = torch.Generator(device=dev).manual_seed(7)
    x = torch.randn(B, N, C, device=dev, generator=gen)
    ones = torch.ones(N, C, device=dev)
    y = whtmix.forward(x, ones)
    err = ((y - x).abs().max() / x.abs().max()).item()
    say(f"  unit gain err {err:.3e}")
    assert err < 1e-5
    del y
    sign = torch.where(torch.rand(N, C, device=dev, generator=gen) < 0.5, -1.0, 1.0)
    y = whtmix.forward(x, sign)
    r = (torch.linalg.vector_norm(y.double()) / torch.linalg.vector_norm(x.double())).item()
    say(f"  energy ratio {r:.9f}")
    assert abs(r - 1) < 1e-5
    del y, sign
    p, q = 17, 3
    n = torch.arange(N, device=dev)
    c = torch.arange(C, device=dev)
    sn = (1 - 2 * ((n >> p) & 1)).double()
    sc = (1 - 2 * ((c >> q) & 1)).double()
    g = torch.zeros(N, C, device=dev)
    g[1 << p, 1 << q] = 1.0
    y = whtmix.forward(x, g)
    scale = 1.0 / np.sqrt(float(N) * C)
    rows = 1 << 18
    for b in range(B):
        coef = 0.0
        for r0 in range(0, N, rows):
            xb = x[b, r0:r0 + rows].double()
            coef += float(torch.mv(xb.t().contiguous(), sn[r0:r0 + rows]).dot(sc))
        # error scale: the coefficient <x, B> has standard deviation rms(x)
        # (B has unit norm), so compare against max(|<x, B>|, rms(x))
        xrms = float(x[b].double().pow(2).mean().sqrt())
        amp = max(abs(coef) * scale, xrms) * scale
        worst = 0.0
        for r0 in range(0, N, rows):
            ref = (coef * scale * scale) * sn[r0:r0 + rows, None] * sc[None, :]
            worst = max(worst, (y[b, r0:r0 + rows].double() - ref).abs().max().item())
        say(f"  one-hot slice {b} err {worst / amp:.3e}")
        assert worst / amp < 1e-5
    torch.cuda.synchronize()
