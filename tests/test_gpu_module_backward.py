"""Gradients of the whole block (eqs. (1)-(4)) on the GPU, through the C ABI,
against the oracle's (oracle_whtmix_module_grad, float64).

dX is held to the block's forward bar for its dtype (1e-5 float32 I/O, 4e-3
bf16 I/O: one RNE of dX, exact bf16 products, the 2^-17 split before W_in^T).
The weight and gain gradients are float32 outputs computed in float32 from
exactly representable inputs, held to 1e-5 normwise as the mixer's gain
gradient is.
"""
import numpy as np
import pytest

from oracle import oracle as oracle_mod
from paper_2607_25234_amd import whtmix, workloads
from tests.gpu_util import device, errors, say, to_device, to_host

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 4e-3}
GRAD_TOL = 1e-5


@pytest.fixture(scope="module")
def dev():
    return device()


@pytest.fixture(scope="module")
def orc():
    return oracle_mod.Oracle()


def check(name, y, ref, tol):
    err, rms = errors(y, ref)
    say(f"  {name}: normwise-max {err:.3e} rms {rms:.3e} (tol {tol:g})")
    assert y.shape == ref.shape
    assert np.all(np.isfinite(y))
    assert err <= tol, (name, err)


def inputs(B, N, C, dtype, seed):
    P = whtmix.padded_tokens(N)
    x, _ = workloads.draw(B, N, C, dtype, seed=seed)
    dy, _ = workloads.draw(B, N, C, dtype, seed=seed + 1)
    _, g = workloads.draw(1, P, C, "f32", seed=seed + 2)
    wi, wo = workloads.draw_weights(C, dtype, seed=seed + 3)
    return x, dy, g, wi, wo


def run(x, dy, wi, wo, dtype, dev, g=None, gt=None, gc=None, plan="auto", alias=False):
    import torch

    xd, dyd = to_device(x, dtype, dev), to_device(dy, dtype, dev)
    wid, wod = to_device(wi, dtype, dev), to_device(wo, dtype, dev)
    dx = dyd if alias else None
    if g is not None:
        gd = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(dev)
        out = whtmix.module_backward(xd, wid, gd, wod, dyd, dx=dx, plan=plan)
    else:
        gtd = torch.from_numpy(np.ascontiguousarray(gt, dtype=np.float32)).to(dev)
        gcd = torch.from_numpy(np.ascontiguousarray(gc, dtype=np.float32)).to(dev)
        out = whtmix.module_backward_separable(xd, wid, gtd, gcd, wod, dyd, dx=dx, plan=plan)
    torch.cuda.synchronize(dev)
    return [to_host(t) for t in out]


def check_all(tag, got, ref, dtype):
    names = ["dx", "dw_in", "dw_out"] + (["dgain"] if len(ref) == 4 else ["dgt", "dgc"])
    for name, a, r in zip(names, got, ref):
        check(f"{tag} {name}", a, r, TOL[dtype] if name == "dx" else GRAD_TOL)


SHAPES = [
    # (B, N, C): VALU projections below C = 32, matrix cores from 32; SMALL,
    # FUSED and THREE_PASS mixers; padded token counts
    (2, 3, 4), (3, 50, 8), (2, 64, 16), (1, 100, 32), (2, 64, 64), (2, 512, 128),
    (1, 3000, 32), (2, 2048, 64), (1, 1024, 128), (1, 64, 256), (2, 300, 256),
    # bf16 32 <= C <= 128 three-pass: projections inside the backward's passes
    (3, 5000, 64), (2, 20000, 32),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_module_backward_shapes(shape, dtype, dev, orc):
    B, N, C = shape
    x, dy, g, wi, wo = inputs(B, N, C, dtype, seed=900 + N + 3 * C + B)
    say(f"module backward {shape} {dtype} plan={whtmix.plan_describe(B, N, C, dtype)['plan']}")
    got = run(x, dy, wi, wo, dtype, dev, g=g)
    check_all(f"{shape}", got, orc.whtmix_module_grad(x, wi, g, wo, dy), dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(2, 100, 64), (1, 4096, 128), (2, 16, 8)],
                         ids=lambda s: "x".join(map(str, s)))
def test_module_backward_separable(shape, dtype, dev, orc):
    B, N, C = shape
    x, dy, _, wi, wo = inputs(B, N, C, dtype, seed=950 + N)
    gt, gc = workloads.draw_log_gains(whtmix.padded_tokens(N), C, seed=951 + N)
    got = run(x, dy, wi, wo, dtype, dev, gt=gt, gc=gc)
    check_all(f"separable {shape}", got,
              orc.whtmix_module_grad_separable(x, wi, gt, gc, wo, dy), dtype)


def test_module_backward_workload_slice(dev, orc):
    """One slice of the benchmarked shape (N = 65536, C = 128, bf16)."""
    w = workloads.WORKLOADS[workloads.BENCH_WORKLOAD]
    x, dy, g, wi, wo = inputs(1, w.N, w.C, w.dtype, seed=77)
    got = run(x, dy, wi, wo, w.dtype, dev, g=g)
    check_all("stereo64k slice", got, orc.whtmix_module_grad(x, wi, g, wo, dy), w.dtype)


def test_module_backward_c256_pair_tiles_against_oracle(dev, orc):
    """One 2^26-element slice (N = 262144, C = 256, bf16): the fused pair-tile
    block backward (2^16-element outer tiles with the projections inside the
    passes) against oracle_whtmix_module_grad in float64 (about a minute of
    host time on every core)."""
    B, N, C = 1, 262144, 256
    d = whtmix.plan_describe(B, N, C, "bf16")
    assert d["module_backward_fused"] and d["module_outer_bits"] == 16, d
    x, dy, g, wi, wo = inputs(B, N, C, "bf16", seed=260)
    say(f"module backward {(B, N, C)} bf16 pair tiles: GPU, then the oracle "
        f"on {orc.threads()} threads")
    got = run(x, dy, wi, wo, "bf16", dev, g=g)
    ref = orc.whtmix_module_grad(x, wi, g, wo, dy)
    check_all("2^26 pair tiles", got, ref, "bf16")


def test_module_backward_separable_pair_tiles_by_joint_gain(dev):
    """One 2^26-element slice (N = 140000 padded, C = 256, bf16): the pair-tile
    block backward with separable gains, whose middle pass forms the log-gain
    sums itself (one slice per chunk, 2^15-element tiles), against the same
    call with the joint gain G = exp(g_t + g_c) (its dG checked against the
    oracle above): dX and both weight gradients agree, and the log-gain
    gradients equal the row and column sums of dG * G taken on the host."""
    B, N, C = 1, 140000, 256
    P = whtmix.padded_tokens(N)
    d = whtmix.plan_describe(B, N, C, "bf16")
    assert d["module_backward_fused"] and d["module_outer_bits"] == 16, d
    x, dy, _, wi, wo = inputs(B, N, C, "bf16", seed=970)
    gt, gc = workloads.draw_log_gains(P, C, seed=971)
    G = np.exp(gt.astype(np.float64)[:, None] + gc.astype(np.float64)[None, :])
    say(f"module backward separable {(B, N, C)} bf16 against the joint gain")
    dx_s, dwi_s, dwo_s, dgt, dgc = run(x, dy, wi, wo, "bf16", dev, gt=gt, gc=gc)
    dx_j, dwi_j, dwo_j, dg = run(x, dy, wi, wo, "bf16", dev, g=G.astype(np.float32))
    # two bf16 roundings of float32 values that agree to about 1e-7 differ by
    # at most one bf16 ulp, 2^-7 of the element at most (not the 2^-8 of one
    # rounding against the exact value)
    check("dx", dx_s, dx_j, 2.0 ** -7 + GRAD_TOL)
    check("dw_in", dwi_s, dwi_j, GRAD_TOL)
    check("dw_out", dwo_s, dwo_j, GRAD_TOL)
    dgg = dg.astype(np.float64).reshape(P, C) * G
    check("dgt", dgt, dgg.sum(axis=1), GRAD_TOL)
    check("dgc", dgc, dgg.sum(axis=0), GRAD_TOL)


def test_module_backward_forced_three_pass_and_alias(dev, orc):
    """The three-pass mixer on a 2^14 slice, with dx written over dy."""
    B, N, C = 2, 128, 128
    x, dy, g, wi, wo = inputs(B, N, C, "bf16", seed=33)
    ref = orc.whtmix_module_grad(x, wi, g, wo, dy)
    check_all("three_pass alias", run(x, dy, wi, wo, "bf16", dev, g=g, plan="three_pass",
                                      alias=True), ref, "bf16")


@pytest.mark.parametrize("shape,dtype", [((1, 140000, 256), "bf16"), ((2, 262144, 256), "bf16"),
                                         ((4, 65536, 128), "bf16"), ((2, 16384, 128), "f32"),
                                         ((32, 4096, 64), "f32"), ((1, 65536, 16), "bf16")],
                         ids=lambda s: "x".join(map(str, s)) if isinstance(s, tuple) else s)
def test_module_backward_by_composition(shape, dtype, dev):
    """Shapes whose oracle takes minutes (2^26-element slices), through the
    projections-inside-the-passes backward, against the chain rule composed
    from the validated mixer (forward, and backward for dgain) and float32
    matrix products on the same device:
        Z = X W_in, Z' = mixer(Z), dZ' = dY W_out^T, dZ = mixer(dZ') (the
        mixer is self-adjoint), dX = dZ W_in^T, dW_in = X^T dZ, dW_out = Z'^T dY.
    Both sides are float32 up to rounding order (the weight gradients' three-
    term split leaves 2^-27), so the float32 bar holds for the float32
    outputs; dX in bf16 is rounded once."""
    import torch

    B, N, C = shape
    d = whtmix.plan_describe(B, N, C, dtype)
    assert d["module_backward_fused"], d
    gen = torch.Generator(device="cpu").manual_seed(N + C)
    P = whtmix.padded_tokens(N)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x = torch.randn(B, N, C, generator=gen).to(dev).to(tdt)
    dy = torch.randn(B, N, C, generator=gen).to(dev).to(tdt)
    wi = (torch.randn(C, C, generator=gen) / C ** 0.5).to(dev).to(tdt)
    wo = (torch.randn(C, C, generator=gen) / C ** 0.5).to(dev).to(tdt)
    g = (torch.rand(P, C, generator=gen) + 0.5).to(dev)
    say(f"module backward by composition {shape} {dtype}")
    torch.backends.cuda.matmul.allow_tf32 = False   # float32 products in float32
    dx, dwi, dwo, dg = whtmix.module_backward(x, wi, g, wo, dy)
    xf, dyf, wif, wof = x.float(), dy.float(), wi.float(), wo.float()
    z = torch.matmul(xf, wif)
    zp = whtmix.forward(z, g)
    dzp = torch.matmul(dyf, wof.t().contiguous())
    dz = whtmix.forward(dzp, g)
    _, dg_ref = whtmix.backward(z, dzp, g, want_dx=False)
    dx_ref = torch.matmul(dz, wif.t().contiguous())
    dwi_ref = torch.matmul(xf.reshape(-1, C).t().contiguous(), dz.reshape(-1, C))
    dwo_ref = torch.matmul(zp.reshape(-1, C).t().contiguous(), dyf.reshape(-1, C))
    torch.cuda.synchronize(dev)
    check("dx", to_host(dx), to_host(dx_ref), TOL[dtype])
    for name, a, r in [("dw_in", dwi, dwi_ref), ("dw_out", dwo, dwo_ref), ("dgain", dg, dg_ref)]:
        check(name, to_host(a), to_host(r), GRAD_TOL)


def test_module_backward_empty_batch_zeroes_gradients(dev):
    import torch

    C, N = 64, 100
    P = whtmix.padded_tokens(N)
    empty = torch.empty((0, N, C), device=dev)
    wi = torch.randn(C, C, device=dev)
    wo = torch.randn(C, C, device=dev)
    g = torch.rand(P, C, device=dev) + 0.5
    dx, dwi, dwo, dg = whtmix.module_backward(empty, wi, g, wo, empty)
    torch.cuda.synchronize(dev)
    assert dx.shape == (0, N, C)
    for t in (dwi, dwo, dg):
        assert torch.count_nonzero(t).item() == 0


def test_module_backward_deterministic(dev):
    B, N, C = 4, 16384, 128
    x, dy, g, wi, wo = inputs(B, N, C, "bf16", seed=41)
    a = run(x, dy, wi, wo, "bf16", dev, g=g)
    b = run(x, dy, wi, wo, "bf16", dev, g=g)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


def test_block_autograd_training_step(dev, orc):
    """torch.autograd through whtmix_block: gradients of a scalar loss reach x,
    both weights and the gain, and match the oracle's."""
    import torch

    from paper_2607_25234_amd.autograd import whtmix_block

    B, N, C = 2, 1000, 64
    x, dy, g, wi, wo = inputs(B, N, C, "f32", seed=51)
    xt = torch.from_numpy(x).to(dev).requires_grad_(True)
    wit = torch.from_numpy(wi).to(dev).requires_grad_(True)
    wot = torch.from_numpy(wo).to(dev).requires_grad_(True)
    gt_ = torch.from_numpy(g).to(dev).requires_grad_(True)
    y = whtmix_block(xt, wit, gt_, wot)
    loss = (y * torch.from_numpy(dy).to(dev)).sum()
    loss.backward()
    torch.cuda.synchronize(dev)
    ref = orc.whtmix_module_grad(x, wi, g, wo, dy)
    for name, t, r in zip(["dx", "dw_in", "dw_out", "dgain"], [xt, wit, wot, gt_],
                          [ref[0], ref[1], ref[2], ref[3]]):
        check(f"autograd {name}", to_host(t.grad), r, GRAD_TOL)
