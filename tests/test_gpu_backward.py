"""Parity of the HIP backward pass (through the C ABI) with the CPU oracle.

dX uses the forward tolerance of its dtype; the gain gradients are float32
outputs computed from exactly representable inputs, held to 1e-5 normwise
maximum relative error for both dtypes.
"""
import numpy as np
import pytest

from oracle import oracle as oracle_mod
from paper_2607_25234_amd import whtmix, workloads
from tests.gpu_util import (DERIVED, TOL, case_ids, device, errors, random_cases, say,
                            to_device, to_host)

pytestmark = pytest.mark.gpu

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
    dy, g = workloads.draw(B, N, C, dtype, seed=seed + 1)
    if P != N:
        _, g = workloads.draw(1, P, C, "f32", seed=seed + 2)
    return x, dy, g


# Three-pass shapes cover one slice per chunk with chunk sums (2x4096x64,
# 2x9216x64), several slices per chunk (6x8192x32) and a short last chunk
# (7x8192x32: chunks of 2, 2, 2, 1); 5x1x2 sums chunks of a 2-element slice.
SHAPES = [(1, 1, 1), (5, 1, 2), (3, 32, 32), (3000, 16, 16), (2, 64, 64), (40, 128, 128), (5, 1000, 16),
          (2, 4096, 64), (2, 9216, 64), (6, 8192, 32), (7, 8192, 32), (1, 4096, 64), (1, 9000, 128)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_backward(shape, dtype, dev, orc):
    import torch
    B, N, C = shape
    x, dy, g = inputs(B, N, C, dtype, seed=500 + N + B)
    plan = whtmix.plan_describe(B, N, C, dtype)["plan"]
    say(f"backward {shape} {dtype} plan={plan}")
    dx, dg = whtmix.backward(to_device(x, dtype, dev), to_device(dy, dtype, dev),
                             torch.from_numpy(g).to(dev))
    torch.cuda.synchronize()
    dx_ref, dg_ref = orc.whtmix_grad(x, dy, g)
    check("dx", to_host(dx), dx_ref, DERIVED[dtype])
    check("dgain", to_host(dg), dg_ref, GRAD_TOL)


def test_backward_workload(dev, orc):
    """The benchmarked workload shape (B=4, N=65536, C=128, bf16)."""
    import torch
    w = workloads.WORKLOADS[workloads.BENCH_WORKLOAD]
    x, g = workloads.inputs(w)
    dy, _ = workloads.draw(w.B, w.N, w.C, w.dtype, seed=91)
    dx, dg = whtmix.backward(to_device(x, w.dtype, dev), to_device(dy, w.dtype, dev),
                             torch.from_numpy(g).to(dev))
    torch.cuda.synchronize()
    dx_ref, dg_ref = orc.whtmix_grad(x, dy, g)
    check("dx", to_host(dx), dx_ref, DERIVED[w.dtype])
    check("dgain", to_host(dg), dg_ref, GRAD_TOL)


def test_backward_largest_tiles(dev, orc):
    """A slice of 2^26 (N = 140000 padded to 2^18, C = 256): 2^16-element
    outer tiles (the straddling one with its second register set partly valid) and
    2^15-element middle tiles, whose gradient kernel stores each slice's
    product as soon as it is formed."""
    import torch
    B, N, C, dtype = 1, 140000, 256, "bf16"
    x, dy, g = inputs(B, N, C, dtype, seed=950)
    info = whtmix.plan_describe(B, N, C, dtype)
    assert info["outer_bits"] == 16
    assert info["log2_slice"] - info["outer_bits"] + info["run_bits"] == 15
    dx, dg = whtmix.backward(to_device(x, dtype, dev), to_device(dy, dtype, dev),
                             torch.from_numpy(g).to(dev))
    torch.cuda.synchronize()
    dx_ref, dg_ref = orc.whtmix_grad(x, dy, g)
    check("dx", to_host(dx), dx_ref, DERIVED[dtype])
    check("dgain", to_host(dg), dg_ref, GRAD_TOL)


BACKWARD_CASES = random_cases(24, 2609)


@pytest.mark.parametrize("case", BACKWARD_CASES, ids=case_ids(BACKWARD_CASES))
def test_random_shapes_backward(case, dev, orc):
    """dX and dG on seeded shapes (every plan's range, padded token counts),
    and the separable log-gain gradients on the same inputs."""
    import torch
    B, N, C, dtype = case
    P = whtmix.padded_tokens(N)
    x, dy, g = inputs(B, N, C, dtype, seed=7000 + 7 * N + C + B)
    say(f"random backward {case} plan={whtmix.plan_describe(B, N, C, dtype)['plan']}")
    xd, dyd = to_device(x, dtype, dev), to_device(dy, dtype, dev)
    dx, dg = whtmix.backward(xd, dyd, torch.from_numpy(g).to(dev))
    torch.cuda.synchronize()
    dx_ref, dg_ref = orc.whtmix_grad(x, dy, g)
    check("dx", to_host(dx), dx_ref, DERIVED[dtype])
    check("dgain", to_host(dg), dg_ref, GRAD_TOL)
    gt, gc = workloads.draw_log_gains(P, C, seed=7001 + N)
    dx, dgt, dgc = whtmix.backward_separable(xd, dyd, torch.from_numpy(gt).to(dev),
                                             torch.from_numpy(gc).to(dev))
    torch.cuda.synchronize()
    dx_ref, dgt_ref, dgc_ref = orc.whtmix_grad_separable(x, dy, gt, gc)
    check("dx (separable)", to_host(dx), dx_ref, DERIVED[dtype])
    check("d log_gain_tokens", to_host(dgt), dgt_ref, GRAD_TOL)
    check("d log_gain_channels", to_host(dgc), dgc_ref, GRAD_TOL)


@pytest.mark.parametrize("shape", [(2, 32, 32), (3, 1000, 16), (2, 4096, 64), (4, 9216, 64)],
                         ids=lambda s: "x".join(map(str, s)))
def test_backward_separable(shape, dev, orc):
    import torch
    B, N, C = shape
    P = whtmix.padded_tokens(N)
    x, dy, _ = inputs(B, N, C, "f32", seed=600 + N)
    gt, gc = workloads.draw_log_gains(P, C, seed=601 + N)
    dx, dgt, dgc = whtmix.backward_separable(
        to_device(x, "f32", dev), to_device(dy, "f32", dev), torch.from_numpy(gt).to(dev),
        torch.from_numpy(gc).to(dev))
    torch.cuda.synchronize()
    dx_ref, dgt_ref, dgc_ref = orc.whtmix_grad_separable(x, dy, gt, gc)
    check("dx", to_host(dx), dx_ref, TOL["f32"])
    check("d log_gain_tokens", to_host(dgt), dgt_ref, GRAD_TOL)
    check("d log_gain_channels", to_host(dgc), dgc_ref, GRAD_TOL)


@pytest.mark.parametrize("shape,dtype", [
    ((1, 8192, 128), "bf16"), ((6, 4096, 64), "f32"), ((2, 16384, 256), "bf16"),
    ((3, 4096, 32), "f32"), ((2, 6000, 64), "f32"), ((4, 65536, 128), "bf16"),
    ((1, 140000, 256), "bf16"), ((2, 65536, 512), "bf16"),
], ids=lambda v: "x".join(map(str, v)) if isinstance(v, tuple) else v)
def test_backward_separable_fused_sums(shape, dtype, dev, orc):
    """Shapes where the middle pass forms the log-gain gradients' partial sums
    itself (three-pass split with R = 5 and 6..10 high bits, 32 <= C <= 2^A):
    one slice (a chunk of one), three chunks of two slices, C = 256 (eight
    channel groups), C = 32 (one), padded N, the benchmarked workload, and
    2^15-element middle tiles (one slice per chunk, the exp factors applied to
    the row and column sums) at 2^26 padded and at 2^25 x 2 with C = 512."""
    import torch
    B, N, C = shape
    P = whtmix.padded_tokens(N)
    info = whtmix.plan_describe(B, N, C, dtype)
    assert info["plan"] == "three_pass" and info["run_bits"] == 5
    assert 6 <= info["log2_slice"] - info["outer_bits"] <= 10
    x, dy, _ = inputs(B, N, C, dtype, seed=640 + N + C)
    gt, gc = workloads.draw_log_gains(P, C, seed=641 + N + C)
    say(f"separable fused sums {shape} {dtype}")
    dx, dgt, dgc = whtmix.backward_separable(
        to_device(x, dtype, dev), to_device(dy, dtype, dev), torch.from_numpy(gt).to(dev),
        torch.from_numpy(gc).to(dev))
    torch.cuda.synchronize()
    dx_ref, dgt_ref, dgc_ref = orc.whtmix_grad_separable(x, dy, gt, gc)
    check("dx", to_host(dx), dx_ref, DERIVED[dtype])
    check("d log_gain_tokens", to_host(dgt), dgt_ref, GRAD_TOL)
    check("d log_gain_channels", to_host(dgc), dgc_ref, GRAD_TOL)


def test_backward_in_place_and_deterministic(dev, orc):
    """dx may overwrite dy (the gain gradient is taken first); repeated calls
    are bitwise identical (fixed-order batch sum)."""
    import torch
    B, N, C = 24, 2048, 64
    x, dy, g = inputs(B, N, C, "f32", seed=700)
    xd, gd = to_device(x, "f32", dev), torch.from_numpy(g).to(dev)
    _, dg1 = whtmix.backward(xd, to_device(dy, "f32", dev), gd, want_dx=False)
    _, dg2 = whtmix.backward(xd, to_device(dy, "f32", dev), gd, want_dx=False)
    torch.cuda.synchronize()
    assert torch.equal(dg1, dg2)
    dyd = to_device(dy, "f32", dev)
    dx, dg = whtmix.backward(xd, dyd, gd, dx=dyd)
    torch.cuda.synchronize()
    assert dx.data_ptr() == dyd.data_ptr()
    dx_ref, dg_ref = orc.whtmix_grad(x, dy, g)
    check("in-place dx", to_host(dx), dx_ref, TOL["f32"])
    check("dgain", to_host(dg), dg_ref, GRAD_TOL)
    assert torch.equal(dg, dg1)


def test_backward_empty_batch_zeroes_the_gain_gradient(dev):
    import torch
    g = torch.ones(64, 64, device=dev)
    dg = torch.full((64, 64), 7.0, device=dev)
    s = torch.cuda.current_stream().cuda_stream
    assert whtmix.backward_raw(0, 0, g.data_ptr(), 0, dg.data_ptr(), 0, 64, 64, 0, s) == 0
    torch.cuda.synchronize()
    assert torch.count_nonzero(dg).item() == 0


def test_autograd_training_step(dev, orc):
    """torch.autograd through the HIP forward/backward (the paper trains the
    gains): gradients of L = sum(y * w) match the oracle's."""
    import torch
    from paper_2607_25234_amd.autograd import whtmix_mix, whtmix_mix_separable
    B, N, C = 2, 1500, 32
    P = whtmix.padded_tokens(N)
    x, w, g = inputs(B, N, C, "f32", seed=800)
    xt = torch.from_numpy(x).to(dev).requires_grad_(True)
    gt_ = torch.from_numpy(g).to(dev).requires_grad_(True)
    loss = (whtmix_mix(xt, gt_) * torch.from_numpy(w).to(dev)).sum()
    loss.backward()
    dx_ref, dg_ref = orc.whtmix_grad(x, w, g)
    check("x.grad", to_host(xt.grad), dx_ref, TOL["f32"])
    check("gain.grad", to_host(gt_.grad), dg_ref, GRAD_TOL)
    lt, lc = workloads.draw_log_gains(P, C, seed=801)
    xt.grad = None
    ltt = torch.from_numpy(lt).to(dev).requires_grad_(True)
    lct = torch.from_numpy(lc).to(dev).requires_grad_(True)
    loss = (whtmix_mix_separable(xt, ltt, lct) * torch.from_numpy(w).to(dev)).sum()
    loss.backward()
    dx_ref, dgt_ref, dgc_ref = orc.whtmix_grad_separable(x, w, lt, lc)
    check("x.grad (separable)", to_host(xt.grad), dx_ref, TOL["f32"])
    check("log_gain_tokens.grad", to_host(ltt.grad), dgt_ref, GRAD_TOL)
    check("log_gain_channels.grad", to_host(lct.grad), dgc_ref, GRAD_TOL)
