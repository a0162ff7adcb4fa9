"""Parity of the whole block (section III-B, eqs. (1)-(4): Z = X W_in, the
mixer, Y = Z W_out) on the GPU, through the C ABI, with the CPU oracle.

Both sides get the same seeded inputs (workloads.draw / draw_weights; bf16
inputs are bf16 values).  The bar is the normwise maximum relative error
max|y - r| / max|r|: 1e-5 for float32 I/O; 4e-3 for bf16 I/O, derived from
the arithmetic: y is rounded to bf16 once (bf16 keeps 8 significant bits, so
the relative error is <= 2^-8 of each element and <= 2^-8 = 3.906e-3 of
max|r| normwise), the bf16 products X W_in are exact in float32, and the
two-term split of Z' before W_out leaves < 2^-17; float32 accumulation adds
~1e-6: 3.915e-3 in all.
"""
import numpy as np
import pytest

from oracle import oracle as oracle_mod
from paper_2607_25234_amd import whtmix, workloads
from tests.gpu_util import device, errors, say, to_device, to_host

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 4e-3}


@pytest.fixture(scope="module")
def dev():
    return device()


@pytest.fixture(scope="module")
def orc():
    return oracle_mod.Oracle()


def run_module(x, wi, wo, dtype, dev, g=None, gt=None, gc=None, plan="auto", inplace=False):
    import torch

    xd = to_device(x, dtype, dev)
    wid = to_device(wi, dtype, dev)
    wod = to_device(wo, dtype, dev)
    out = xd if inplace else None
    if g is not None:
        gd = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(dev)
        y = whtmix.module_forward(xd, wid, gd, wod, out=out, plan=plan)
    else:
        gtd = torch.from_numpy(np.ascontiguousarray(gt, dtype=np.float32)).to(dev)
        gcd = torch.from_numpy(np.ascontiguousarray(gc, dtype=np.float32)).to(dev)
        y = whtmix.module_forward_separable(xd, wid, gtd, gcd, wod, out=out, plan=plan)
    torch.cuda.synchronize(dev)
    return to_host(y)


def check(name, y, ref, dtype):
    err, rms = errors(y, ref)
    say(f"  {name}: normwise-max {err:.3e} rms {rms:.3e} (tol {TOL[dtype]:g})")
    assert y.shape == ref.shape
    assert np.all(np.isfinite(y))
    assert err <= TOL[dtype], (name, err)


def inputs(B, N, C, dtype, seed):
    P = whtmix.padded_tokens(N)
    x, _ = workloads.draw(B, N, C, dtype, seed=seed)
    _, g = workloads.draw(1, P, C, "f32", seed=seed + 1)
    wi, wo = workloads.draw_weights(C, dtype, seed=seed + 2)
    return x, g, wi, wo


def path(B, N, C, dtype, plan="auto"):
    d = whtmix.plan_describe(B, N, C, dtype, plan)
    if d["module_path"] == "small":
        return "small"
    return f"{d['module_path']}-{d['plan']}"


@pytest.mark.parametrize("name", list(workloads.WORKLOADS))
def test_module_workload(name, dev, orc):
    """Every workload's shape through the block, in the plan the benchmark
    runs; the oracle checks a few whole slices (each slice is independent)."""
    w = workloads.WORKLOADS[name]
    x, g = workloads.inputs(w)
    wi, wo = workloads.draw_weights(w.C, w.dtype, seed=w.seed + 50)
    say(f"module workload {name}: B={w.B} N={w.N} C={w.C} {w.dtype} "
        f"{path(w.B, w.N, w.C, w.dtype)}")
    y = run_module(x, wi, wo, w.dtype, dev, g=g)
    for b in sorted({0, w.B // 2, w.B - 1}):
        check(f"{name}[{b}]", y[b], orc.whtmix_module(x[b], wi, g, wo), w.dtype)


SHAPES = [
    # SMALL (N_pad*C <= 2^10): projections on the VALU, any C
    (1, 1, 1), (2, 3, 4), (3, 8, 16), (2, 16, 64), (1, 4, 256),
    # FUSED with MFMA projections: C in [16, 128], 2^11..2^15, padded N too
    (2, 128, 16), (3, 100, 32), (1, 64, 64), (2, 50, 64), (2, 256, 128), (1, 1000, 32),
    (1, 2048, 16),
    # THREE_PASS with MFMA projections
    (2, 4096, 16), (1, 3000, 32), (2, 2048, 128), (1, 9216, 64), (1, 8192, 128),
    (1, 1 << 15, 32),
    # C = 256: bf16 THREE_PASS on 2^16 outer tiles (ragged and wholly padded
    # tiles included); float32 and the FUSED plan UNFUSED
    (1, 512, 256), (2, 700, 256), (1, 4096, 256), (1, 9216, 256),
    # UNFUSED: C outside [16, 128] (matrix-core projections from C = 256; VALU below 16
    # and for float32 C = 4096, whose weight slice does not fit LDS)
    (2, 512, 8), (1, 64, 256), (3, 1000, 256), (1, 8, 512), (1, 3, 1024), (1, 16, 2048),
    (1, 4, 4096),
]



@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_module_shapes(shape, dtype, dev, orc):
    B, N, C = shape
    x, g, wi, wo = inputs(B, N, C, dtype, seed=500 + N + 7 * C + B)
    say(f"module {shape} {dtype} {path(B, N, C, dtype)}")
    y = run_module(x, wi, wo, dtype, dev, g=g)
    check(f"{shape}", y, orc.whtmix_module(x, wi, g, wo), dtype)


FORCED = [(2, 128, 32), (1, 256, 64), (1, 100, 128), (2, 256, 128), (3, 1024, 16)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", FORCED, ids=lambda s: "x".join(map(str, s)))
def test_module_forced_three_pass(shape, dtype, dev, orc):
    """Slices of 2^12..2^15 through the three-pass kernels (every outer tile
    size and split class of the forced plan)."""
    B, N, C = shape
    x, g, wi, wo = inputs(B, N, C, dtype, seed=600 + N + C)
    say(f"module forced three_pass {shape} {dtype}")
    y = run_module(x, wi, wo, dtype, dev, g=g, plan="three_pass")
    check(f"{shape} three_pass", y, orc.whtmix_module(x, wi, g, wo), dtype)


SEPARABLE = [(2, 16, 32), (2, 200, 64), (1, 4096, 128), (2, 9216, 64), (1, 100, 256),
             (1, 2000, 256)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SEPARABLE, ids=lambda s: "x".join(map(str, s)))
def test_module_separable(shape, dtype, dev, orc):
    """The paper's literal parametrisation: log gains g_t, g_c."""
    B, N, C = shape
    x, _, wi, wo = inputs(B, N, C, dtype, seed=700 + N + C)
    gt, gc = workloads.draw_log_gains(whtmix.padded_tokens(N), C, seed=701 + N)
    say(f"module separable {shape} {dtype} {path(B, N, C, dtype)}")
    y = run_module(x, wi, wo, dtype, dev, gt=gt, gc=gc)
    check(f"separable {shape}", y, orc.whtmix_module_separable(x, wi, gt, gc, wo), dtype)


def test_module_separable_workload(dev, orc):
    w = workloads.WORKLOADS[workloads.BENCH_WORKLOAD]
    x, _ = workloads.inputs(w)
    wi, wo = workloads.draw_weights(w.C, w.dtype, seed=w.seed + 50)
    gt, gc = workloads.draw_log_gains(w.N, w.C, seed=77)
    y = run_module(x, wi, wo, w.dtype, dev, gt=gt, gc=gc)
    for b in (0, w.B - 1):
        check(f"separable {w.name}[{b}]", y[b],
              orc.whtmix_module_separable(x[b], wi, gt, gc, wo), w.dtype)


@pytest.mark.parametrize("shape,plan", [((2, 16, 64), "auto"), ((2, 100, 64), "auto"),
                                        ((1, 4096, 128), "auto"), ((2, 128, 32), "three_pass"),
                                        ((1, 512, 8), "auto"), ((1, 1000, 256), "auto")])
def test_module_in_place(shape, plan, dev, orc):
    """y may be x itself (every path reads all of its x before writing y)."""
    B, N, C = shape
    x, g, wi, wo = inputs(B, N, C, "bf16", seed=800 + N)
    y = run_module(x, wi, wo, "bf16", dev, g=g, plan=plan, inplace=True)
    check(f"in place {shape}", y, orc.whtmix_module(x, wi, g, wo), "bf16")


def test_module_identity_weights_reduce_to_the_mixer(dev):
    """W_in = W_out = I gives the mixer alone (eqs. (2)-(3))."""
    import torch

    B, N, C = 2, 8192, 64
    x, g = workloads.draw(B, N, C, "f32", seed=9)
    eye = np.eye(C, dtype=np.float32)
    y = run_module(x, eye, eye, "f32", dev, g=g)
    xd = to_device(x, "f32", dev)
    gd = torch.from_numpy(g).to(dev)
    ym = to_host(whtmix.forward(xd, gd))
    assert errors(y, ym)[0] < 1e-6


@pytest.mark.parametrize("shape", [(1, 1 << 19, 256), (1, 139872, 256), (3, 32768, 256),
                                   (5, 20000, 256)],
                         ids=lambda s: "x".join(map(str, s)))
def test_module_c256_large_identity_weights(shape, dev):
    """bf16 C = 256 at 2^27 elements (runs of 16 floats, renumbered outer
    blocks) and at 2^26 with padding; 3 and 5 slices of 2^23 (384 and 640
    outer tiles over the inverse pass's 256 persistent workgroups, so some
    take one tile more than others; the 5 slices padded, with wholly padded
    tiles stepped over): W_in = W_out = I gives the mixer alone.
    Each output is the nearest bf16 of a float32 value, and the two float32
    values differ by rounding only, so an element may differ by one bf16 ulp
    (2^-7 of its magnitude at most): the bar is 2^-7 normwise."""
    import torch

    B, N, C = shape
    d = whtmix.plan_describe(B, N, C, "bf16")
    assert (d["module_path"], d["module_outer_bits"]) == ("mfma", 16)
    gen = torch.Generator(device="cpu").manual_seed(N)
    x = torch.randn(B, N, C, generator=gen).to(dev).to(torch.bfloat16)
    P = whtmix.padded_tokens(N)
    g = (torch.rand(P, C, generator=gen) + 0.5).to(dev)
    eye = torch.eye(C, device=dev, dtype=torch.bfloat16)
    say(f"module identity {shape} bf16")
    y = whtmix.module_forward(x, eye, g, eye)
    ym = whtmix.forward(x, g)
    torch.cuda.synchronize(dev)
    err, rms = errors(to_host(y), to_host(ym))
    say(f"  normwise-max {err:.3e} rms {rms:.3e}")
    assert err <= 2.0 ** -7 and rms < 1e-3, (err, rms)


def test_module_deterministic(dev):
    B, N, C = 4, 16384, 128
    x, g, wi, wo = inputs(B, N, C, "bf16", seed=31)
    a = run_module(x, wi, wo, "bf16", dev, g=g)
    b = run_module(x, wi, wo, "bf16", dev, g=g)
    assert np.array_equal(a, b)
