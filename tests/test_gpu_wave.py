"""The wave-tile plans (csrc/whtmix_wave.hip) against the CPU oracle, through
the C ABI.

Both run the mixer (section III-B, eqs. (2)-(3)) as three passes on one-wave
2^9-element tiles whose butterflies stay in the wave: WAVE_TILES as three
launches, ONE_LAUNCH in one cooperative launch ordered by per-slice counters.
TWO_PASS (2^15- and 2^16-element slices) replaces the first two passes by a
fold pass whose workgroups each read the whole slice.
Checked here: parity at every supported slice size, batch counts from 1 to
2046 (several tiles per workgroup when a single launch outgrows the resident
grid), padded N, both dtypes, both gain forms, in place; back-to-back calls
(the single launch returns its counters to zero); and the give-up path forced
from the host with a poll limit of one, after which the stream reports the
error once and later calls are correct.
"""
import numpy as np
import pytest

from oracle import oracle as oracle_mod
from paper_2607_25234_amd import whtmix, workloads
from tests.gpu_util import (DERIVED, TOL, device, errors, run_gpu, run_gpu_separable, say,
                            to_device, to_host)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return device()


@pytest.fixture(scope="module")
def orc():
    return oracle_mod.Oracle()


def check(name, y, ref, dtype):
    err, rms = errors(y, ref)
    say(f"  {name}: normwise-max {err:.3e} rms {rms:.3e}")
    assert y.shape == ref.shape and np.all(np.isfinite(y))
    assert err <= TOL[dtype] and err <= DERIVED[dtype], (name, err)


def status_ok():
    st = whtmix.stream_status()
    assert st == whtmix.SUCCESS, whtmix.status_string(st)


PLANS = ["one_launch", "wave_tiles"]


@pytest.mark.parametrize("plan", PLANS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 64, 64), (2, 128, 64), (1, 256, 64), (3, 256, 128),
                                   (1, 1024, 64), (2, 512, 128), (16, 1024, 64),
                                   (47, 512, 128), (1, 65536, 1), (1, 8, 8192),
                                   (300, 1024, 64), (2046, 64, 64)],
                         ids=lambda s: "x".join(map(str, s)))
def test_parity(shape, dtype, plan, dev, orc):
    B, N, C = shape
    say(f"{plan} B={B} N={N} C={C} {dtype}")
    x, g = workloads.draw(B, N, C, dtype, seed=B * 1000 + N + C)
    y = run_gpu(x, g, dtype, dev, plan=plan)
    status_ok()
    check(plan, y, orc.whtmix(x, g), dtype)


@pytest.mark.parametrize("plan", PLANS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 1000, 64), (2, 9, 512), (3, 200, 128), (1, 33, 128)],
                         ids=lambda s: "x".join(map(str, s)))
def test_padded_tokens(shape, dtype, plan, dev, orc):
    """Non-power-of-two N: rows N..N_pad-1 are zeros; only the straddling
    tile is partial, tiles wholly in the padding skip their loads and stores."""
    B, N, C = shape
    say(f"{plan} padded B={B} N={N} C={C} {dtype}")
    P = whtmix.padded_tokens(N)
    x, _ = workloads.draw(B, N, C, dtype, seed=N)
    g = np.random.default_rng(N).uniform(0.5, 1.5, (P, C)).astype(np.float32)
    y = run_gpu(x, g, dtype, dev, plan=plan)
    status_ok()
    check(f"{plan} padded", y, orc.whtmix(x, g), dtype)


TWO_PASS_SHAPES = [(3, 256, 128), (1, 512, 64), (1, 1024, 64), (2, 512, 128), (16, 1024, 64),
                   (47, 512, 128), (1, 65536, 1), (1, 8, 8192), (300, 1024, 64),
                   (1, 32768, 1), (5, 128, 256), (600, 256, 128)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", TWO_PASS_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_two_pass_parity(shape, dtype, dev, orc):
    B, N, C = shape
    say(f"two_pass B={B} N={N} C={C} {dtype}")
    x, g = workloads.draw(B, N, C, dtype, seed=B * 1000 + N + C + 1)
    y = run_gpu(x, g, dtype, dev, plan="two_pass")
    check("two_pass", y, orc.whtmix(x, g), dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 1000, 64), (3, 200, 128), (2, 300, 128), (1, 129, 256),
                                   (2, 17, 2048), (1, 24584, 1)],
                         ids=lambda s: "x".join(map(str, s)))
def test_two_pass_padded_tokens(shape, dtype, dev, orc):
    """The fold reads zeros for rows past N (whole 16-byte groups: N*C is a
    multiple of 8); pass 3 stores only the valid rows."""
    B, N, C = shape
    say(f"two_pass padded B={B} N={N} C={C} {dtype}")
    P = whtmix.padded_tokens(N)
    x, _ = workloads.draw(B, N, C, dtype, seed=N + 1)
    g = np.random.default_rng(N + 1).uniform(0.5, 1.5, (P, C)).astype(np.float32)
    y = run_gpu(x, g, dtype, dev, plan="two_pass")
    check("two_pass padded", y, orc.whtmix(x, g), dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(3, 200, 128), (9, 1000, 64)], ids=lambda s: "x".join(map(str, s)))
def test_two_pass_separable_padded(shape, dtype, dev, orc):
    """The fold forms exp(g_t[n] + g_c[c]) for all N_pad token frequencies,
    padded rows included; with 9 slices the last group of eight slices has
    seven slices' blocks idle."""
    B, N, C = shape
    say(f"two_pass separable padded B={B} N={N} C={C} {dtype}")
    x, _ = workloads.draw(B, N, C, dtype, seed=N + 3)
    gt, gc = workloads.draw_log_gains(whtmix.padded_tokens(N), C, seed=N + 4)
    y = run_gpu_separable(x, gt, gc, dtype, dev, plan="two_pass")
    check("two_pass separable padded", y, orc.whtmix_separable(x, gt, gc), dtype)


@pytest.mark.parametrize("plan", PLANS + ["two_pass"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_separable(dtype, plan, dev, orc):
    B, N, C = 2, 1024, 64
    x, _ = workloads.draw(B, N, C, dtype, seed=5)
    gt, gc = workloads.draw_log_gains(N, C, seed=6)
    y = run_gpu_separable(x, gt, gc, dtype, dev, plan=plan)
    status_ok()
    check(f"{plan} separable", y, orc.whtmix_separable(x, gt, gc), dtype)


@pytest.mark.parametrize("plan", PLANS + ["two_pass", "auto"])
def test_image1k_workload(plan, dev, orc):
    """image1k_f32 (B=1, N=1024, C=64); AUTO takes WAVE_TILES for it."""
    w = workloads.WORKLOADS["image1k_f32"]
    assert whtmix.plan_describe(w.B, w.N, w.C, w.dtype)["plan"] == "wave_tiles"
    x, g = workloads.inputs(w)
    y = run_gpu(x, g, w.dtype, dev, plan=plan)
    status_ok()
    check(f"image1k_f32 {plan}", y, orc.whtmix(x, g), w.dtype)


@pytest.mark.parametrize("plan", PLANS + ["two_pass"])
def test_back_to_back_and_in_place(plan, dev, orc):
    """Consecutive calls on one stream reuse the counter block (each kernel
    returns it to zero); in place (y == x) reads every x before any y store
    of the same slice."""
    import torch
    B, N, C = 4, 1024, 64
    outs, refs = [], []
    for i in range(3):
        x, g = workloads.draw(B, N, C, "f32", seed=40 + i)
        xd = to_device(x, "f32", dev)
        gd = torch.from_numpy(g).to(dev)
        whtmix.forward(xd, gd, out=xd, plan=plan)
        outs.append(xd)
        refs.append(orc.whtmix(x, g))
    torch.cuda.synchronize()
    status_ok()
    for i, (o, r) in enumerate(zip(outs, refs)):
        check(f"call {i} in place", to_host(o), r, "f32")


def test_give_up_path_reports_and_recovers(dev, orc):
    """A poll limit of one makes the counter waits give up (forced from the
    host; every wave still exits).  The stream then reports
    WHTMIX_ERROR_DEVICE_TIMEOUT once, and the next default call is correct."""
    import torch
    B, N, C = 16, 1024, 64
    x, g = workloads.draw(B, N, C, "f32", seed=77)
    xd = to_device(x, "f32", dev)
    gd = torch.from_numpy(g).to(dev)
    status_ok()
    seen = 0
    for _ in range(3):
        whtmix.forward(xd, gd, plan="one_launch", spin_limit=1)
        st = whtmix.stream_status()
        assert st in (whtmix.SUCCESS, whtmix.ERROR_DEVICE_TIMEOUT)
        seen += st == whtmix.ERROR_DEVICE_TIMEOUT
    say(f"  calls that gave up: {seen} of 3")
    assert seen >= 1
    assert whtmix.stream_status() == whtmix.SUCCESS       # cleared once read
    y = whtmix.forward(xd, gd, plan="one_launch")
    status_ok()
    check("after give-up", to_host(y), orc.whtmix(x, g), "f32")


def test_two_streams_run_independently(dev, orc):
    """Calls on two streams at once: each stream has its own workspace and
    counter block, so the two kernels may overlap on the GPU."""
    import torch
    B, N, C = 8, 1024, 64
    streams = [torch.cuda.Stream(dev), torch.cuda.Stream(dev)]
    outs, refs = [], []
    for i, s in enumerate(streams):
        x, g = workloads.draw(B, N, C, "f32", seed=500 + i)
        xd, gd = to_device(x, "f32", dev), torch.from_numpy(g).to(dev)
        torch.cuda.synchronize(dev)
        with torch.cuda.stream(s):
            outs.append([whtmix.forward(xd, gd, plan="one_launch", stream=s) for _ in range(3)])
        refs.append(orc.whtmix(x, g))
    for s in streams:
        assert whtmix.stream_status(s.cuda_stream) == whtmix.SUCCESS
    for i, (o, r) in enumerate(zip(outs, refs)):
        for j, y in enumerate(o):
            check(f"stream {i} call {j}", to_host(y), r, "f32")


def test_status_of_a_stream_without_single_launch_calls(dev):
    import torch
    s = torch.cuda.Stream(dev)
    assert whtmix.stream_status(s.cuda_stream) == whtmix.SUCCESS
