"""whtmix_forward_noalloc (the entry point that allocates nothing, its
three-pass, two-pass or wave-tile workspace in a fixed device array) against whtmix_forward,
through the C ABI: two calls in a row, the second with a smaller input.
Both run the same kernels, so the outputs agree bit for bit; each is also
held to the oracle's bar.
"""
import numpy as np
import pytest

from oracle import oracle as oracle_mod
from paper_2607_25234_amd import whtmix, workloads
from tests.gpu_util import DERIVED, TOL, device, errors, say, to_device, to_host

pytestmark = pytest.mark.gpu


def _run(entry, x, g, dtype, dev):
    import torch
    xd = to_device(x, dtype, dev)
    gd = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(dev)
    yd = torch.empty_like(xd)
    B, N, C = x.shape
    dt = whtmix.DTYPE_BF16 if dtype == "bf16" else whtmix.DTYPE_F32
    stream = torch.cuda.current_stream(dev).cuda_stream
    if entry == "noalloc":
        st = whtmix.forward_noalloc_raw(xd.data_ptr(), gd.data_ptr(), yd.data_ptr(), B, N, C,
                                        dt, stream)
    else:
        st = whtmix.forward_raw(xd.data_ptr(), gd.data_ptr(), yd.data_ptr(), B, N, C, dt,
                                stream)
    assert st == whtmix.SUCCESS, whtmix.status_string(st)
    torch.cuda.synchronize(dev)
    return to_host(yd)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_matches_forward_twice(dtype):
    """The first call fills the scratch (2^23 floats), the second, smaller one
    reuses it, the third runs the wave-tile plan in it and the fourth the
    two-pass plan; a FUSED-plan call needs no scratch at all."""
    dev = device()
    orc = oracle_mod.Oracle()
    for i, (B, N, C) in enumerate([(4, 16384, 128), (3, 4096, 64), (1, 1024, 64), (5, 512, 64),
                                   (2, 256, 64)]):
        say(f"noalloc call {i}: B={B} N={N} C={C} {dtype} "
            f"plan={whtmix.plan_describe(B, N, C, dtype)['plan']}")
        x, g = workloads.draw(B, N, C, dtype, seed=900 + i)
        y0 = _run("noalloc", x, g, dtype, dev)
        y1 = _run("forward", x, g, dtype, dev)
        assert np.array_equal(y0, y1)
        err, _ = errors(y0, orc.whtmix(x, g))
        say(f"  normwise-max vs oracle {err:.3e}")
        assert err <= TOL[dtype] and err <= DERIVED[dtype]


def test_noalloc_rejects_beyond_the_scratch():
    """B * N_pad * C above 2^23 with a workspace plan: TOO_LARGE, nothing
    enqueued (checked on the host before any HIP call; the pointers are
    never dereferenced)."""
    st = whtmix.forward_noalloc_raw(1 << 40, 1 << 41, 1 << 42, 5, 16384, 128,
                                    whtmix.DTYPE_F32, 0)
    assert st == 7
    assert "scratch" in whtmix.last_error()
