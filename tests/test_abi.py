"""The C ABI on the host: the library loads, exports what include/whtmix.h
declares, and rejects bad arguments before any HIP call (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2607_25234_amd import whtmix
from paper_2607_25234_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "whtmix.h")

ALIGNED = 0x10000          # fake device addresses: never dereferenced, every
ALIGNED2 = 0x40000000      # call below is rejected or is a no-op on the host


def header_symbols():
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"WHTMIX_API\s+[\w\s\*]*?\b(whtmix_\w+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert header_symbols() == sorted(whtmix.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = whtmix.lib()
    for name in header_symbols():
        assert hasattr(lib, name), name
        assert ctypes.cast(getattr(lib, name), ctypes.c_void_p).value


def test_library_exports_nothing_else():
    """Only the C API is visible (internal C++ symbols are hidden)."""
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", whtmix.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    text_syms = sorted(l.split()[-1] for l in out.splitlines() if " T " in l)
    assert text_syms == sorted(header_symbols())


def test_version_and_status_strings():
    assert whtmix.lib().whtmix_version() == 10200
    for st in range(9):
        assert whtmix.status_string(st)
    assert whtmix.status_string(99) == "unknown status"


def call(x=ALIGNED, g=ALIGNED2, y=ALIGNED, B=1, N=64, C=64, dtype=0, plan=0):
    return whtmix.forward_raw(x, g, y, B, N, C, dtype, 0, plan)


@pytest.mark.parametrize("kwargs,status", [
    (dict(dtype=2), 3),
    (dict(dtype=-1), 3),
    (dict(B=-1), 1),
    (dict(C=3), 2),
    (dict(C=0), 2),
    (dict(C=96), 2),
    (dict(N=0), 1),
    (dict(N=-4), 1),
    (dict(N=1 << 16, C=1 << 15), 7),          # N*C = 2^31 > 2^30
    (dict(N=(1 << 24) + 1, C=64), 7),         # N pads to 2^25: 2^31 > 2^30
    (dict(B=1 << 30, N=1 << 10, C=1 << 10), 7),  # B*N*C beyond the grid limit
    (dict(x=0), 1),
    (dict(g=0), 1),
    (dict(y=0), 1),
    (dict(x=ALIGNED + 4, y=ALIGNED2 * 2), 4),
    (dict(g=ALIGNED2 + 8), 4),
    (dict(y=ALIGNED + 4 * 64), 1),            # partial overlap of x and y
    (dict(g=ALIGNED + 16, y=ALIGNED), 1),     # gain inside y
    (dict(plan=9), 1),
    (dict(plan=1, N=64, C=64), 1),            # SMALL needs N*C <= 2^10
    (dict(plan=2, N=8, C=8), 1),              # FUSED needs 2^11..2^16
    (dict(plan=2, N=2048, C=64), 1),
    (dict(plan=3, N=32, C=64), 1),            # THREE_PASS needs >= 2^12
    (dict(plan=4, N=32, C=64), 1),            # ONE_LAUNCH needs 2^12..2^16
    (dict(plan=4, N=2048, C=64), 1),
    (dict(plan=4, N=4095, C=1), 1),           # ... and N*C a multiple of 8
    (dict(plan=4, B=2047, N=1024, C=64), 1),  # ... and B <= 2046
    (dict(plan=5, N=32, C=64), 1),            # WAVE_TILES needs 2^12..2^16
    (dict(plan=5, N=4096, C=32), 1),
    (dict(plan=5, N=4095, C=1), 1),           # ... and N*C a multiple of 8
    (dict(plan=5, B=1 << 19, N=1024, C=64), 7),   # ... and B*N*C/8 < 2^32 work-items
    (dict(B=1 << 21, N=1024, C=64), 7),           # tiled plans: B*N*C/32 < 2^32
    (dict(plan=6, N=32, C=64), 1),                # TWO_PASS needs 2^15..2^16
    (dict(plan=6, N=32767, C=1), 1),              # ... and N*C a multiple of 8
    (dict(plan=6, B=(1 << 19) - 7, N=1024, C=64), 7),   # ... and B rounded up to 8
])
def test_rejected_before_any_hip_call(kwargs, status):
    assert call(**kwargs) == status


def sep(x=ALIGNED, gt=ALIGNED2, gc=ALIGNED2 + 4096, y=ALIGNED, B=1, N=64, C=64, dtype=0):
    return whtmix.forward_separable_raw(x, gt, gc, y, B, N, C, dtype, 0)


@pytest.mark.parametrize("kwargs,status", [
    (dict(gt=0), 1),
    (dict(gc=0), 1),
    (dict(gc=ALIGNED2 + 4), 4),
    (dict(gt=ALIGNED + 64), 1),               # token gains inside y
    (dict(gc=ALIGNED + 64 * 64 * 4 - 16), 1),  # channel gains overlap y's end
    (dict(C=12), 2),
    (dict(dtype=5), 3),
])
def test_separable_rejected_before_any_hip_call(kwargs, status):
    assert sep(**kwargs) == status


def bwd(x=ALIGNED, dy=ALIGNED * 16, g=ALIGNED2, dx=ALIGNED * 64, dg=ALIGNED2 * 2, B=1, N=64,
        C=64, dtype=0):
    return whtmix.backward_raw(x, dy, g, dx, dg, B, N, C, dtype, 0)


@pytest.mark.parametrize("kwargs,status", [
    (dict(dx=0, dg=0), 1),                    # nothing to compute
    (dict(dy=0), 1),
    (dict(x=0), 1),                           # x needed for the gain gradient
    (dict(g=0), 1),
    (dict(dx=ALIGNED + 64), 1),               # dx overlaps x
    (dict(dx=ALIGNED * 16 + 64), 1),          # dx partially overlaps dy
    (dict(dg=ALIGNED * 16), 1),               # dgain inside dy
    (dict(dg=ALIGNED2 + 256), 1),             # dgain overlaps the gain
    (dict(dg=ALIGNED * 64), 1),               # dgain overlaps dx
    (dict(dx=ALIGNED * 64 + 4), 4),
    (dict(C=6), 2),
    (dict(dtype=3), 3),
])
def test_backward_rejected_before_any_hip_call(kwargs, status):
    assert bwd(**kwargs) == status


def test_backward_separable_rejected_before_any_hip_call():
    f = whtmix.backward_separable_raw
    # one log-gain gradient without the other
    assert f(ALIGNED, ALIGNED * 16, ALIGNED2, ALIGNED2 + 4096, 0, ALIGNED2 * 2, 0,
             1, 64, 64, 0, 0) == 1
    # nothing to compute
    assert f(ALIGNED, ALIGNED * 16, ALIGNED2, ALIGNED2 + 4096, 0, 0, 0, 1, 64, 64, 0, 0) == 1
    # token-gain gradient overlapping the channel gains
    assert f(ALIGNED, ALIGNED * 16, ALIGNED2, ALIGNED2 + 4096, 0, ALIGNED2 + 4096 - 64,
             ALIGNED2 * 2, 1, 64, 64, 0, 0) == 1


def mod(x=ALIGNED, wi=ALIGNED2, g=ALIGNED2 * 2, wo=ALIGNED2 * 3, y=ALIGNED, B=1, N=64, C=64,
        dtype=0, plan="auto"):
    return whtmix.module_forward_raw(x, wi, g, wo, y, B, N, C, dtype, 0, plan)


@pytest.mark.parametrize("kwargs,status", [
    (dict(wi=0), 1),
    (dict(wo=0), 1),
    (dict(g=0), 1),
    (dict(x=0), 1),
    (dict(wi=ALIGNED2 + 8), 4),
    (dict(wo=ALIGNED2 * 3 + 4), 4),
    (dict(wi=ALIGNED + 64 * 64 * 4 - 16), 1),  # w_in overlaps y's end
    (dict(wo=ALIGNED + 256), 1),              # w_out inside y
    (dict(y=ALIGNED + 64), 1),                # partial overlap of x and y
    (dict(C=1 << 13, N=1), 7),                # weights of C*C beyond C = 4096
    (dict(C=48), 2),
    (dict(dtype=2), 3),
    (dict(plan=2, N=8, C=8), 1),
])
def test_module_rejected_before_any_hip_call(kwargs, status):
    assert mod(**kwargs) == status


def test_module_separable_rejected_before_any_hip_call():
    f = whtmix.module_forward_separable_raw
    ok = dict(x=ALIGNED, wi=ALIGNED2, gt=ALIGNED2 * 2, gc=ALIGNED2 * 2 + 4096, wo=ALIGNED2 * 3,
              y=ALIGNED)

    def call_sep(**kw):
        a = {**ok, **kw}
        return f(a["x"], a["wi"], a["gt"], a["gc"], a["wo"], a["y"], 1, 64, 64, 0, 0)

    assert call_sep(gt=0) == 1
    assert call_sep(gc=0) == 1
    assert call_sep(gc=ALIGNED + 128) == 1    # channel gains inside y
    assert call_sep(gt=ALIGNED2 * 2 + 4) == 4


def test_module_empty_batch_is_a_no_op():
    assert whtmix.module_forward_raw(0, 0, 0, 0, 0, 0, 64, 64, 1, 0) == 0


def mbwd(x=ALIGNED, wi=ALIGNED2, g=ALIGNED2 * 2, wo=ALIGNED2 * 3, dy=ALIGNED * 16,
         dx=ALIGNED * 64, dwi=ALIGNED2 * 4, dwo=ALIGNED2 * 5, dg=ALIGNED2 * 6, B=1, N=64, C=64,
         dtype=0):
    return whtmix.module_backward_raw(x, wi, g, wo, dy, dx, dwi, dwo, dg, B, N, C, dtype, 0)


@pytest.mark.parametrize("kwargs,status", [
    (dict(dwi=0), 1),
    (dict(dwo=0), 1),
    (dict(dx=0), 1),
    (dict(dy=0), 1),
    (dict(x=0), 1),
    (dict(wi=0), 1),
    (dict(dx=ALIGNED + 64), 1),               # dx overlaps x (read after dx is written)
    (dict(dwi=ALIGNED2 * 3 + 16), 1),         # dW_in overlaps W_out
    (dict(dwo=ALIGNED2 * 4), 1),              # dW_out is dW_in
    (dict(dg=ALIGNED * 64 + 128), 1),         # dgain inside dx
    (dict(dwi=ALIGNED2 * 4 + 4), 4),
    (dict(C=1 << 13, N=1), 7),
    (dict(B=1 << 16, N=1 << 15, C=1), 7),     # B*N >= 2^31
    (dict(C=12), 2),
])
def test_module_backward_rejected_before_any_hip_call(kwargs, status):
    assert mbwd(**kwargs) == status


def test_module_backward_separable_rejected_before_any_hip_call():
    f = whtmix.module_backward_separable_raw
    args = [ALIGNED, ALIGNED2, ALIGNED2 * 2, ALIGNED2 * 2 + 4096, ALIGNED2 * 3, ALIGNED * 16,
            ALIGNED * 64, ALIGNED2 * 4, ALIGNED2 * 5]
    assert f(*args, ALIGNED2 * 6, 0, 1, 64, 64, 0, 0) == 1      # one log-gain gradient only
    assert f(*args, ALIGNED2 * 6, ALIGNED2 * 6 + 64, 1, 64, 64, 0, 0) == 1   # overlapping
    # dx == dy is allowed: passes every host check (then would launch; not called here)


def test_padded_plans():
    """Non-power-of-two token counts are zero-padded (section III-B)."""
    for N, C, P in [(3, 4, 4), (5, 1, 8), (9216, 64, 16384), (25600, 64, 32768),
                    (50176, 64, 65536), (1, 1, 1)]:
        d = whtmix.plan_describe(2, N, C)
        assert d["padded_tokens"] == P == whtmix.padded_tokens(N)
        assert 1 << d["log2_slice"] == P * C
    assert whtmix.plan_describe(2, 9216, 64)["workspace_bytes"] == 2 * 16384 * 64 * 4


def test_empty_batch_is_a_no_op():
    assert whtmix.forward_raw(0, 0, 0, 0, 64, 64, 0, 0) == 0
    assert whtmix.forward_raw(0, 0, 0, 0, 1 << 20, 1 << 7, 1, 0) == 0


def test_default_options_pass_null():
    """With every option at its default the binding passes NULL options
    (documented as the defaults); any other option builds the structure."""
    assert whtmix._opt_arg() is None
    assert whtmix._opt_arg("auto", None, 0) is None and whtmix._opt_arg(0) is None
    assert whtmix._opt_arg("three_pass") is not None
    assert whtmix._opt_arg("auto", spin_limit=5) is not None
    assert whtmix._opt_arg("auto", events=[None] * 4) is not None
    # the NULL path is checked like the structure path, before any HIP call
    assert whtmix.forward_raw(0, 0, 0, 1, 64, 64, 0, 0) == 1
    assert whtmix.forward_raw(0, 0, 0, 1, 64, 64, 0, 0, "fused") == 1
    assert call(C=12) == 2 and call(C=12, plan=3) == 2


def test_call_module_marshals_only():
    """The forward entry points go through the binding's CPython call module,
    bound to the same library functions ctypes sees; its argument checks
    mirror ctypes' (ints or None for pointers) and every status comes from
    the library."""
    m = whtmix._call()
    L = whtmix.lib()
    assert whtmix._opt_address("auto", None, 0) == (None, 0)
    o, addr = whtmix._opt_address("three_pass", None, 0)
    assert addr == ctypes.addressof(o) and o.plan == whtmix.PLANS["three_pass"]
    # identical statuses through both routes, for defaults and forced plans
    for args in [(0, 0, 0, 1, 64, 64, 0, 0), (ALIGNED, ALIGNED2, ALIGNED, 1, 64, 12, 0, 0),
                 (ALIGNED, ALIGNED2, ALIGNED, 1, 64, 64, 9, 0),
                 (ALIGNED + 4, ALIGNED2, ALIGNED2 * 2, 1, 64, 64, 0, 0)]:
        assert m.forward_ex(*args, 0) == L.whtmix_forward_ex(*args, None)
        assert m.forward_ex(*args, None) == L.whtmix_forward_ex(*args, None)
    o, addr = whtmix._opt_address(9, None, 0)     # an invalid plan, in the structure
    assert m.forward_ex(ALIGNED, ALIGNED2, ALIGNED, 1, 64, 64, 0, 0, addr) == 1
    assert m.forward_separable(0, 0, 0, 0, 1, 64, 64, 0, 0, 0) == 1
    with pytest.raises(TypeError):
        m.forward_ex(1.5, 0, 0, 1, 64, 64, 0, 0, 0)
    with pytest.raises(TypeError):
        m.forward_ex(0, 0, 0, 1, 64, 64, 0, 0)          # 8 arguments
    with pytest.raises(OverflowError):
        m.forward_ex(0, 0, 0, 1 << 64, 64, 64, 0, 0, 0)
    with pytest.raises(OverflowError):
        m.forward_ex(0, 0, 0, 1, 64, 64, 1 << 40, 0, 0)


def test_plan_table():
    d = whtmix.plan_describe(1, 1, 1)
    assert d["plan"] == "small" and d["kernels"] == 1 and d["workspace_bytes"] == 0
    assert whtmix.plan_describe(3, 32, 32)["plan"] == "small"
    assert whtmix.plan_describe(3, 32, 64)["plan"] == "fused"
    assert whtmix.plan_describe(3, 256, 64)["plan"] == "fused"
    assert whtmix.plan_describe(3, 256, 128)["plan"] == "two_pass"   # 2^15, up to 48 slices
    d = whtmix.plan_describe(3, 1024, 128, "bf16")
    assert d["plan"] == "three_pass" and d["kernels"] == 3
    assert d["workspace_bytes"] == 3 * 1024 * 128 * 4
    # 2^16 from 48 slices: one workgroup of two register sets for the forward;
    # the block and the backward pass take the three-pass plan; ONE_LAUNCH
    # only when asked for
    assert whtmix.plan_describe(47, 512, 128, "bf16")["plan"] == "three_pass"
    d = whtmix.plan_describe(47, 512, 128, "bf16", "one_launch")
    assert (d["plan"], d["kernels"], d["workspace_bytes"]) == ("one_launch", 1, 47 << 18)
    assert (d["outer_bits"], d["run_bits"]) == (9, 2)
    d = whtmix.plan_describe(2, 64, 64, plan="one_launch")
    assert (d["plan"], d["outer_bits"], d["run_bits"]) == ("one_launch", 9, 6)
    # TWO_PASS: slices of 2^15 and 2^16 only, two launches, the wave tiles'
    # workspace; the block and the backward pass run as for WAVE_TILES
    d = whtmix.plan_describe(3, 1024, 64, "bf16", "two_pass")
    assert (d["plan"], d["kernels"], d["workspace_bytes"]) == ("two_pass", 2, 3 << 18)
    assert (d["outer_bits"], d["run_bits"], d["module_outer_bits"]) == (9, 2, 11)
    d = whtmix.plan_describe(5, 256, 128, plan="two_pass")
    assert (d["plan"], d["outer_bits"], d["run_bits"], d["module_outer_bits"]) == \
        ("two_pass", 9, 3, 0)
    for B, N, C in [(1, 256, 64), (1, 128, 64), (1, 1024, 128), (1, 32767, 1)]:
        with pytest.raises(whtmix.WhtmixError):
            whtmix.plan_describe(B, N, C, plan="two_pass")   # K < 15, K > 16, N*C % 8
    # small batches of 2^15 and 2^16 slices: three launches of one-wave tiles
    for B, N, C, plan in [(1, 1024, 64, "wave_tiles"), (3, 1024, 64, "wave_tiles"),
                          (4, 1024, 64, "two_pass"), (16, 1024, 64, "two_pass"),
                          (17, 1024, 64, "three_pass"), (16, 512, 64, "two_pass"),
                          (48, 512, 64, "two_pass"), (49, 512, 64, "fused"),
                          (1, 32767, 1, "fused"),
                          (1, 65535, 1, "three_pass"), (2, 256, 64, "fused")]:
        assert whtmix.plan_describe(B, N, C)["plan"] == plan, (B, N, C)
    d = whtmix.plan_describe(1, 1024, 64)
    assert (d["kernels"], d["workspace_bytes"], d["module_path"], d["module_outer_bits"]) == \
        (3, 1 << 18, "mfma", 11)
    assert whtmix.plan_describe(2, 512, 64)["module_outer_bits"] == 0   # the block: FUSED
    d = whtmix.plan_describe(48, 512, 128, "bf16")
    assert (d["plan"], d["kernels"], d["workspace_bytes"]) == ("fused", 1, 0)
    assert (d["module_path"], d["module_outer_bits"]) == ("mfma", 11)
    assert d["module_backward_fused"]
    d = whtmix.plan_describe(3, 512, 128, "bf16", "fused")
    assert (d["plan"], d["workspace_bytes"]) == ("fused", 0)
    d = whtmix.plan_describe(2, 64, 64, plan="three_pass")
    assert d["plan"] == "three_pass" and d["outer_bits"] == 11
    d = whtmix.plan_describe(4, 65536, 128, "bf16")
    assert (d["outer_bits"], d["run_bits"], d["workspace_bytes"]) == (14, 5, 4 << 25)
    d = whtmix.plan_describe(1, 262144, 256, "bf16")   # 2^16 outer tiles
    assert (d["outer_bits"], d["run_bits"], d["workspace_bytes"]) == (16, 5, 1 << 28)
    for w in workloads.WORKLOADS.values():
        d = whtmix.plan_describe(w.B, w.N, w.C, w.dtype)
        K = d["log2_slice"]
        assert 1 << K == w.N * w.C
        if K == 16:   # image1k: one 2^16 slice
            assert (d["plan"], d["kernels"], d["outer_bits"], d["run_bits"]) == ("wave_tiles", 3, 9, 2)
        if K > 16:
            A, R = d["outer_bits"], d["run_bits"]
            assert d["plan"] == "three_pass"
            assert 11 <= A <= 16 and 11 <= K - A + R <= 15 and R <= A
            assert (A == 16) == (K >= 26)


@pytest.mark.parametrize("shape", [(1, 512, 256), (2, 700, 256), (1, 262144, 256)],
                         ids=lambda s: "x".join(map(str, s)))
def test_block_c256_takes_pair_tiles(shape):
    """bf16 C = 256 from 2^17 elements per slice: the projections fused into
    2^16-element outer tiles; float32 C = 256 stays unfused."""
    B, N, C = shape
    d = whtmix.plan_describe(B, N, C, "bf16")
    assert (d["plan"], d["module_path"], d["module_outer_bits"]) == ("three_pass", "mfma", 16)
    f = whtmix.plan_describe(B, N, C, "f32")
    assert f["module_path"] == "unfused" and f["module_outer_bits"] == f["outer_bits"]


def test_block_paths():
    assert whtmix.plan_describe(1, 256, 256, "bf16")["module_path"] == "unfused"   # 2^16
    assert whtmix.plan_describe(1, 64, 256, "bf16")["module_path"] == "unfused"    # FUSED plan
    assert whtmix.plan_describe(2, 4, 4, "bf16")["module_path"] == "small"
    d = whtmix.plan_describe(4, 65536, 128, "bf16")
    assert (d["module_path"], d["module_outer_bits"]) == ("mfma", 14)
    assert whtmix.plan_describe(1, 256, 64)["module_outer_bits"] == 0    # FUSED plan
    assert whtmix.plan_describe(1, 4, 8192)["module_path"] is None      # C above the limit


def test_block_backward_paths():
    """The block's backward fuses its projections for 16 <= C <= 128 on
    three-pass slices up to 2^25 elements, and bf16 C = 256 on 2^26..2^28."""
    fused = lambda *a: whtmix.plan_describe(*a)["module_backward_fused"]
    assert fused(4, 65536, 128, "bf16")
    assert fused(1, 3000, 32, "bf16") and fused(2, 128, 128, "bf16", "three_pass")
    assert fused(4, 65536, 128, "f32") and fused(1, 65536, 16, "bf16")
    assert not fused(1, 65536, 8, "bf16")               # C = 8: VALU projections
    assert not fused(1, 262144, 256, "f32")             # float32 C = 256
    assert fused(1, 262144, 256, "bf16") and fused(1, 1 << 20, 256, "bf16")   # C = 256, 2^26..2^28
    assert not fused(1, 65536, 256, "bf16")             # C = 256 below 2^26 (module split)
    assert not fused(1, 1 << 21, 256, "bf16")           # 2^29
    assert not fused(1, 256, 64, "bf16")                # FUSED plan
    assert not fused(1, 1 << 19, 128, "bf16")           # 2^26 elements


def test_every_three_pass_split_fits_the_tiles():
    for K in range(12, 31):
        N = 1 << (K // 2)
        C = 1 << (K - K // 2)
        d = whtmix.plan_describe(1, N, C, plan="three_pass")
        A, R = d["outer_bits"], d["run_bits"]
        assert 11 <= A <= 15 or (A == 16 and K >= 26), K   # 2^16 outer tiles from 2^26
        assert 1 <= K - A and 11 <= K - A + R <= 15 and 0 <= R <= A, K


def test_workspace_failure_is_reported_before_any_launch(monkeypatch):
    """A workspace that cannot be allocated returns OUT_OF_MEMORY with its text
    and enqueues nothing (the library's test hook refuses every workspace
    request before any HIP call, so this runs without a GPU)."""
    torch = pytest.importorskip("torch")
    if torch.cuda.device_count() > 0:
        pytest.skip("fake device addresses are for hosts without a GPU")
    monkeypatch.setenv("WHTMIX_TEST_FAIL_WORKSPACE", "1")
    lib = whtmix.lib()
    # three-pass shapes need a workspace: forward, backward, the block
    assert whtmix.forward_raw(ALIGNED, ALIGNED2, ALIGNED, 2, 4096, 64, 0, 0) == 5
    assert "WHTMIX_TEST_FAIL_WORKSPACE" in whtmix.last_error()
    assert whtmix.backward_raw(ALIGNED, ALIGNED + (1 << 22), ALIGNED2, ALIGNED + (2 << 22),
                               ALIGNED2 + (1 << 22), 2, 4096, 64, 0, 0) == 5
    assert lib.whtmix_status_string(5).decode()
    # a shape with no workspace (the fused plan) never reaches the allocator,
    # so it would launch: it is not called here without a GPU
    assert whtmix.plan_describe(2, 256, 64)["workspace_bytes"] == 0


def test_python_forward_rejects_host_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(1, 64, 64)
    g = torch.ones(64, 64)
    with pytest.raises(ValueError):
        whtmix.forward(x, g)


def test_noalloc_rejects_beyond_its_scratch_before_any_hip_call():
    """whtmix_forward_noalloc: B * N_pad * C above 2^23 with a workspace plan
    is TOO_LARGE; the usual argument checks come first."""
    big = (1 << 40, 1 << 41, 1 << 42)
    assert whtmix.forward_noalloc_raw(*big, 5, 16384, 128, 0, 0) == 7
    assert "scratch" in whtmix.last_error()
    assert whtmix.forward_noalloc_raw(*big, 1, 65536, 256, 1, 0) == 7
    assert whtmix.forward_noalloc_raw(0, 1 << 41, 1 << 42, 1, 64, 64, 0, 0) == 1
    assert whtmix.forward_noalloc_raw(*big, 1, 64, 63, 0, 0) == 2
    assert whtmix.forward_noalloc_raw(*big, 0, 64, 64, 0, 0) == 0
