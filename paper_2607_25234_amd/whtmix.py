"""Python binding of the WHTMix C ABI (include/whtmix.h).

Argument marshalling only: every step of the mixer runs in the HIP kernels of
``libwhtmix.so``.  PyTorch supplies device memory and the current stream.
There is no fallback: if the library is missing, importing the functions
that need it raises.

    y = forward(x, gain)          # x [B, N, C] (or [N, C]) f32/bf16, gain [N, C] f32
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libwhtmix.so")

SUCCESS = 0
DTYPE_F32, DTYPE_BF16 = 0, 1
PLANS = {"auto": 0, "small": 1, "fused": 2, "three_pass": 3, "one_launch": 4,
         "wave_tiles": 5, "two_pass": 6}
PLAN_NAMES = {v: k for k, v in PLANS.items()}

# Every symbol include/whtmix.h declares.
EXPORTS = (
    "whtmix_backward",
    "whtmix_backward_separable",
    "whtmix_forward",
    "whtmix_forward_ex",
    "whtmix_forward_noalloc",
    "whtmix_forward_separable",
    "whtmix_module_backward",
    "whtmix_module_backward_separable",
    "whtmix_module_forward",
    "whtmix_module_forward_separable",
    "whtmix_plan_describe",
    "whtmix_status_string",
    "whtmix_last_error",
    "whtmix_release_workspaces",
    "whtmix_stream_status",
    "whtmix_version",
)
ERROR_DEVICE_TIMEOUT = 8


class WhtmixError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})"
                         + (f" [{last_error()}]" if last_error() else ""))


class Options(ctypes.Structure):
    _fields_ = [("plan", ctypes.c_int), ("events", ctypes.c_void_p * 4),
                ("spin_limit", ctypes.c_uint32)]


MODULE_PATHS = {0: "small", 1: "mfma", 2: "unfused"}


class PlanInfo(ctypes.Structure):
    _fields_ = [("plan", ctypes.c_int), ("kernels", ctypes.c_int),
                ("log2_slice", ctypes.c_int), ("outer_bits", ctypes.c_int),
                ("run_bits", ctypes.c_int), ("workspace_bytes", ctypes.c_int64),
                ("padded_tokens", ctypes.c_int64), ("module_path", ctypes.c_int),
                ("module_outer_bits", ctypes.c_int), ("module_backward_fused", ctypes.c_int)]


_lib = None


def lib():
    """The loaded libwhtmix.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2607_25234_amd.build` (there is no fallback)")
        try:
            # Load torch's HIP runtime first so that the library binds to the
            # same runtime instance (same soname) as the tensors and streams.
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        i64, vp = ctypes.c_int64, ctypes.c_void_p
        L.whtmix_forward.argtypes = [vp, vp, vp, i64, i64, i64, ctypes.c_int, vp]
        L.whtmix_forward.restype = ctypes.c_int
        L.whtmix_forward_ex.argtypes = [vp, vp, vp, i64, i64, i64, ctypes.c_int, vp,
                                        ctypes.POINTER(Options)]
        L.whtmix_forward_ex.restype = ctypes.c_int
        L.whtmix_forward_noalloc.argtypes = [vp, vp, vp, i64, i64, i64, ctypes.c_int, vp]
        L.whtmix_forward_noalloc.restype = ctypes.c_int
        L.whtmix_forward_separable.argtypes = [vp, vp, vp, vp, i64, i64, i64, ctypes.c_int, vp,
                                               ctypes.POINTER(Options)]
        L.whtmix_forward_separable.restype = ctypes.c_int
        L.whtmix_module_forward.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, ctypes.c_int,
                                            vp, ctypes.POINTER(Options)]
        L.whtmix_module_forward.restype = ctypes.c_int
        L.whtmix_module_forward_separable.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64,
                                                      ctypes.c_int, vp, ctypes.POINTER(Options)]
        L.whtmix_module_forward_separable.restype = ctypes.c_int
        L.whtmix_module_backward.argtypes = [vp] * 9 + [i64, i64, i64, ctypes.c_int, vp,
                                                         ctypes.POINTER(Options)]
        L.whtmix_module_backward.restype = ctypes.c_int
        L.whtmix_module_backward_separable.argtypes = [vp] * 11 + [i64, i64, i64, ctypes.c_int,
                                                                   vp, ctypes.POINTER(Options)]
        L.whtmix_module_backward_separable.restype = ctypes.c_int
        L.whtmix_backward.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, ctypes.c_int, vp,
                                      ctypes.POINTER(Options)]
        L.whtmix_backward.restype = ctypes.c_int
        L.whtmix_backward_separable.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64,
                                                ctypes.c_int, vp, ctypes.POINTER(Options)]
        L.whtmix_backward_separable.restype = ctypes.c_int
        L.whtmix_plan_describe.argtypes = [i64, i64, i64, ctypes.c_int,
                                           ctypes.POINTER(Options), ctypes.POINTER(PlanInfo)]
        L.whtmix_plan_describe.restype = ctypes.c_int
        L.whtmix_status_string.argtypes = [ctypes.c_int]
        L.whtmix_status_string.restype = ctypes.c_char_p
        L.whtmix_last_error.argtypes = []
        L.whtmix_last_error.restype = ctypes.c_char_p
        L.whtmix_release_workspaces.argtypes = []
        L.whtmix_release_workspaces.restype = ctypes.c_int
        L.whtmix_version.argtypes = []
        L.whtmix_version.restype = ctypes.c_int
        L.whtmix_stream_status.argtypes = [vp]
        L.whtmix_stream_status.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().whtmix_status_string(status).decode()


def last_error() -> str:
    return lib().whtmix_last_error().decode()


def _options(plan: str | int = "auto", events=None, spin_limit: int = 0) -> Options:
    o = Options()
    o.plan = PLANS[plan] if isinstance(plan, str) else int(plan)
    for i, ev in enumerate(events or ()):
        o.events[i] = ev
    o.spin_limit = int(spin_limit)
    return o


def _opt_arg(plan: str | int = "auto", events=None, spin_limit: int = 0):
    """The options argument of an entry point: NULL when every option is
    its default (the library then takes AUTO, no events, the default spin
    limit), which saves building the structure on each call."""
    if events is None and not spin_limit and (plan == "auto" or plan == 0):
        return None
    return ctypes.byref(_options(plan, events, spin_limit))


def stream_status(stream: int | None = None) -> int:
    """whtmix_stream_status: synchronise the stream and return (and clear)
    the error word of its single-launch calls (SUCCESS or
    ERROR_DEVICE_TIMEOUT).  stream: a hipStream_t as int (default: torch's
    current stream)."""
    if stream is None:
        import torch
        stream = torch.cuda.current_stream().cuda_stream
    return int(lib().whtmix_stream_status(stream))


def plan_describe(B: int, N: int, C: int, dtype: str = "f32", plan: str | int = "auto") -> dict:
    """How a shape would run; raises WhtmixError on an invalid shape."""
    info = PlanInfo()
    opt = _options(plan)
    st = lib().whtmix_plan_describe(B, N, C, DTYPE_BF16 if dtype == "bf16" else DTYPE_F32,
                                    ctypes.byref(opt), ctypes.byref(info))
    if st != SUCCESS:
        raise WhtmixError(st, "whtmix_plan_describe")
    return {"plan": PLAN_NAMES[info.plan], "kernels": info.kernels,
            "log2_slice": info.log2_slice, "outer_bits": info.outer_bits,
            "run_bits": info.run_bits, "workspace_bytes": info.workspace_bytes,
            "padded_tokens": info.padded_tokens,
            "module_path": MODULE_PATHS.get(info.module_path),
            "module_outer_bits": info.module_outer_bits,
            "module_backward_fused": bool(info.module_backward_fused)}


_call_mod = None


def _call():
    """The CPython call module of the forward entry points
    (csrc/whtmix_pycall.c), bound to the functions of the loaded library.
    It is built with the library; there is no fallback."""
    global _call_mod
    if _call_mod is None:
        L = lib()
        try:
            from paper_2607_25234_amd import _whtmix_call as m
        except ImportError as e:
            raise ImportError("the binding's call module (_whtmix_call) is missing: build it "
                              "with `python -m paper_2607_25234_amd.build`") from e
        m.bind(ctypes.cast(L.whtmix_forward_ex, ctypes.c_void_p).value,
               ctypes.cast(L.whtmix_forward_separable, ctypes.c_void_p).value)
        _call_mod = m
    return _call_mod


def _opt_address(plan, events, spin_limit):
    """(structure, address) of the options argument; (None, 0) for NULL.  The
    caller keeps the structure alive across the call."""
    if events is None and not spin_limit and (plan == "auto" or plan == 0):
        return None, 0
    o = _options(plan, events, spin_limit)
    return o, ctypes.addressof(o)


def forward_raw(x_ptr: int, gain_ptr: int, y_ptr: int, B: int, N: int, C: int,
                dtype: int, stream: int, plan: str | int = "auto", events=None,
                spin_limit: int = 0) -> int:
    """Direct call of whtmix_forward_ex with integer pointers; returns the status."""
    o, addr = _opt_address(plan, events, spin_limit)
    st = _call().forward_ex(x_ptr, gain_ptr, y_ptr, B, N, C, dtype, stream, addr)
    del o
    return st


def forward_noalloc_raw(x_ptr: int, gain_ptr: int, y_ptr: int, B: int, N: int, C: int,
                        dtype: int, stream: int) -> int:
    """Direct call of whtmix_forward_noalloc (the fixed-scratch variant that
    allocates nothing); returns the status."""
    return lib().whtmix_forward_noalloc(x_ptr, gain_ptr, y_ptr, B, N, C, dtype, stream)


def padded_tokens(N: int) -> int:
    """N_pad: rows N .. N_pad-1 are taken as zeros so that H_N acts on a
    power-of-two length (section III-B)."""
    return 1 << max(0, (int(N) - 1).bit_length())


def forward_separable_raw(x_ptr: int, gt_ptr: int, gc_ptr: int, y_ptr: int, B: int, N: int,
                          C: int, dtype: int, stream: int, plan: str | int = "auto",
                          events=None) -> int:
    """Direct call of whtmix_forward_separable; returns the status."""
    o, addr = _opt_address(plan, events, 0)
    st = _call().forward_separable(x_ptr, gt_ptr, gc_ptr, y_ptr, B, N, C, dtype, stream, addr)
    del o
    return st


def _check(x, out):
    import torch

    if x.device.type != "cuda":
        raise ValueError("x must be on a GPU device")
    if x.dtype == torch.float32:
        dt = DTYPE_F32
    elif x.dtype == torch.bfloat16:
        dt = DTYPE_BF16
    else:
        raise TypeError(f"x must be float32 or bfloat16, got {x.dtype}")
    xx = x.unsqueeze(0) if x.dim() == 2 else x
    if xx.dim() != 3:
        raise ValueError("x must be [B, N, C] or [N, C]")
    if not xx.is_contiguous():
        raise ValueError("x must be contiguous")
    if out is None:
        out = torch.empty_like(x)
    elif out.shape != x.shape or out.dtype != x.dtype or not out.is_contiguous() \
            or out.device != x.device:
        raise ValueError("out must be a contiguous tensor like x")
    return xx, dt, out


def _gain(t, shape, x, what):
    import torch

    if t.device != x.device or t.dtype != torch.float32 or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous float32 tensor on x's device")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} shape {tuple(t.shape)} != {tuple(shape)}")


def forward(x, gain, out=None, plan: str | int = "auto", stream=None, events=None,
            spin_limit: int = 0):
    """y[b] = H_N (G o (H_N x[b] H_C)) H_C on the GPU (section III-B, eqs. (2)-(3)).

    x: torch tensor [B, N, C] or [N, C], float32 or bfloat16, on a ROCm device.
    gain: float32 [N_pad, C] (N_pad = N rounded up to a power of two; rows past
    N count as zeros) on the same device.  out: optional tensor like x (may
    be x itself for in-place).  stream: a torch.cuda.Stream (default: the
    current stream)."""
    import torch

    xx, dt, out = _check(x, out)
    B, N, C = xx.shape
    _gain(gain, (padded_tokens(N), C), x, "gain")
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    with torch.cuda.device(x.device):
        status = forward_raw(xx.data_ptr(), gain.data_ptr(), out.data_ptr(), B, N, C, dt,
                             st.cuda_stream, plan, events, spin_limit)
    if status != SUCCESS:
        raise WhtmixError(status, "whtmix_forward")
    return out


def forward_separable(x, log_gain_tokens, log_gain_channels, out=None,
                      plan: str | int = "auto", stream=None, events=None):
    """The paper's parametrisation (eq. (2) then eq. (3)) with log-domain gains:
    log_gain_tokens float32 [N_pad], log_gain_channels float32 [C]."""
    import torch

    xx, dt, out = _check(x, out)
    B, N, C = xx.shape
    _gain(log_gain_tokens, (padded_tokens(N),), x, "log_gain_tokens")
    _gain(log_gain_channels, (C,), x, "log_gain_channels")
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    with torch.cuda.device(x.device):
        status = forward_separable_raw(xx.data_ptr(), log_gain_tokens.data_ptr(),
                                       log_gain_channels.data_ptr(), out.data_ptr(), B, N, C,
                                       dt, st.cuda_stream, plan, events)
    if status != SUCCESS:
        raise WhtmixError(status, "whtmix_forward_separable")
    return out


def module_forward_raw(x_ptr: int, w_in_ptr: int, gain_ptr: int, w_out_ptr: int, y_ptr: int,
                       B: int, N: int, C: int, dtype: int, stream: int,
                       plan: str | int = "auto", events=None) -> int:
    """Direct call of whtmix_module_forward; returns the status."""
    return lib().whtmix_module_forward(x_ptr, w_in_ptr, gain_ptr, w_out_ptr, y_ptr, B, N, C,
                                       dtype, stream, _opt_arg(plan, events))


def module_forward_separable_raw(x_ptr: int, w_in_ptr: int, gt_ptr: int, gc_ptr: int,
                                 w_out_ptr: int, y_ptr: int, B: int, N: int, C: int,
                                 dtype: int, stream: int, plan: str | int = "auto",
                                 events=None) -> int:
    """Direct call of whtmix_module_forward_separable; returns the status."""
    return lib().whtmix_module_forward_separable(x_ptr, w_in_ptr, gt_ptr, gc_ptr, w_out_ptr,
                                                 y_ptr, B, N, C, dtype, stream,
                                                 _opt_arg(plan, events))


def _weight(w, C, x, what):
    if w.device != x.device or w.dtype != x.dtype or not w.is_contiguous():
        raise ValueError(f"{what} must be a contiguous tensor of x's dtype on x's device")
    if tuple(w.shape) != (C, C):
        raise ValueError(f"{what} shape {tuple(w.shape)} != {(C, C)}")


def module_forward(x, w_in, gain, w_out, out=None, plan: str | int = "auto", stream=None,
                   events=None):
    """The whole block of section III-B, eqs. (1)-(4): Y = mixer(X W_in) W_out with
    the joint gain.  w_in, w_out: [C, C] tensors of x's dtype (Z[n][j] = sum_i
    X[n][i] W_in[i][j]); gain: float32 [N_pad, C]."""
    import torch

    xx, dt, out = _check(x, out)
    B, N, C = xx.shape
    _weight(w_in, C, x, "w_in")
    _weight(w_out, C, x, "w_out")
    _gain(gain, (padded_tokens(N), C), x, "gain")
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    with torch.cuda.device(x.device):
        status = module_forward_raw(xx.data_ptr(), w_in.data_ptr(), gain.data_ptr(),
                                    w_out.data_ptr(), out.data_ptr(), B, N, C, dt,
                                    st.cuda_stream, plan, events)
    if status != SUCCESS:
        raise WhtmixError(status, "whtmix_module_forward")
    return out


def module_forward_separable(x, w_in, log_gain_tokens, log_gain_channels, w_out, out=None,
                             plan: str | int = "auto", stream=None, events=None):
    """The whole block with the paper's log-domain gains (eqs. (1)-(4))."""
    import torch

    xx, dt, out = _check(x, out)
    B, N, C = xx.shape
    _weight(w_in, C, x, "w_in")
    _weight(w_out, C, x, "w_out")
    _gain(log_gain_tokens, (padded_tokens(N),), x, "log_gain_tokens")
    _gain(log_gain_channels, (C,), x, "log_gain_channels")
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    with torch.cuda.device(x.device):
        status = module_forward_separable_raw(xx.data_ptr(), w_in.data_ptr(),
                                              log_gain_tokens.data_ptr(),
                                              log_gain_channels.data_ptr(), w_out.data_ptr(),
                                              out.data_ptr(), B, N, C, dt, st.cuda_stream,
                                              plan, events)
    if status != SUCCESS:
        raise WhtmixError(status, "whtmix_module_forward_separable")
    return out


def backward_raw(x_ptr, dy_ptr, gain_ptr, dx_ptr, dgain_ptr, B, N, C, dtype, stream,
                 plan: str | int = "auto", events=None) -> int:
    """Direct call of whtmix_backward (0 for a skipped output); returns the status."""
    return lib().whtmix_backward(x_ptr, dy_ptr, gain_ptr, dx_ptr, dgain_ptr, B, N, C, dtype,
                                 stream, _opt_arg(plan, events))


def backward_separable_raw(x_ptr, dy_ptr, gt_ptr, gc_ptr, dx_ptr, dgt_ptr, dgc_ptr, B, N, C,
                           dtype, stream, plan: str | int = "auto", events=None) -> int:
    """Direct call of whtmix_backward_separable; returns the status."""
    return lib().whtmix_backward_separable(x_ptr, dy_ptr, gt_ptr, gc_ptr, dx_ptr, dgt_ptr,
                                           dgc_ptr, B, N, C, dtype, stream, _opt_arg(plan, events))


def _same(a, x, what):
    if a.shape != x.shape or a.dtype != x.dtype or a.device != x.device or not a.is_contiguous():
        raise ValueError(f"{what} must be a contiguous tensor like x")


def backward(x, dy, gain, want_dx: bool = True, want_dgain: bool = True, dx=None,
             plan: str | int = "auto", stream=None):
    """Gradients through forward(x, gain) for the upstream gradient dy:
    returns (dx, dgain); dx = the mixer applied to dy, dgain [N_pad, C]
    float32 = sum_b T(x_b) o T(dy_b).  An output not wanted is None."""
    import torch

    xx, dt, _ = _check(x, x)
    _same(dy, x, "dy")
    B, N, C = xx.shape
    _gain(gain, (padded_tokens(N), C), x, "gain")
    if want_dx and dx is None:
        dx = torch.empty_like(dy)
    if dx is not None:
        _same(dx, x, "dx")
    dgain = torch.empty_like(gain) if want_dgain else None
    if dx is None and dgain is None:
        raise ValueError("nothing to compute")
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    with torch.cuda.device(x.device):
        status = backward_raw(xx.data_ptr(), dy.data_ptr(), gain.data_ptr(),
                              dx.data_ptr() if dx is not None else 0,
                              dgain.data_ptr() if dgain is not None else 0, B, N, C, dt,
                              st.cuda_stream, plan)
    if status != SUCCESS:
        raise WhtmixError(status, "whtmix_backward")
    return dx, dgain


def backward_separable(x, dy, log_gain_tokens, log_gain_channels, want_dx: bool = True,
                       want_dgains: bool = True, dx=None, plan: str | int = "auto",
                       stream=None):
    """Gradients through forward_separable: returns (dx, d_log_gain_tokens,
    d_log_gain_channels); outputs not wanted are None."""
    import torch

    xx, dt, _ = _check(x, x)
    _same(dy, x, "dy")
    B, N, C = xx.shape
    _gain(log_gain_tokens, (padded_tokens(N),), x, "log_gain_tokens")
    _gain(log_gain_channels, (C,), x, "log_gain_channels")
    if want_dx and dx is None:
        dx = torch.empty_like(dy)
    if dx is not None:
        _same(dx, x, "dx")
    dgt = torch.empty_like(log_gain_tokens) if want_dgains else None
    dgc = torch.empty_like(log_gain_channels) if want_dgains else None
    if dx is None and dgt is None:
        raise ValueError("nothing to compute")
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    with torch.cuda.device(x.device):
        status = backward_separable_raw(
            xx.data_ptr(), dy.data_ptr(), log_gain_tokens.data_ptr(),
            log_gain_channels.data_ptr(), dx.data_ptr() if dx is not None else 0,
            dgt.data_ptr() if dgt is not None else 0, dgc.data_ptr() if dgc is not None else 0,
            B, N, C, dt, st.cuda_stream, plan)
    if status != SUCCESS:
        raise WhtmixError(status, "whtmix_backward_separable")
    return dx, dgt, dgc


def module_backward_raw(x_ptr, w_in_ptr, gain_ptr, w_out_ptr, dy_ptr, dx_ptr, dw_in_ptr,
                        dw_out_ptr, dgain_ptr, B, N, C, dtype, stream,
                        plan: str | int = "auto", events=None) -> int:
    """Direct call of whtmix_module_backward; returns the status."""
    return lib().whtmix_module_backward(x_ptr, w_in_ptr, gain_ptr, w_out_ptr, dy_ptr, dx_ptr,
                                        dw_in_ptr, dw_out_ptr, dgain_ptr, B, N, C, dtype, stream,
                                        _opt_arg(plan, events))


def module_backward_separable_raw(x_ptr, w_in_ptr, gt_ptr, gc_ptr, w_out_ptr, dy_ptr, dx_ptr,
                                  dw_in_ptr, dw_out_ptr, dgt_ptr, dgc_ptr, B, N, C, dtype,
                                  stream, plan: str | int = "auto", events=None) -> int:
    """Direct call of whtmix_module_backward_separable; returns the status."""
    return lib().whtmix_module_backward_separable(x_ptr, w_in_ptr, gt_ptr, gc_ptr, w_out_ptr,
                                                  dy_ptr, dx_ptr, dw_in_ptr, dw_out_ptr, dgt_ptr,
                                                  dgc_ptr, B, N, C, dtype, stream,
                                                  _opt_arg(plan, events))


def module_backward(x, w_in, gain, w_out, dy, want_dgain: bool = True, dx=None,
                    plan: str | int = "auto", stream=None):
    """Gradients through module_forward for the upstream gradient dy: returns
    (dx, dw_in, dw_out, dgain), the weight and gain gradients in float32
    (dgain None when not wanted)."""
    import torch

    xx, dt, _ = _check(x, x)
    _same(dy, x, "dy")
    B, N, C = xx.shape
    _weight(w_in, C, x, "w_in")
    _weight(w_out, C, x, "w_out")
    _gain(gain, (padded_tokens(N), C), x, "gain")
    if dx is None:
        dx = torch.empty_like(dy)
    _same(dx, x, "dx")
    f32 = dict(dtype=torch.float32, device=x.device)
    dw_in, dw_out = torch.empty((C, C), **f32), torch.empty((C, C), **f32)
    dgain = torch.empty_like(gain) if want_dgain else None
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    with torch.cuda.device(x.device):
        status = module_backward_raw(xx.data_ptr(), w_in.data_ptr(), gain.data_ptr(),
                                     w_out.data_ptr(), dy.data_ptr(), dx.data_ptr(),
                                     dw_in.data_ptr(), dw_out.data_ptr(),
                                     dgain.data_ptr() if dgain is not None else 0, B, N, C, dt,
                                     st.cuda_stream, plan)
    if status != SUCCESS:
        raise WhtmixError(status, "whtmix_module_backward")
    return dx, dw_in, dw_out, dgain


def module_backward_separable(x, w_in, log_gain_tokens, log_gain_channels, w_out, dy,
                              want_dgains: bool = True, dx=None, plan: str | int = "auto",
                              stream=None):
    """Gradients through module_forward_separable: returns (dx, dw_in, dw_out,
    d_log_gain_tokens, d_log_gain_channels)."""
    import torch

    xx, dt, _ = _check(x, x)
    _same(dy, x, "dy")
    B, N, C = xx.shape
    _weight(w_in, C, x, "w_in")
    _weight(w_out, C, x, "w_out")
    _gain(log_gain_tokens, (padded_tokens(N),), x, "log_gain_tokens")
    _gain(log_gain_channels, (C,), x, "log_gain_channels")
    if dx is None:
        dx = torch.empty_like(dy)
    _same(dx, x, "dx")
    f32 = dict(dtype=torch.float32, device=x.device)
    dw_in, dw_out = torch.empty((C, C), **f32), torch.empty((C, C), **f32)
    dgt = torch.empty_like(log_gain_tokens) if want_dgains else None
    dgc = torch.empty_like(log_gain_channels) if want_dgains else None
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    with torch.cuda.device(x.device):
        status = module_backward_separable_raw(
            xx.data_ptr(), w_in.data_ptr(), log_gain_tokens.data_ptr(),
            log_gain_channels.data_ptr(), w_out.data_ptr(), dy.data_ptr(), dx.data_ptr(),
            dw_in.data_ptr(), dw_out.data_ptr(), dgt.data_ptr() if dgt is not None else 0,
            dgc.data_ptr() if dgc is not None else 0, B, N, C, dt, st.cuda_stream, plan)
    if status != SUCCESS:
        raise WhtmixError(status, "whtmix_module_backward_separable")
    return dx, dw_in, dw_out, dgt, dgc


def release_workspaces() -> None:
    st = lib().whtmix_release_workspaces()
    if st != SUCCESS:
        raise WhtmixError(st, "whtmix_release_workspaces")
