"""ctypes binding for the WHTMix CPU oracle -- TEST INFRASTRUCTURE ONLY.

The oracle (``whtmix_oracle.c``) is a plain double-precision statement of the
Walsh-Hadamard token mixer of section III-B (eqs. (2)-(3)).  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this module.  The product path (``paper_2607_25234_amd``) never imports it.

``build()`` compiles the C source with gcc into ``liboracle.so`` beside it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "whtmix_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

_lib = None


def build(src: str = SRC, out: str = LIB, extra_flags: tuple = ()) -> str:
    """Compile the oracle with gcc (OpenMP, no fast-math, no FP contraction)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
           *extra_flags, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def load(path: str = LIB):
    """Load a compiled oracle library (building the default one if absent)."""
    global _lib
    if path == LIB and _lib is not None:
        return _lib
    if not os.path.exists(path):
        if path != LIB:
            raise FileNotFoundError(path)
        build()
    lib = ctypes.CDLL(path)
    dp = ctypes.POINTER(ctypes.c_double)
    L = ctypes.c_long
    lib.oracle_whtmix.argtypes = [dp, dp, dp, L, L, L]
    lib.oracle_whtmix.restype = ctypes.c_int
    lib.oracle_whtmix_separable.argtypes = [dp, dp, dp, dp, L, L, L]
    lib.oracle_whtmix_separable.restype = ctypes.c_int
    lib.oracle_fwht.argtypes = [dp, L]
    lib.oracle_fwht.restype = ctypes.c_int
    lib.oracle_whtmix_grad.argtypes = [dp, dp, dp, dp, dp, L, L, L]
    lib.oracle_whtmix_grad.restype = ctypes.c_int
    lib.oracle_whtmix_grad_separable.argtypes = [dp, dp, dp, dp, dp, dp, dp, L, L, L]
    lib.oracle_whtmix_grad_separable.restype = ctypes.c_int
    lib.oracle_whtmix_module.argtypes = [dp, dp, dp, dp, dp, L, L, L]
    lib.oracle_whtmix_module.restype = ctypes.c_int
    lib.oracle_whtmix_module_separable.argtypes = [dp, dp, dp, dp, dp, dp, L, L, L]
    lib.oracle_whtmix_module_separable.restype = ctypes.c_int
    lib.oracle_whtmix_module_grad.argtypes = [dp, dp, dp, dp, dp, dp, dp, dp, dp, L, L, L]
    lib.oracle_whtmix_module_grad.restype = ctypes.c_int
    lib.oracle_whtmix_module_grad_separable.argtypes = [dp] * 11 + [L, L, L]
    lib.oracle_whtmix_module_grad_separable.restype = ctypes.c_int
    lib.oracle_threads.argtypes = []
    lib.oracle_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_threads.restype = ctypes.c_int
    if path == LIB:
        _lib = lib
    return lib


def padded(n: int) -> int:
    """P: the token count rounded up to a power of two (zero padding)."""
    p = 1
    while p < n:
        p *= 2
    return p


def _dptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _as_f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


class Oracle:
    """Thin wrapper over one compiled oracle library (default: liboracle.so)."""

    def __init__(self, path: str = LIB):
        self.lib = load(path)

    def whtmix(self, x, g) -> np.ndarray:
        """Y[b] = H_N (G o (H_N X[b] H_C)) H_C in float64.

        x: [B, N, C] or [N, C]; g: [P, C] with P = N rounded up to a power of
        two (the token axis is zero-padded).  Returns float64 of x's shape."""
        x64 = _as_f64(x)
        squeeze = x64.ndim == 2
        if squeeze:
            x64 = x64[None]
        B, N, C = x64.shape
        g64 = _as_f64(g)
        if g64.shape != (padded(N), C):
            raise ValueError(f"gain shape {g64.shape} != {(padded(N), C)}")
        y = np.empty_like(x64)
        rc = self.lib.oracle_whtmix(_dptr(x64), _dptr(g64), _dptr(y), B, N, C)
        if rc != 0:
            raise ValueError(f"oracle_whtmix rejected shape {(B, N, C)}")
        return y[0] if squeeze else y

    def whtmix_separable(self, x, g_t, g_c) -> np.ndarray:
        """The paper's eq. (2) then eq. (3) with log-domain gains g_t[P], g_c[C]."""
        x64 = _as_f64(x)
        squeeze = x64.ndim == 2
        if squeeze:
            x64 = x64[None]
        B, N, C = x64.shape
        gt = _as_f64(g_t).reshape(-1)
        gc = _as_f64(g_c).reshape(-1)
        if gt.shape != (padded(N),) or gc.shape != (C,):
            raise ValueError("g_t must have P entries and g_c C entries")
        y = np.empty_like(x64)
        rc = self.lib.oracle_whtmix_separable(_dptr(x64), _dptr(gt), _dptr(gc),
                                              _dptr(y), B, N, C)
        if rc != 0:
            raise ValueError(f"oracle_whtmix_separable rejected {(B, N, C)}")
        return y[0] if squeeze else y

    def whtmix_grad(self, x, dy, g):
        """(dX, dG) for upstream gradient dy through the joint-gain mixer:
        dX = the mixer applied to dy, dG = sum_b (H X_b H) o (H dY_b H)."""
        x64, dy64 = _as_f64(x), _as_f64(dy)
        squeeze = x64.ndim == 2
        if squeeze:
            x64, dy64 = x64[None], dy64[None]
        B, N, C = x64.shape
        if dy64.shape != x64.shape:
            raise ValueError("dy must have x's shape")
        g64 = _as_f64(g)
        if g64.shape != (padded(N), C):
            raise ValueError(f"gain shape {g64.shape} != {(padded(N), C)}")
        dx = np.empty_like(x64)
        dg = np.empty_like(g64)
        rc = self.lib.oracle_whtmix_grad(_dptr(x64), _dptr(dy64), _dptr(g64), _dptr(dx),
                                         _dptr(dg), B, N, C)
        if rc != 0:
            raise ValueError(f"oracle_whtmix_grad rejected shape {(B, N, C)}")
        return (dx[0] if squeeze else dx), dg

    def whtmix_grad_separable(self, x, dy, g_t, g_c):
        """(dX, dg_t, dg_c) for upstream gradient dy through eq. (2)-(3)."""
        x64, dy64 = _as_f64(x), _as_f64(dy)
        squeeze = x64.ndim == 2
        if squeeze:
            x64, dy64 = x64[None], dy64[None]
        B, N, C = x64.shape
        if dy64.shape != x64.shape:
            raise ValueError("dy must have x's shape")
        gt = _as_f64(g_t).reshape(-1)
        gc = _as_f64(g_c).reshape(-1)
        if gt.shape != (padded(N),) or gc.shape != (C,):
            raise ValueError("g_t must have P entries and g_c C entries")
        dx = np.empty_like(x64)
        dgt = np.empty_like(gt)
        dgc = np.empty_like(gc)
        rc = self.lib.oracle_whtmix_grad_separable(_dptr(x64), _dptr(dy64), _dptr(gt),
                                                   _dptr(gc), _dptr(dx), _dptr(dgt),
                                                   _dptr(dgc), B, N, C)
        if rc != 0:
            raise ValueError(f"oracle_whtmix_grad_separable rejected {(B, N, C)}")
        return (dx[0] if squeeze else dx), dgt, dgc

    def whtmix_module(self, x, w_in, g, w_out) -> np.ndarray:
        """The full block, eqs. (1)-(4): Y = mixer(X W_in) W_out (joint gain)."""
        x64 = _as_f64(x)
        squeeze = x64.ndim == 2
        if squeeze:
            x64 = x64[None]
        B, N, C = x64.shape
        wi, wo, g64 = _as_f64(w_in), _as_f64(w_out), _as_f64(g)
        if wi.shape != (C, C) or wo.shape != (C, C) or g64.shape != (padded(N), C):
            raise ValueError("w_in, w_out must be [C, C] and g [P, C]")
        y = np.empty_like(x64)
        rc = self.lib.oracle_whtmix_module(_dptr(x64), _dptr(wi), _dptr(g64), _dptr(wo),
                                           _dptr(y), B, N, C)
        if rc != 0:
            raise ValueError(f"oracle_whtmix_module rejected {(B, N, C)}")
        return y[0] if squeeze else y

    def whtmix_module_separable(self, x, w_in, g_t, g_c, w_out) -> np.ndarray:
        """The full block with the paper's log-domain gains."""
        x64 = _as_f64(x)
        squeeze = x64.ndim == 2
        if squeeze:
            x64 = x64[None]
        B, N, C = x64.shape
        wi, wo = _as_f64(w_in), _as_f64(w_out)
        gt, gc = _as_f64(g_t).reshape(-1), _as_f64(g_c).reshape(-1)
        if wi.shape != (C, C) or wo.shape != (C, C) or gt.shape != (padded(N),) \
                or gc.shape != (C,):
            raise ValueError("bad weight or gain shapes")
        y = np.empty_like(x64)
        rc = self.lib.oracle_whtmix_module_separable(_dptr(x64), _dptr(wi), _dptr(gt),
                                                     _dptr(gc), _dptr(wo), _dptr(y), B, N, C)
        if rc != 0:
            raise ValueError(f"oracle_whtmix_module_separable rejected {(B, N, C)}")
        return y[0] if squeeze else y

    def _module_grad_args(self, x, w_in, w_out, dy):
        x64, dy64 = _as_f64(x), _as_f64(dy)
        squeeze = x64.ndim == 2
        if squeeze:
            x64, dy64 = x64[None], dy64[None]
        B, N, C = x64.shape
        wi, wo = _as_f64(w_in), _as_f64(w_out)
        if wi.shape != (C, C) or wo.shape != (C, C) or dy64.shape != x64.shape:
            raise ValueError("w_in, w_out must be [C, C] and dy like x")
        return x64, dy64, wi, wo, squeeze, (B, N, C)

    def whtmix_module_grad(self, x, w_in, g, w_out, dy):
        """(dX, dW_in, dW_out, dG) of the block (joint gain) for upstream dY."""
        x64, dy64, wi, wo, squeeze, (B, N, C) = self._module_grad_args(x, w_in, w_out, dy)
        g64 = _as_f64(g)
        if g64.shape != (padded(N), C):
            raise ValueError("gain must be [P, C]")
        dx, dwi, dwo, dg = (np.empty_like(x64), np.empty_like(wi), np.empty_like(wo),
                            np.empty_like(g64))
        rc = self.lib.oracle_whtmix_module_grad(_dptr(x64), _dptr(wi), _dptr(g64), _dptr(wo),
                                                _dptr(dy64), _dptr(dx), _dptr(dwi),
                                                _dptr(dwo), _dptr(dg), B, N, C)
        if rc != 0:
            raise ValueError(f"oracle_whtmix_module_grad rejected {(B, N, C)}")
        return (dx[0] if squeeze else dx), dwi, dwo, dg

    def whtmix_module_grad_separable(self, x, w_in, g_t, g_c, w_out, dy):
        """(dX, dW_in, dW_out, dg_t, dg_c) of the block with log gains."""
        x64, dy64, wi, wo, squeeze, (B, N, C) = self._module_grad_args(x, w_in, w_out, dy)
        gt, gc = _as_f64(g_t).reshape(-1), _as_f64(g_c).reshape(-1)
        if gt.shape != (padded(N),) or gc.shape != (C,):
            raise ValueError("g_t must have P entries and g_c C entries")
        dx, dwi, dwo = np.empty_like(x64), np.empty_like(wi), np.empty_like(wo)
        dgt, dgc = np.empty_like(gt), np.empty_like(gc)
        rc = self.lib.oracle_whtmix_module_grad_separable(
            _dptr(x64), _dptr(wi), _dptr(gt), _dptr(gc), _dptr(wo), _dptr(dy64), _dptr(dx),
            _dptr(dwi), _dptr(dwo), _dptr(dgt), _dptr(dgc), B, N, C)
        if rc != 0:
            raise ValueError(f"oracle_whtmix_module_grad_separable rejected {(B, N, C)}")
        return (dx[0] if squeeze else dx), dwi, dwo, dgt, dgc

    def fwht(self, v) -> np.ndarray:
        """Unnormalised Sylvester butterfly of a 1-D vector (H_n v, +/-1 H)."""
        v64 = _as_f64(v).copy()
        if v64.ndim != 1:
            raise ValueError("fwht takes a 1-D vector")
        rc = self.lib.oracle_fwht(_dptr(v64), v64.shape[0])
        if rc != 0:
            raise ValueError("length must be a power of two")
        return v64

    def threads(self) -> int:
        """OpenMP threads the oracle's parallel loops use."""
        return int(self.lib.oracle_threads())

    def set_threads(self, n: int) -> int:
        """Use n OpenMP threads from now on; returns the previous count."""
        return int(self.lib.oracle_set_threads(int(n)))


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def whtmix(x, g) -> np.ndarray:
    return default().whtmix(x, g)


def whtmix_separable(x, g_t, g_c) -> np.ndarray:
    return default().whtmix_separable(x, g_t, g_c)


def fwht(v) -> np.ndarray:
    return default().fwht(v)
