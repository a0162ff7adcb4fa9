"""Seeded synthetic WHTMix inputs (shapes and distributions only, no mixer arithmetic).

Both sides of every parity check draw their inputs here: the HIP path receives
them as device tensors, the CPU oracle as float64 arrays.  Nothing in this
module computes any part of the mixer.

Workloads (X: [B, N, C] tokens x channels, G: [N, C] float32 gain):

* ``image1k_f32``     B=1,  N=1024   (32x32 grid, row-major),       C=64,  fp32
* ``stereo16k_f32``   B=2,  N=16384  (two 64x128 view grids),       C=128, fp32
* ``stereo64k_bf16``  B=4,  N=65536  (two 128x256 view grids),      C=128, bf16
* ``text4k_f32``      B=32, N=4096   (embedded integer tokens),     C=64,  fp32
* ``stereo256k_bf16`` B=1,  N=262144 (two 256x512 view grids),      C=256, bf16

The stereo workloads stand in for the CNN-plus-positional-encoding features of
the stereo backbone (section III-A: N = 2 (H/8)(W/8) joint tokens of the left
and right views), the 1k and 4k ones for the byte-level image and text
sequence-classification tasks (section IV-D).  No dataset item is reproduced:
X ~ N(0, 1) (or embeddings of uniform random integer tokens through a
N(0, 0.02) table for the text workload) and G ~ U(0.5, 1.5), drawn in float32 with
numpy's PCG64 generator seeded per workload, in the order X then G (text
workload: table, tokens, G).  bf16 workloads round X to bf16 with round-to-nearest-even
before either side sees it, so both sides receive identical values.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    N: int
    C: int
    dtype: str          # "f32" or "bf16": the element type of X and Y
    seed: int
    x_dist: str = "normal"   # "normal" or "embed"
    note: str = ""

    @property
    def elements(self) -> int:
        return self.B * self.N * self.C

    @property
    def io_bytes(self) -> int:
        """Ideal HBM bytes of one call: read X, read G once, write Y."""
        s = 4 if self.dtype == "f32" else 2
        return self.elements * 2 * s + 4 * self.N * self.C


WORKLOADS = {
    w.name: w
    for w in [
        Workload("image1k_f32", 1, 1024, 64, "f32", 1, "normal",
                 "32x32 feature grid, row-major"),
        Workload("stereo16k_f32", 2, 16384, 128, "f32", 2, "normal",
                 "two 64x128 view grids concatenated along tokens"),
        Workload("stereo64k_bf16", 4, 65536, 128, "bf16", 3, "normal",
                 "two 128x256 view grids concatenated, bf16 in/out"),
        Workload("text4k_f32", 32, 4096, 64, "f32", 4, "embed",
                 "uniform integer tokens in [0,256) through a N(0,0.02) table"),
        Workload("stereo256k_bf16", 1, 262144, 256, "bf16", 5, "normal",
                 "two 256x512 view grids concatenated, bf16 in/out"),
    ]
}

# The workload the benchmark times (the N=65536, C=128 bf16 configuration).
BENCH_WORKLOAD = "stereo64k_bf16"


def round_to_bf16(x: np.ndarray, inplace: bool = False) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), kept as float32."""
    out = x if inplace else np.array(x, dtype=np.float32, copy=True, order="C")
    if out.dtype != np.float32 or not out.flags.c_contiguous:
        raise ValueError("round_to_bf16 works on contiguous float32 arrays")
    flat = out.reshape(-1)
    u = flat.view(np.uint32)
    step = 1 << 20
    lsb = np.empty(min(step, u.size), dtype=np.uint32)
    for i in range(0, u.size, step):
        seg = u[i:i + step]
        t = lsb[:seg.size]
        nan = np.isnan(flat[i:i + step])
        np.right_shift(seg, 16, out=t)
        np.bitwise_and(t, 1, out=t)
        seg += t          # finite values: u + lsb + 0x7FFF stays below 2^32
        seg += 0x7FFF
        seg &= 0xFFFF0000
        if nan.any():
            flat[i:i + step][nan] = np.float32("nan")
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The uint16 bf16 bit patterns of float32 values that are exactly bf16."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("values are not exactly representable in bf16")
    return (u >> 16).astype(np.uint16)


def draw(B: int, N: int, C: int, dtype: str = "f32", seed: int = 0,
         x_dist: str = "normal", gain_lo: float = 0.5, gain_hi: float = 1.5):
    """Return (x, g): x float32 [B, N, C] (bf16-rounded if dtype == "bf16"),
    g float32 [N, C] ~ U(gain_lo, gain_hi)."""
    rng = np.random.default_rng(seed)
    if x_dist == "normal":
        x = rng.standard_normal((B, N, C), dtype=np.float32)
    elif x_dist == "embed":
        table = np.float32(0.02) * rng.standard_normal((256, C), dtype=np.float32)
        tokens = rng.integers(0, 256, size=(B, N))
        x = table[tokens]
    else:
        raise ValueError(f"unknown x distribution {x_dist!r}")
    g = rng.random((N, C), dtype=np.float32)
    g *= np.float32(gain_hi - gain_lo)
    g += np.float32(gain_lo)
    if dtype == "bf16":
        x = round_to_bf16(x, inplace=True)
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype!r}")
    return np.ascontiguousarray(x), np.ascontiguousarray(g)


def draw_log_gains(P: int, C: int, seed: int):
    """Seeded log-domain gains for the separable form: g_t[P], g_c[C], each
    ~ N(0, 0.3^2), float32 (the paper initialises them at zero)."""
    rng = np.random.default_rng(seed)
    gt = np.float32(0.3) * rng.standard_normal(P, dtype=np.float32)
    gc = np.float32(0.3) * rng.standard_normal(C, dtype=np.float32)
    return gt, gc


def draw_weights(C: int, dtype: str, seed: int):
    """Seeded projection weights of the block (eqs. (1), (4)): W_in, W_out
    float32 [C, C] ~ N(0, 1/C) (variance-preserving, as a trained projection
    would roughly be), rounded to bf16 when dtype == "bf16"."""
    rng = np.random.default_rng(seed)
    s = np.float32(1.0 / np.sqrt(C))
    w_in = s * rng.standard_normal((C, C), dtype=np.float32)
    w_out = s * rng.standard_normal((C, C), dtype=np.float32)
    if dtype == "bf16":
        w_in = round_to_bf16(w_in, inplace=True)
        w_out = round_to_bf16(w_out, inplace=True)
    return np.ascontiguousarray(w_in), np.ascontiguousarray(w_out)


def inputs(w: Workload | str):
    """Inputs of a named workload, as (x float32 [B,N,C], g float32 [N,C])."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    return draw(w.B, w.N, w.C, w.dtype, w.seed, w.x_dist)
