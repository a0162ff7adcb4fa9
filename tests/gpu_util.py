"""Helpers shared by the GPU tests (not collected by pytest)."""
from __future__ import annotations

import sys

import numpy as np

TOL = {"f32": 1e-5, "bf16": 2e-2}
# The bar the arithmetic itself allows (checked beside TOL): float32 I/O as
# TOL; bf16 I/O rounds y once to nearest even, at most 2^-8 of each output
# element (bf16 keeps 8 significant bits), so at most 2^-8 of max|r|
# normwise, plus float32 accumulation (~1e-7 normwise measured; 1e-5 allowed).
DERIVED = {"f32": 1e-5, "bf16": 2.0 ** -8 + 1e-5}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def device():
    import pytest
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    return torch.device("cuda:0")


def to_device(x: np.ndarray, dtype: str, dev):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev)
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def to_host(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy()


def run_gpu(x: np.ndarray, g: np.ndarray, dtype: str, dev, plan="auto") -> np.ndarray:
    import torch
    from paper_2607_25234_amd import whtmix
    xd = to_device(x, dtype, dev)
    gd = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(dev)
    y = whtmix.forward(xd, gd, plan=plan)
    torch.cuda.synchronize(dev)
    return to_host(y)


def errors(y: np.ndarray, ref: np.ndarray) -> tuple[float, float]:
    """(normwise max relative error, rms relative error)."""
    y = np.asarray(y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0, 0.0
    den = max(float(np.max(np.abs(ref))), 1e-300)
    d = y - ref
    rms_den = max(float(np.sqrt(np.mean(ref * ref))), 1e-300)
    return float(np.max(np.abs(d)) / den), float(np.sqrt(np.mean(d * d)) / rms_den)


def run_gpu_separable(x: np.ndarray, gt: np.ndarray, gc: np.ndarray, dtype: str, dev,
                      plan="auto") -> np.ndarray:
    import torch
    from paper_2607_25234_amd import whtmix
    xd = to_device(x, dtype, dev)
    gtd = torch.from_numpy(np.ascontiguousarray(gt, dtype=np.float32)).to(dev)
    gcd = torch.from_numpy(np.ascontiguousarray(gc, dtype=np.float32)).to(dev)
    y = whtmix.forward_separable(xd, gtd, gcd, plan=plan)
    torch.cuda.synchronize(dev)
    return to_host(y)



def random_cases(n: int, seed: int, max_elems: int = 1 << 21) -> list[tuple]:
    """Seeded (B, N, C, dtype) cases over every plan's range: N*C from 1 to
    2^20 elements, token counts that are powers of two or not, 1-6 slices
    (B * N_pad * C <= max_elems), float32 and bf16 alternately."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        K = int(rng.integers(0, 21))
        c = int(rng.integers(0, min(K, 9) + 1))
        hi = 1 << (K - c)
        N = hi if rng.random() < 0.5 or hi == 1 else int(rng.integers(hi // 2 + 1, hi + 1))
        B = int(rng.integers(1, 7))
        while B > 1 and B * hi * (1 << c) > max_elems:
            B -= 1
        cases.append((B, N, 1 << c, "bf16" if i % 2 else "f32"))
    return cases


def case_ids(cases) -> list[str]:
    return [f"r{i:02d}-{b}x{n}x{c}-{d}" for i, (b, n, c, d) in enumerate(cases)]
