"""Build the WHTMix HIP library (libwhtmix.so) in-tree for gfx950.

    python -m paper_2607_25234_amd.build

Compiles every HIP / C++ source under csrc/ with hipcc, one process per
source in parallel, and links them into one shared library beside this file.
Packed FP32 instructions are disabled for all device code.  Then builds the
binding's CPython call module (csrc/whtmix_pycall.c, host code only) with the
host C compiler.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import sysconfig
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libwhtmix.so")
PYCALL = os.path.join(HERE, "_whtmix_call" + sysconfig.get_config_var("EXT_SUFFIX"))
ARCH = "gfx950"

COMPILE_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-fvisibility=hidden",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}",
    f"-I{CSRC}",
]
LINK_FLAGS = [f"--offload-arch={ARCH}", "-shared", "-fPIC"]


def sources() -> list[str]:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) +
                  glob.glob(os.path.join(CSRC, "*.cpp")))


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def _run(cmd: list[str], verbose: bool, what: str) -> None:
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"{cmd[0]} failed: {what}")


def build_pycall(out: str = PYCALL, verbose: bool = False) -> str:
    """The CPython call module of the forward entry points (no HIP code)."""
    cc = os.environ.get("CC", "gcc")
    src = os.path.join(CSRC, "whtmix_pycall.c")
    _run([cc, "-O2", "-shared", "-fPIC", "-Wall", "-Wextra", "-Werror",
          f"-I{sysconfig.get_paths()['include']}", src, "-o", out + ".tmp"], verbose, src)
    os.replace(out + ".tmp", out)
    return out


def build(out: str = LIB, extra: tuple = (), verbose: bool = False, jobs: int = 0) -> str:
    """Compile each source to an object (in parallel), then link."""
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, min(16, os.cpu_count() or 1)))
    with tempfile.TemporaryDirectory(prefix="whtmix_build_") as tmp:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in srcs]
        cmds = [[hipcc(), *COMPILE_FLAGS, *extra, "-c", s, "-o", o] for s, o in zip(srcs, objs)]
        with ThreadPoolExecutor(max_workers=jobs) as pool:
            list(pool.map(lambda c: _run(c, verbose, c[-3]), cmds))
        _run([hipcc(), *LINK_FLAGS, *extra, *objs, "-o", out + ".tmp"], verbose, "link")
    os.replace(out + ".tmp", out)
    if out == LIB:
        build_pycall(verbose=verbose)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
