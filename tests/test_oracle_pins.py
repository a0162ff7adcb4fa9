"""The CPU oracle against the paper and mathematics (no GPU)."""
import os
import subprocess
import sys

import numpy as np
import pytest

from oracle import oracle as oracle_mod
from tests import pins


@pytest.fixture(scope="module")
def o():
    return oracle_mod.Oracle()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(o, pin):
    pin(o)


def test_bitwise_independent_of_thread_count(tmp_path):
    """Every per-vector operation runs in a fixed order, so the result must not
    depend on how many OpenMP threads split the rows and columns."""
    outs = []
    for threads in ("1", "4"):
        out = tmp_path / f"y{threads}.npy"
        code = (
            "import sys, numpy as np; sys.path.insert(0, %r);"
            "from oracle import oracle as o;"
            "from paper_2607_25234_amd import workloads as w;"
            "x, g = w.draw(3, 512, 64, 'f32', 7);"
            "np.save(%r, o.whtmix(x, g))" % (os.getcwd(), str(out)))
        env = dict(os.environ, OMP_NUM_THREADS=threads)
        subprocess.run([sys.executable, "-c", code], check=True, env=env,
                       cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
        outs.append(np.load(out))
    assert np.array_equal(outs[0], outs[1])


def test_full_size_unit_gain_identity(o):
    """At a full workload size (one 65536 x 128 slice) G = 1 still returns X
    to double rounding: the forward-error growth of the butterfly is tiny."""
    rng = np.random.default_rng(9)
    x = rng.standard_normal((65536, 128)).astype(np.float32)
    y = o.whtmix(x, np.ones((65536, 128)))
    assert np.max(np.abs(y - x)) < 1e-12
