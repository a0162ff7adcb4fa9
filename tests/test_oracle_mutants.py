"""Plant plausible mistakes in copies of the oracle and check the pins catch them.

Each mutant is a one-place textual edit of ``oracle/whtmix_oracle.c``,
compiled with gcc into a temporary library (CPU only; the real oracle is never
modified).  A pin set that let any of these through would not be strong
enough to trust the oracle.
"""
import os

import pytest

from oracle import oracle as oracle_mod
from tests import pins

MUTANTS = {
    # butterfly: wrong sign on the difference output
    "butterfly_sign": ("v[(j + h) * s] = a - b;", "v[(j + h) * s] = b - a;"),
    # butterfly: last stage dropped
    "butterfly_last_stage": ("for (long h = 1; h < n; h *= 2)",
                             "for (long h = 1; h < n / 2; h *= 2)"),
    # butterfly: one pair per block skipped
    "butterfly_pair_skipped": ("for (long j = i; j < i + h; ++j)",
                               "for (long j = i + (h > 1); j < i + h; ++j)"),
    # normalisation 1/n instead of 1/sqrt(n)
    "normalisation": ("double f = 1.0 / sqrt((double)n);",
                      "double f = 1.0 / (double)n;"),
    # token transform left unnormalised
    "token_unnormalised": ("wht_orthonormal(z + c, N, C);",
                           "fwht_strided(z + c, N, C);"),
    # token transform applied along the wrong stride (transposed operand)
    "token_stride": ("wht_orthonormal(z + c, N, C);",
                     "wht_orthonormal(z + c * N, N, 1);"),
    # gain read transposed, G[c][n] instead of G[n][c]
    "gain_transposed": ("z[i] *= g[i];", "z[i] *= g[(i % C) * P + i / C];"),
    # forward token transform dropped
    "forward_token_dropped": (
        "        channel_transform(z, P, C);\n        token_transform(z, P, C);\n"
        "        /* per-frequency gain */",
        "        channel_transform(z, P, C);\n        /* per-frequency gain */"),
    # batch slice offset wrong
    "batch_offset": ("load_padded(z, x + b * N * C, N, P, C);\n        /* forward",
                     "load_padded(z, x + b * C, N, P, C);\n        /* forward"),
    # token axis extended periodically instead of zero-padded
    "padding_not_zero": (
        "memset(z + N * C, 0, (size_t)((P - N) * C) * sizeof(double));",
        "for (long i = N * C; i < P * C; ++i) z[i] = xb[i % (N * C)];"),
    # the wrong N rows kept after the padded transform
    "crop_offset": ("channel_transform(z, P, C);\n        memcpy(y + b * N * C, z, ",
                    "channel_transform(z, P, C);\n        memcpy(y + b * N * C, z + (P - N) * C, "),
    # gradient: dG accumulated from the wrong operand
    "grad_operand": ("dg[i] += tx[i] * td[i];", "dg[i] += tx[i] * tx[i];"),
    # gradient: dY transformed over channels only
    "grad_dy_token_dropped": ("        channel_transform(td, P, C);\n        token_transform(td, P, C);",
                              "        channel_transform(td, P, C);"),
    # separable gradient: chain rule through exp forgotten
    "grad_separable_chain": ("            s += dG[n * C + c] * G[n * C + c];\n        dg_t[n] = s;",
                             "            s += dG[n * C + c];\n        dg_t[n] = s;"),
    # projection with the weight transposed
    "projection_transposed": ("zn[j] += xi * w[i * C + j];",
                              "zn[j] += xi * w[j * C + i];"),
    # W_out applied to the mixer's input instead of its output
    "projection_order": ("project(m, w_out, y + b * N * C, N, C);",
                         "project(z, w_out, y + b * N * C, N, C);"),
    # backward through a projection with the weight not transposed
    "grad_projection_not_transposed": ("s += x[n * C + j] * w[i * C + j];",
                                       "s += x[n * C + j] * w[j * C + i];"),
    # dW_out with its operands swapped (its transpose)
    "grad_weight_operands": ("accumulate_at_b(zp + b * S, dy + b * S, dw_out, N, C);",
                             "accumulate_at_b(dy + b * S, zp + b * S, dw_out, N, C);"),
    # separable form: log gains used without exponentiation
    "separable_no_exp": ("z[n * C + c] *= exp(g_c[c]);", "z[n * C + c] *= g_c[c];"),
    # separable form: token gain indexed by channel
    "separable_gain_index": ("z[n * C + c] *= exp(g_t[n]);",
                             "z[n * C + c] *= exp(g_t[c % N]);"),
}


@pytest.fixture(scope="module")
def source():
    with open(oracle_mod.SRC) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, source, tmp_path):
    old, new = MUTANTS[name]
    assert source.count(old) == 1, f"mutation site for {name} not unique"
    src = tmp_path / f"{name}.c"
    src.write_text(source.replace(old, new))
    lib = oracle_mod.build(str(src), str(tmp_path / f"{name}.so"))
    mutant = oracle_mod.Oracle(lib)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(mutant)
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutant {name}"


def test_unmutated_copy_passes(source, tmp_path):
    """The mutation harness itself: an unmodified copy passes every pin."""
    src = tmp_path / "same.c"
    src.write_text(source)
    mutant = oracle_mod.Oracle(oracle_mod.build(str(src), str(tmp_path / "same.so")))
    for pin in pins.ALL_PINS:
        pin(mutant)
    assert os.path.exists(tmp_path / "same.so")
