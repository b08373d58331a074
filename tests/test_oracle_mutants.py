"""Plant plausible mistakes in copies of the oracle; the pins must catch each.

Every mutant is a textual edit of oracle/cats_oracle.c compiled on the CPU
into a temporary library.  A mutant passes this test when at least one pin
of oracle_pins.py fails on it, i.e. the pins are strong enough to notice
that mistake.  Nothing here touches a GPU.
"""
import os

import pytest

import oracle
from oracle_pins import ALL_PINS

MUTANTS = {
    # Eq. 2 with the wrong sign in the exponent
    "silu_sign": ("R_EXP(-z)", "R_EXP(z)"),
    # Eq. 4 with a strict comparison (ties dropped)
    "strict_compare": ("!(R_FABS(v) < t)", "(R_FABS(v) > t)"),
    # Eq. 4 without the absolute value (negative activations dropped)
    "no_abs": ("!(R_FABS(v) < t)", "!(v < t)"),
    # x1 = v instead of v * (x W_up)
    "drop_up": ("const real h = v * u[j];", "const real h = v;"),
    # the first input channel dropped from both dot products
    "drop_first_term": ("for (int32_t i = 0; i < d; ++i) {\n        const real xi = (real)xb[i];",
                        "for (int32_t i = 1; i < d; ++i) {\n        const real xi = (real)xb[i];"),
    # W_down read transposed
    "transposed_down": ("s[k] += h * (real)wd_row[k];", "s[k] += h * (real)w_down[(size_t)k * m + j];"),
    # W_gate and W_up swapped
    "swap_gate_up": ("g[j] += xi * (real)wg_row[j];\n          u[j] += xi * (real)wu_row[j];",
                     "g[j] += xi * (real)wu_row[j];\n          u[j] += xi * (real)wg_row[j];"),
    # the dense flag ignored
    "dense_ignored": ("if (!(dense || cats_keeps(v, t))) continue;", "if (!cats_keeps(v, t)) continue;"),
    # residual dropped
    "drop_residual": ("if (residual) out = (real)residual[(size_t)b * d + k] + out;", ""),
    # Eq. 3 rank off by one
    "rank_plus_one": ("double r = ceil(k * (double)n - 1e-6);", "double r = ceil(k * (double)n - 1e-6) + 1;"),
    # order statistic read one slot early
    "threshold_index": ("*t = fabs(c[r - 1]);", "*t = fabs(c[r > 1 ? r - 2 : 0]);"),
    # calibration on signed instead of absolute activations
    "calib_no_abs": ("acts[(size_t)n * m + j] = (double)R_FABS(silu(g[j]));",
                     "acts[(size_t)n * m + j] = (double)silu(g[j]);"),
    # RMSNorm over the sum instead of the mean
    "rms_sum": ("ss / (real)d + (real)eps", "ss + (real)eps"),
    # stack: the MLP fed the raw residual stream instead of its RMSNorm
    "stack_no_norm": ("rc = oracle_cats_mlp(xn, B, d, m,", "rc = oracle_cats_mlp((float*)xl, B, d, m,"),
    # stack: the residual connection dropped
    "stack_no_residual": ("dense ? 0.0 : t[l], dense, xl,", "dense ? 0.0 : t[l], dense, NULL,"),
    # stack: layer 0's threshold used for every layer
    "stack_first_t": ("dense ? 0.0 : t[l], dense, xl,", "dense ? 0.0 : t[0], dense, xl,"),
    # input sparsity: strict comparison (ties dropped)
    "gemv_strict": ("if (!cats_keeps(xc, t)) continue;", "if (!(R_FABS(xc) > t)) continue;"),
    # input sparsity: W read transposed
    "gemv_transposed": ("for (int32_t k = 0; k < n; ++k) s[k] += xc * (real)w_row[k];",
                        "for (int32_t k = 0; k < n; ++k) s[k] += xc * (real)w[((size_t)k * d + i) % ((size_t)d * n)];"),
    # top-k: one cutoff computed from row 0 used for every row
    "topk_row0": ("if (oracle_calib_acts(x + (size_t)b * d, 1, d, m, w_gate, a) != 0) {",
                  "if (oracle_calib_acts(x, 1, d, m, w_gate, a) != 0) {"),
    # v reported before the activation
    "v_before_silu": ("if (v_all) v_all[(size_t)b * m + j] = (double)v;",
                      "if (v_all) v_all[(size_t)b * m + j] = (double)g[j];"),
}


@pytest.mark.parametrize("precision", ["f32", "f64"])
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name, precision):
    old, new = MUTANTS[name]
    with open(oracle.SOURCE) as f:
        src = f.read()
    assert src.count(old) == 1, f"mutation target for {name} not found exactly once"
    mutated = tmp_path / "cats_oracle.c"
    mutated.write_text(src.replace(old, new))
    lib = oracle.compile_oracle(str(tmp_path / f"lib_{name}.so"), source=str(mutated), precision=precision)
    O = oracle.Oracle(lib)
    caught = []
    for pin in ALL_PINS:
        try:
            pin(O)
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutant {name} ({precision})"


def test_unmutated_copy_passes(tmp_path):
    """Compiling the oracle from a copy changes nothing."""
    with open(oracle.SOURCE) as f:
        src = f.read()
    p = tmp_path / "cats_oracle.c"
    p.write_text(src)
    O = oracle.Oracle(oracle.compile_oracle(str(tmp_path / "lib.so"), source=str(p)))
    for pin in ALL_PINS:
        pin(O)
