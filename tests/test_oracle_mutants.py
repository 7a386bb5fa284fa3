"""Plant plausible mistakes in copies of the oracle's C source (on the CPU) and
check that the pins catch every one of them: a dropped term, a wrong sign, a
wrong index, a transposed operand, a wrong offset."""
import os
import shutil
import subprocess

import pytest

import oracle
from tests import pins

SRC = open(oracle.SOURCE).read()

# (name, exact text in optimus_oracle.c, replacement)
MUTANTS = [
    ("transposed_weight", "s += x[m * ldx + k] * w[n * ldw + k];", "s += x[m * ldx + k] * w[k * ldw + n];"),
    ("dropped_last_k_term", "for (int64_t k = 0; k < K; ++k) s += x[m * ldx + k]",
     "for (int64_t k = 0; k + 1 < K; ++k) s += x[m * ldx + k]"),
    ("dropped_bias", "      if (bias) s += bias[n];\n      y[m * ldy + n]", "      y[m * ldy + n]"),
    ("bias_wrong_index", "if (bias) s += bias[n];\n      y[m * ldy", "if (bias) s += bias[m % N];\n      y[m * ldy"),
    ("rows_wrong_row", "const double* xr = x + rows[i] * ldx;", "const double* xr = x + i * ldx;"),
    ("unbiased_variance", "var /= (double)cols;\n  double inv", "var /= (double)(cols > 1 ? cols - 1 : 1);\n  double inv"),
    ("bwd_ln_unbiased_variance", "var /= (double)cols;\n    const double rstd",
     "var /= (double)(cols > 1 ? cols - 1 : 1);\n    const double rstd"),
    ("eps_outside_sqrt", "double inv = 1.0 / sqrt(var + eps);", "double inv = 1.0 / (sqrt(var) + eps);"),
    ("mean_not_subtracted", "double v = (x[c] - mu) * inv;", "double v = x[c] * inv;"),
    ("beta_dropped", "if (beta) v += beta[c];", ""),
    ("gamma_beta_swapped", "if (gamma) v *= gamma[c];\n    if (beta) v += beta[c];",
     "if (beta) v *= beta[c];\n    if (gamma) v += gamma[c];"),
    ("sigmoid_wrong_sign", "return 1.0 / (1.0 + exp(-x));", "return 1.0 / (1.0 + exp(x));"),
    ("silu_without_x", "return x * orc_sigmoid(x);", "return orc_sigmoid(x);"),
    ("relu_leaky", "return x > 0.0 ? x : 0.0;", "return x > 0.0 ? x : 0.01 * x;"),
    ("tanh_half_arg", "return tanh(x);", "return tanh(0.5 * x);"),
    ("split_offset_dropped", "piece[r * w + c] = in[r * ldin + off + c];", "piece[r * w + c] = in[r * ldin + c];"),
    ("cat_offset_dropped", "out[r * ldout + off + c] = res[r * w + c];", "out[r * ldout + c] = res[r * w + c];"),
    ("piece_params_shifted", "gamma ? gamma[j] : NULL,\n                       beta ? beta[j] : NULL",
     "gamma ? gamma[0] : NULL,\n                       beta ? beta[0] : NULL"),
    ("fp8_bias_off", "ldexp(1.0 + m / 8.0, e - 7)", "ldexp(1.0 + m / 8.0, e - 8)"),
    ("fp8_truncate", "long q = (long)nearbyint(a / ldexp(1.0, e - 3));", "long q = (long)floor(a / ldexp(1.0, e - 3));"),
    ("fp8_subnormal_truncate", "code = (int)nearbyint(a / ldexp(1.0, -9));", "code = (int)floor(a / ldexp(1.0, -9));"),
    ("fp8_sign_dropped", "const int s = signbit(v) ? 0x80 : 0;", "const int s = 0;"),
    ("fp8_overflow_threshold", "if (a > 464.0)", "if (a >= 464.0)"),
    ("fp8_nan_unsigned", "if (isnan(v)) return s | 0x7F;", "if (isnan(v)) return 0x7F;"),
    ("bwd_dw_uses_w", "for (int64_t m = 0; m < M; ++m) s += dy[m * lddy + n] * x[m * ldx + k];",
     "for (int64_t m = 0; m < M; ++m) s += dy[m * lddy + n] * w[n * ldw + k];"),
    ("bwd_dx_transposed_w", "for (int64_t n = 0; n < N; ++n) s += dy[m * lddy + n] * w[n * ldw + k];",
     "for (int64_t n = 0; n < N; ++n) s += dy[m * lddy + n] * w[k * ldw + n];"),
    ("bwd_db_first_row", "for (int64_t m = 0; m < M; ++m) s += dy[m * lddy + n];\n      db[n] = s;",
     "s = dy[n];\n      db[n] = s;"),
    ("bwd_relu_at_zero", "case ORC_ACT_RELU: return x > 0.0 ? 1.0 : 0.0;", "case ORC_ACT_RELU: return x >= 0.0 ? 1.0 : 0.0;"),
    ("bwd_sigmoid_grad_s", "return s * (1.0 - s);\n    }\n    case ORC_ACT_TANH:", "return s;\n    }\n    case ORC_ACT_TANH:"),
    ("bwd_tanh_grad_linear", "return 1.0 - t * t;", "return 1.0 - t;"),
    ("bwd_silu_no_x_term", "return s + x * s * (1.0 - s);", "return s;"),
    ("bwd_ln_no_mean_g", "dx[r * lddx + c] = (g - mg - xhat * mgx) * rstd;", "dx[r * lddx + c] = (g - xhat * mgx) * rstd;"),
    ("bwd_ln_no_xhat_term", "dx[r * lddx + c] = (g - mg - xhat * mgx) * rstd;", "dx[r * lddx + c] = (g - mg) * rstd;"),
    ("bwd_ln_gamma_ignored", "const double g = gr[c] * (gamma ? gamma[c] : 1.0);\n        dx[", "const double g = gr[c];\n        dx["),
    ("bwd_ln_dgamma_no_xhat", "if (dgamma) dgamma[c] += gr[c] * xhat;", "if (dgamma) dgamma[c] += gr[c];"),
    ("fp8_nan_sign_of_product", "isnan(v) ? (uint8_t)(signbit(xv) ? 0xFF : 0x7F)", "isnan(v) ? (uint8_t)(signbit(v) ? 0xFF : 0x7F)"),
    ("fp8_scale_inverted", "inv = 448.0f / amax;", "inv = amax / 448.0f;"),
    ("fp8_no_carry", "if (q == 16) { q = 8; ef = e + 1; }", ""),
    ("fp8_dequant_no_scale", "y[r * ldy + c] = (double)(v * scale);", "y[r * ldy + c] = (double)v;"),
]


@pytest.mark.parametrize("name,find,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, find, repl):
    assert SRC.count(find) == 1, f"mutation site for {name} not found exactly once"
    src = tmp_path / "mutant.c"
    src.write_text(SRC.replace(find, repl))
    lib = str(tmp_path / "libmutant.so")
    oracle.compile_library(str(src), lib)
    orc = oracle.Oracle(lib)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(orc)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {name}"


# Plausible mistakes in the fused Linear + LayerNorm composition.
COMPOSITION_MUTANTS = {
    "act_before_layernorm": lambda o, x, w, b, g, be, eps, act: o.layernorm(o.linear(x, w, b, act), g, be, eps),
    "bias_dropped": lambda o, x, w, b, g, be, eps, act: o.layernorm(o.linear(x, w, None), g, be, eps, act),
    "gamma_beta_swapped": lambda o, x, w, b, g, be, eps, act: o.layernorm(o.linear(x, w, b), be, g, eps, act),
    "no_normalisation": lambda o, x, w, b, g, be, eps, act: o.pointwise(o.linear(x, w, b) * (1 if g is None else g)
                                                                         + (0 if be is None else be), act),
}


@pytest.mark.parametrize("name", list(COMPOSITION_MUTANTS))
def test_pins_catch_composition_mutant(name):
    orc = oracle.Oracle()
    bad = COMPOSITION_MUTANTS[name]
    orc.linear_layernorm = lambda x, w, b, g=None, be=None, eps=1e-5, act="none": bad(orc, x, w, b, g, be, eps, act)
    caught = []
    for pin in (pins.linear_layernorm_reductions, pins.linear_layernorm_invariants):
        try:
            pin(orc)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {name}"
