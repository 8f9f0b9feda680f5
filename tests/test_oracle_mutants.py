"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a temporary copy of the oracle's C source (a
dropped term, a wrong sign, a swapped or transposed operand, a wrong tie rule,
...), builds it, and checks that at least one pin fails on it.  CPU only; the
real oracle file is never modified.
"""

import os
import shutil

import pytest

import pins
from oracle import oracle as orc_mod

SRC = os.path.join(os.path.dirname(orc_mod.__file__), "moe_oracle.c")

MUTANTS = {
    "silu_sign": ("return z / (1.0 + exp(-z));", "return z / (1.0 + exp(z));"),
    "silu_dropped": ("h[rows[q] * ffn + n] = silu(u) * v;", "h[rows[q] * ffn + n] = u * v;"),
    "w1_w3_swapped": ("h[rows[q] * ffn + n] = silu(u) * v;", "h[rows[q] * ffn + n] = silu(v) * u;"),
    "tie_to_higher_index": ("(la == lb && a < b)", "(la == lb && a > b)"),
    "softmax_over_all_experts": (
        "for (int j = 0; j < k; ++j) denom += exp(l[s[j]] - top);",
        "for (int m = 0; m < E; ++m) denom += exp(l[m] - top);"),
    "gate_unshifted_numerator": ("gates[t * k + j] = exp(l[s[j]] - top) / denom;",
                                 "gates[t * k + j] = exp(l[s[j]]) / denom;"),
    "bias_dropped": ("if (bias) s += (double)bias[e];", ";"),
    "router_transposed": ("widen(wr[e * d + i])", "widen(wr[i * E + e])"),
    "w2_row_stride": ("widen_row(w2, (int64_t)e * d + i, ffn, r2)", "widen_row(w2, (int64_t)e * ffn + i, ffn, r2)"),
    "w1_row_stride": ("widen_row(w1, (int64_t)e * ffn + n, d, r1)", "widen_row(w1, (int64_t)e * d + n, d, r1)"),
    "weight_row_reversed": ("out[i] = widen(w.bf16[r * cols + i]);", "out[i] = widen(w.bf16[r * cols + (cols - 1 - i)]);"),
    "fp8_bias_8": ("ldexp(1.0 + (double)m / 8.0, e - 7)", "ldexp(1.0 + (double)m / 8.0, e - 8)"),
    "fp8_subnormal_as_normal": ("v = ldexp((double)m / 8.0, -6);", "v = ldexp(1.0 + (double)m / 8.0, -7);"),
    "fp8_scale_dropped": ("out[i] = fp8_e4m3(w.q[r * cols + i]) * s;", "out[i] = fp8_e4m3(w.q[r * cols + i]);"),
    "fp8_sign_dropped": ("return sign ? -v : v;", "return v;"),
    "token_index": ("xd + (rows[q] / k) * d", "xd + (rows[q] % k) * d"),
    "combine_first_gate_only": ("s += gates[t * k + j] * y", "s += gates[t * k] * y"),
    "combine_unweighted": ("s += gates[t * k + j] * y", "s += y"),
    "offsets_not_cumulative": ("offsets[e + 1] = offsets[e] + counts[e];",
                               "offsets[e + 1] = counts[e];"),
    "perm_descending": ("for (int64_t a = 0; a < A; ++a)\n            if (ids[a] == e) perm[r++]",
                        "for (int64_t a = A - 1; a >= 0; --a)\n            if (ids[a] == e) perm[r++]"),
    "rmsnorm_eps_dropped": ("sqrt(ss / (double)d + eps)", "sqrt(ss / (double)d)"),
    "rmsnorm_mean_as_sum": ("sqrt(ss / (double)d + eps)", "sqrt(ss + eps)"),
    "rmsnorm_gamma_dropped": ("* inv * widen(gamma[i])", "* inv"),
    "topk_second_best_repeats": ("taken |= (s[m] == e);", "taken |= 0;"),
    # the decoder layer around the MoE block
    "rope_interleaved_pairs": ("const double a = v[i], b = v[i + half];\n                v[i] = a * c - b * s;\n"
                               "                v[i + half] = b * c + a * s;",
                               "const double a = v[2 * i], b = v[2 * i + 1];\n                v[2 * i] = a * c - b * s;\n"
                               "                v[2 * i + 1] = b * c + a * s;"),
    "rope_sign": ("v[i] = a * c - b * s;", "v[i] = a * c + b * s;"),
    "rope_frequency": ("pow(base, -2.0 * i / hd)", "pow(base, -1.0 * i / hd)"),
    "attention_scale_dropped": ("sc[s] = scale * dot;", "sc[s] = dot;"),
    "attention_gqa_modulo": ("const int g = h / group;", "const int g = h % Hkv;"),
    "attention_context_short": ("const int L = ctx[t];", "const int L = ctx[t] > 1 ? ctx[t] - 1 : 1;"),
    "attention_slot_off_by_one": ("const uint16_t* vr = vc + ((pg * Hkv + g) * page + s % page) * hd;",
                                  "const uint16_t* vr = vc + ((pg * Hkv + g) * page + (s + 1) % page) * hd;"),
    "round_bf16_truncates": ("nearbyint(ldexp(f, bits))", "floor(ldexp(f, bits))"),
}


@pytest.fixture(scope="module")
def workdir(tmp_path_factory):
    return tmp_path_factory.mktemp("mutants")


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, workdir):
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) >= 1, f"mutation site for {name} not found"
    src = os.path.join(workdir, f"{name}.c")
    with open(src, "w") as f:
        f.write(text.replace(old, new, 1))
    lib = os.path.join(workdir, f"lib_{name}.so")
    orc_mod.build(src, lib, extra=("-Wno-unused-variable", "-Wno-unused-but-set-variable",
                                   "-Wno-unused-function", "-Wno-error"))
    mutant = orc_mod.Oracle(lib)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(mutant)
        except (AssertionError, orc_mod.OracleError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches mutant {name}"


def test_real_oracle_source_untouched():
    assert shutil.which("gcc")
    assert "return z / (1.0 + exp(-z));" in open(SRC).read()
