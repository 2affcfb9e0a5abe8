"""Planted mistakes in the oracle (CPU only): each mutant is a copy of the
oracle source with one plausible error — a wrong mask, sign, index, constant,
an unfused multiply-add, a dropped term — compiled to a temporary library.
The scalar and operator pins must fail on every one of them, which shows the
pins are strong enough to catch that class of mistake in the real oracle.
"""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "quake_oracle.c")

MUTANTS = {
    "mantissa_mask": ("#define MASK_MANT 0x007FFFFFu", "#define MASK_MANT 0x003FFFFFu"),
    "exponent_rejoin": ("+ f2u(ym) - EXP_B;", "+ f2u(ym) - 0x3F000000u;"),
    "unfused_affine": ("float l = fmaf(x, c0, c1);", "float l = x * c0 + c1;"),
    "coefficient_a0": ("return (float)(1.0 / 3.0);", "return (float)(1.0 / 3.01);"),
    "coefficient_a2": ("ym = fmaf(am, am, 2.0f) * third();", "ym = fmaf(am, am, 1.98f) * third();"),
    "no_schraudolph_bias": ("(mode == QO_Q1) ? 0.0436 : 0.0", "(mode == QO_Q1) ? 0.0 : 0.0"),
    "softmax_c1_sign": ("float c1 = fmaf(-c0, m, k127());", "float c1 = fmaf(c0, m, k127());"),
    "softmax_c1_two_roundings": ("fmaf(-c0, m, k127())", "(k127() - c0 * m)"),
    "softmax_c1_two_roundings_rows": ("float c1 = fmaf(-c0, m, k127());          /* 127*2^23 - c0*m */",
                                      "float c1 = k127() - c0 * m;"),
    "softmax_c1_two_roundings_causal": ("(mode == QO_EXACT) ? fmaf(-c0, m, 0.0f) : fmaf(-c0, m, k127());",
                                        "(mode == QO_EXACT) ? fmaf(-c0, m, 0.0f) : k127() - c0 * m;"),
    "softmax_c1_two_roundings_numerators": ("      float c1 = fmaf(-c0, m, k127());\n      for (int64_t j = 0; j < cols; ++j) {\n        pr[j]",
                                            "      float c1 = k127() - c0 * m;\n      for (int64_t j = 0; j < cols; ++j) {\n        pr[j]"),
    "softmax_drop_last_term": ("tmp[j] = (double)quake_one(load_el(x, bx + j, dt), c0, c1, mode);\n        sum += tmp[j];",
                               "tmp[j] = (double)quake_one(load_el(x, bx + j, dt), c0, c1, mode);\n        if (j + 1 < cols) sum += tmp[j];"),
    "softmax_min_not_max": ("if (v > m) m = v;", "if (v > m || m == -INFINITY) m = (m == -INFINITY) ? v : fminf(m, v);"),
    "gelu_fma_constant": ("static float a_gelu(void) { return (float)(1.0 / 0.044715); }",
                          "static float a_gelu(void) { return (float)(0.044715); }"),
    "gelu_scale": ("sqrt(2.0 / 3.14159265358979323846264338327950288)", "sqrt(3.14159265358979323846264338327950288 / 2.0)"),
    "sigmoid_sign": ("float c0 = c0_of(-1.0), c1 = c1_of(0.0, mode);\n  float c0e = (float)(-1.0 / LN2);",
                     "float c0 = c0_of(1.0), c1 = c1_of(0.0, mode);\n  float c0e = (float)(-1.0 / LN2);"),
    "round_truncates": ("double r = nearbyint(a / quantum) * quantum;", "double r = floor(a / quantum) * quantum;"),
    "f16_decode_bias": ("else v = ldexpf((float)(1024 + m), e - 25);", "else v = ldexpf((float)(1024 + m), e - 24);"),
    "clamp_missing": ("if (l > l_hi()) l = l_hi();", ""),
    "unfused_no_temperature": ("float s = d * t;                        /* temperature     */",
                               "float s = d;"),
    "unfused_gelu_sign": ("double e = (double)std_exp(-s, mode);", "double e = (double)std_exp(s, mode);"),
    "causal_off_by_one": ("int64_t L = r % period + shift + 1;", "int64_t L = r % period + shift;"),
    "q2m_no_alternation": ("m[i][3] = (i % 2) ? 1.0 : -1.0;   /* -(-1)^i E */", "m[i][3] = -1.0;"),
    "q2m_horner_swap": ("ym = fmaf(fmaf(q2m_f[0], am, q2m_f[1]), am, q2m_f[2]);",
                        "ym = fmaf(fmaf(q2m_f[0], am, q2m_f[2]), am, q2m_f[1]);"),
    "q2m_integer_rule_missing": ("  if (order == QO_Q2M && ((uint32_t)z & MASK_MANT) == 0) yi = (uint32_t)z;\n", ""),
    "exp16_f16_bias": ("const int bias = (dt == QO_F16) ? 15 : 127;", "const int bias = (dt == QO_F16) ? 16 : 127;"),
    "exp16_mask": ("const uint32_t mant = (1u << lm) - 1u;", "const uint32_t mant = (1u << (lm - 1)) - 1u;"),
    "exp16_third_unrounded": ("const double third16 = (double)dec_f16(enc_f16(1.0 / 3.0));",
                              "const double third16 = 1.0 / 3.0;"),
    "unfused_no_max": ("float d = load_el(x, bx + j, dt) - m;   /* max subtraction */",
                       "float d = load_el(x, bx + j, dt);"),
}


def _build(name, tmp_path):
    src = open(SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, name          # every copy of the pattern is mutated
    mpath = tmp_path / ("mut_%s.c" % name)
    mpath.write_text(src.replace(old, new))
    so = tmp_path / ("mut_%s.so" % name)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
                           "-shared", "-o", str(so), str(mpath), "-lm"])
    return so


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    so = _build(name, tmp_path)
    env = dict(os.environ, QUAKE_ORACLE_LIB=str(so))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle_scalar.py"),
                        os.path.join(HERE, "test_oracle_ops.py"),
                        os.path.join(HERE, "test_oracle_q2m.py"),
                        os.path.join(HERE, "test_oracle_native16.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, "mutant %s survived the pins:\n%s" % (name, r.stdout[-2000:])
    assert "failed" in r.stdout or "error" in r.stdout.lower()
