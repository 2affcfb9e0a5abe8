"""Pins of the oracle's QuAKE built in a 16-bit format's own layout (qo_exp16):
Eq. 3 with the l_m and B of binary16 (10, 15) and bfloat16 (7, 127), and
Algorithm 1 with the 16-bit masks and the refinement in that format's
arithmetic. Checked against closed forms whose bit patterns are written out
here independently, against numpy's float16 / torch's bfloat16 rounding for
the refinement, and exhaustively over all 65536 inputs for the error bound and
monotonicity."""
import math

import numpy as np
import pytest
import torch

FMT = {"f16": dict(lm=10, B=15, emin=-14, emax=15), "bf16": dict(lm=7, B=127, emin=-126, emax=127)}
LN2 = math.log(2.0)
A_BASE2 = float(np.float32(LN2))          # a = fl32(ln 2) makes c0 = 2^l_m exactly


def _bits(v: np.ndarray, dt: str) -> np.ndarray:
    if dt == "f16":
        return np.asarray(v, np.float16).view(np.uint16)
    return torch.from_numpy(np.asarray(v, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _value(b: np.ndarray, dt: str) -> np.ndarray:
    if dt == "f16":
        return b.view(np.float16).astype(np.float64)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _ym_ref(am: np.ndarray, dt: str) -> np.ndarray:
    """(a_m^2 + 2)/3 in the format's arithmetic, from numpy / torch rounding."""
    if dt == "f16":
        a = am.astype(np.float16)
        t = (a.astype(np.float32) * a.astype(np.float32) + np.float32(2)).astype(np.float16)  # exact in f32, one rounding
        third = np.float16(1.0 / 3.0)
        return (t.astype(np.float32) * np.float32(third)).astype(np.float16).astype(np.float64)
    a = am.astype(np.float32)
    p = (a * a + np.float32(2)) * np.float32(1.0 / 3.0)
    return torch.from_numpy(p.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_quake2_exact_at_integer_powers(oracle, dt):
    f = FMT[dt]
    k = np.arange(f["emin"], f["emax"] + 1)
    y = oracle.exp16(_bits(k, dt), dt, oracle.Q2, a=A_BASE2)
    assert np.array_equal(_value(y, dt), np.ldexp(1.0, k))


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_first_order_closed_form(oracle, dt):
    # Eq. 3 in the 16-bit layout: the pattern of 2^k (1 + j / 2^fb) is
    # ((k + B) << l_m) | (j << (l_m - fb)); b cancels the Schraudolph bias
    f = FMT[dt]
    fb = 6 if dt == "f16" else 3                       # fraction bits the input format holds at |x| < 16
    b = float(np.float32(0.0436 * LN2))
    k = np.repeat(np.arange(max(f["emin"], -15), min(f["emax"], 15) + 1), 1 << fb)
    j = np.tile(np.arange(1 << fb), k.size // (1 << fb))
    x = k + j / 2.0 ** fb
    xb = _bits(x, dt)
    assert np.array_equal(_value(xb, dt), x)          # inputs exact in the format
    y = oracle.exp16(xb, dt, oracle.Q1, a=A_BASE2, b=b)
    want = (((k + f["B"]) << f["lm"]) | (j << (f["lm"] - fb))).astype(np.uint16)
    assert np.array_equal(y, want)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_second_order_closed_form(oracle, dt):
    f = FMT[dt]
    fb = 6 if dt == "f16" else 3
    k = np.repeat(np.arange(max(f["emin"], -15), min(f["emax"], 15) + 1), 1 << fb)
    j = np.tile(np.arange(1 << fb), k.size // (1 << fb))
    x = k + j / 2.0 ** fb
    y = oracle.exp16(_bits(x, dt), dt, oracle.Q2, a=A_BASE2)
    ym = _ym_ref(1.0 + j / 2.0 ** fb, dt)
    assert np.all((ym >= 1) & (ym < 2))
    assert np.array_equal(_value(y, dt), np.ldexp(ym, k))


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_refined_mantissa_continuous_and_below_two(oracle, dt):
    # every mantissa: x = 1 + m / 2^l_m exact in the format and in l
    f = FMT[dt]
    m = np.arange(1 << f["lm"])
    x = 1.0 + m / 2.0 ** f["lm"]
    y = _value(oracle.exp16(_bits(x, dt), dt, oracle.Q2, a=A_BASE2), dt) / 2.0
    assert y[0] == 1.0 and np.all(y < 2.0) and np.all(np.diff(y) >= 0)
    assert np.array_equal(y, _ym_ref(x, dt))


def _all_inputs(dt):
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    v = _value(b, dt)
    keep = np.isfinite(v)
    b, v = b[keep], v[keep]
    order = np.argsort(v, kind="stable")
    return b[order], v[order]


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("mode", [1, 2])
def test_every_input_error_bound_and_monotone(oracle, dt, mode):
    f = FMT[dt]
    b, v = _all_inputs(dt)
    y = _value(oracle.exp16(b, dt, mode), dt)
    assert np.all(y[1:] >= y[:-1])                     # monotone over all inputs
    with np.errstate(over="ignore"):
        ref = np.exp(v)
    # normal results only (below 2^emin the exponent field is 0 and Eq. 2
    # no longer describes the pattern)
    ok = (ref >= 2.0 ** (f["emin"] + 1)) & (y < np.inf) & (ref < 2.0 ** (f["emax"] + 1))
    rel = y[ok] / ref[ok] - 1
    # Error sources beyond the approximation itself: truncating l to an integer
    # drops up to 2^-l_m of the base-2 exponent (q); QuAKE2 rounds t = a_m^2 + 2,
    # then t * fl(1/3), to the format (each at most half an ulp, r each) and
    # binary16's 1/3 is 2^-12 relative low (binary32's for bfloat16: negligible).
    q = LN2 * 2.0 ** -f["lm"]
    r = 2.0 ** -(f["lm"] + 1)
    third = 1 - 3 * float(np.float16(1 / 3)) if dt == "f16" else 1e-7
    if mode == 2:
        assert rel.min() >= -(0.0018748 + q + 2 * r + third) and rel.max() <= 0.0034185 + 2 * r + 1e-6
        assert rel.max() > 0.0034 and rel.min() < -0.0018       # the approximation error is there
    else:
        assert rel.min() >= -(0.0297765 + q + 1e-6) and rel.max() <= 0.0298805 + 1e-6
    assert np.count_nonzero(ok) > (10000 if dt == "f16" else 2000)
    # special values: e^0 (QuAKE2) = 1, overflow -> +inf, underflow -> 0
    s = oracle.exp16(_bits(np.array([0.0, 100.0, -200.0]), dt), dt, mode)
    sv = _value(s, dt)
    assert sv[1] == np.inf and sv[2] == 0.0
    if mode == 2:
        assert sv[0] == 1.0


def test_rejects_binary32_and_exact(oracle):
    with pytest.raises(ValueError):
        oracle.exp16(np.zeros(4, np.float32), "f32", 2)
    with pytest.raises(ValueError):
        oracle.exp16(np.zeros(4, np.uint16), "f16", 0)
