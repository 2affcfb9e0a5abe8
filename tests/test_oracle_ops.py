"""Pins of the oracle's operators: Softmax (Algorithm 2), GELU (Eq. 4 / Eq. 7),
Logistic and SiLU, and e^(a x + b) with the affine map folded (Eq. 5).

Reference values come from numpy / scipy in double precision, and the bounds
from the exhaustive error range of the scalar approximation: QuAKE2's relative
error lies in [-0.18748 %, +0.34185 %], first order's in [-2.9777 %, +2.9881 %],
QuAKE2 with the minimax coefficients of Eq. 6 (mode 3) in [-0.17248 %, +0.17248 %].
"""
import math
from fractions import Fraction

import numpy as np
import pytest
from scipy.special import expit, softmax as sp_softmax

from fp32ref import add32, bits32, f32, fma32, from_bits32, mul32, rne32

LN2 = math.log(2.0)
# max |rel err| of e, + l spacing; mode 3 is QuAKE2 with the minimax coefficients (+-0.17248 %)
EPS = {1: 0.0298805 + 2e-5, 2: 0.0034185 + 2e-5, 3: 0.0017248 + 2e-5}
RATIO = {1: (1 + 0.0298805) / (1 - 0.0297765) - 1 + 4e-5,
         2: (1 + 0.0034185) / (1 - 0.0018748) - 1 + 4e-5,
         3: (1 + 0.0017248) / (1 - 0.0017248) - 1 + 4e-5}


def _rows(seed, rows, cols, scale):
    return (np.random.default_rng(seed).standard_normal((rows, cols)) * scale).astype(np.float32)


# ------------------------------ softmax ------------------------------------

@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("cols,t", [(1, 1.0), (7, 1.0), (128, 0.125), (1000, 3.0), (4099, 1.0)])
def test_softmax_rows_sum_to_one(oracle, mode, cols, t):
    x = _rows(cols, 6, cols, 4.0)
    y = oracle.softmax(x, "f32", mode, t=t)
    s = y.astype(np.float64).sum(axis=1)
    assert np.all(np.abs(s - 1) <= cols * 2.0 ** -24 + 1e-12)


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_softmax_single_and_constant_rows(oracle, mode):
    assert oracle.softmax(np.array([[3.5]], np.float32), "f32", mode)[0, 0] == 1.0
    for n in (2, 3, 10, 512, 1000):
        y = oracle.softmax(np.full((1, n), -2.25, np.float32), "f32", mode, t=0.7)
        assert np.all(y == y[0, 0])
        assert abs(float(y[0, 0]) * n - 1) <= 2.0 ** -23


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("t", [1.0, 0.125, 2.5])
def test_softmax_against_exact(oracle, mode, t):
    x = _rows(3, 32, 300, 3.0)
    y = oracle.softmax(x, "f32", mode, t=t).astype(np.float64)
    ref = sp_softmax(t * x.astype(np.float64), axis=1)
    rel = np.abs(y / ref - 1)
    big = ref > 1e-30
    if mode == 0:
        # binary32 rounding of c0, c1 and of s grows with |s| = t |x - m| / ln 2
        arg = t * (x.max(axis=1, keepdims=True) - x).astype(np.float64)
        bound = (4 * 2.0 ** -24 * (1 + arg) + 2e-7)[big]
    else:
        bound = RATIO[mode]
    assert np.all(rel[big] <= bound)
    if mode == 2:
        assert rel[big].max() > 0.002        # the approximation is really used
    if mode == 3:
        assert 0.001 < rel[big].max() <= RATIO[3]


@pytest.mark.parametrize("mode", [1, 2, 3])
def test_softmax_shift_invariance(oracle, mode):
    # Algorithm 2 folds the max into c1, so adding a constant to a row changes
    # only the binary32 rounding of l.
    # The minimax coefficients (mode 3) give up continuity at binade edges
    # (y(1) > 1, y(2-) < 2): a rounding step of l across an edge can move one
    # exponent by the jump 2 y(1) / y(2-) - 1, about 0.35 %.
    x = (np.round(_rows(4, 16, 200, 2.0) * 256) / 256).astype(np.float32)
    y0 = oracle.softmax(x, "f32", mode).astype(np.float64)
    bound = 1e-4
    if mode == 3:
        a = oracle.q2m_coefficients()["a"]
        bound += 2 * a.sum() / (4 * a[0] + 2 * a[1] + a[2]) - 1
    for c in (0.5, -7.0, 40.0):
        y1 = oracle.softmax((x + np.float32(c)).astype(np.float32), "f32", mode).astype(np.float64)
        assert np.max(np.abs(y1 / y0 - 1)) < bound


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_softmax_masking(oracle, mode):
    x = _rows(5, 8, 64, 2.0)
    keep = np.random.default_rng(6).random((8, 64)) < 0.6
    keep[:, 0] = True
    xm = np.where(keep, x, -np.inf).astype(np.float32)
    y = oracle.softmax(xm, "f32", mode)
    assert np.all(y[~keep] == 0.0)
    for r in range(8):
        sub = oracle.softmax(x[r, keep[r]][None, :].copy(), "f32", mode)
        assert np.array_equal(y[r, keep[r]], sub[0])
    z = oracle.softmax(np.full((2, 16), -np.inf, np.float32), "f32", mode)
    assert np.all(z == 0.0)


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
def test_softmax_row_strides(oracle, dt):
    x = _rows(7, 5, 40, 1.5)
    xs = oracle.round_to(x.astype(np.float64), dt)
    padded = np.zeros((5, 48), xs.dtype)
    padded[:, :40] = xs
    a = oracle.softmax(padded, dt, 2, cols=40, ldx=48, ldy=44)
    b = oracle.softmax(xs, dt, 2)
    assert np.array_equal(a[:, :40], b)
    assert np.all(a[:, 40:] == 0)


# Reading R8: Algorithm 2 computes the row constant c1 = 127*2^23 - c0*m in
# binary32. The oracle evaluates it as one fused multiply-add (one rounding).
# Rows are built whose max m makes that value differ from a separate product
# and subtraction (two roundings); the expected first-order results are then
# evaluated exactly with IEEE-754 arithmetic written in the test.

K127 = float(127 * 2 ** 23)


def _split_c1_maxima(c0, n, seed):
    """Binary32 row maxima in [-60, 60] for which fl(K127 - fl(c0 m)) differs
    from the singly rounded fl(K127 - c0 m)."""
    r = np.random.default_rng(seed)
    out = []
    for m in r.uniform(-60, 60, 4000).astype(np.float32):
        m = float(m)
        if fma32(-c0, m, K127) != add32(K127, -mul32(c0, m)):
            out.append(m)
        if len(out) == n:
            break
    assert len(out) == n
    return out


def _r8_rows(c0, seed, cols=24, rows=12):
    """Rows whose first entry is the row max m (from _split_c1_maxima) and whose
    other entries lie up to 12 below it."""
    ms = _split_c1_maxima(c0, rows, seed)
    r = np.random.default_rng(seed + 1)
    x = np.empty((rows, cols), np.float32)
    for i, m in enumerate(ms):
        x[i, 0] = m
        x[i, 1:] = (np.float32(m) - r.uniform(0.0, 12.0, cols - 1).astype(np.float32)).astype(np.float32)
        assert x[i].max() == np.float32(m)
    return x


def _first_order_bits(row, c0):
    """z of every entry: l = fl(x c0 + c1) with c1 = fl(K127 - c0 m), clamped to
    [0, 255 * 2^23] and truncated (Eq. 3, recipe step a5)."""
    m = float(row.max())
    c1 = fma32(-c0, m, K127)
    z = []
    for v in row:
        l = min(max(fma32(float(v), c0, c1), 0.0), float(255 * 2 ** 23))
        z.append(int(l))
    return z


def _softmax_of_bits(z):
    """Exact Fraction quotient z_j-as-float / sum, rounded once to binary32."""
    y = [Fraction(from_bits32(b)) for b in z]
    s = sum(y)
    return [rne32(v / s) for v in y]


@pytest.mark.parametrize("t", [1.0, 0.125])
def test_softmax_row_c1_is_one_fused_multiply_add(oracle, t):
    c0 = f32(2.0 ** 23 * t / LN2)
    x = _r8_rows(c0, seed=81 + int(t * 8))
    # numerators of Algorithm 2 (first order): the bits are z itself
    p, _ = oracle.softmax_numerators(x, 1, t=t)
    for i in range(x.shape[0]):
        assert [bits32(float(v)) for v in p[i]] == _first_order_bits(x[i], c0), i
    # the normalised rows: within one binary32 ulp of the exact quotient
    # (the oracle sums and divides in double, then rounds once)
    y = oracle.softmax(x, "f32", 1, t=t)
    far = 0
    for i in range(x.shape[0]):
        z = _first_order_bits(x[i], c0)
        want = _softmax_of_bits(z)
        got = [float(v) for v in y[i]]
        assert all(abs(bits32(g) - bits32(w)) <= 1 for g, w in zip(got, want)), i
        # the two-rounding c1 would move this row by more than one ulp somewhere
        m = float(x[i].max())
        c1_two = add32(K127, -mul32(c0, m))
        z2 = [int(min(max(fma32(float(v), c0, c1_two), 0.0), float(255 * 2 ** 23))) for v in x[i]]
        alt = _softmax_of_bits(z2)
        far += any(abs(bits32(a) - bits32(w)) > 1 for a, w in zip(alt, want))
    assert far >= x.shape[0] // 2


def test_causal_softmax_row_c1_is_one_fused_multiply_add(oracle):
    # the implicit-mask softmax folds the max of each live prefix the same way;
    # entry 0 holds the row max, so every prefix has it
    c0 = f32(2.0 ** 23 / LN2)
    x = _r8_rows(c0, seed=97, cols=12, rows=12)
    y = oracle.softmax_causal(x, 12, 0, "f32", 1, t=1.0)
    for i in range(12):
        z = _first_order_bits(x[i, :i + 1], c0)
        want = _softmax_of_bits(z)
        got = [float(v) for v in y[i, :i + 1]]
        assert all(abs(bits32(g) - bits32(w)) <= 1 for g, w in zip(got, want)), i
        assert np.all(y[i, i + 1:] == 0)


# ------------------------------ GELU ----------------------------------------

def _gelu_tanh(x):
    """Eq. 4 in double. 0.5 (1 + tanh a) is evaluated as expit(2 a), the same
    function without the cancellation of 1 + tanh a for very negative a."""
    x = x.astype(np.float64)
    a = math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)
    return x * expit(2 * a)


def _gelu_tanh_literal(x):
    x = x.astype(np.float64)
    return 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)))


def test_gelu_exact_mode_is_eq4(oracle):
    # Eq. 7 is an exact rewrite of Eq. 4: with exact exp the two agree up to
    # the binary32 rounding of u, w and the scaled argument.
    x = np.concatenate([np.linspace(-10, 10, 200001), [0.0, -0.0, 1e-30, -1e-30]]).astype(np.float32)
    y = oracle.gelu(x, "f32", 0).astype(np.float64)
    ref = _gelu_tanh(x)
    err = np.abs(y - ref)
    assert np.all(err <= 2e-5 * np.abs(ref) + 1e-44)
    mid = np.abs(x) <= 4
    lit = _gelu_tanh_literal(x[mid])
    assert np.all(np.abs(y[mid] - lit) <= 2e-5 * np.abs(lit) + 1e-15)


@pytest.mark.parametrize("mode", [1, 2, 3])
def test_gelu_quake_bound(oracle, mode):
    x = np.linspace(-12, 12, 400001).astype(np.float32)
    y = oracle.gelu(x, "f32", mode).astype(np.float64)
    ref = _gelu_tanh(x)
    eps = EPS[mode]
    bound = np.abs(x.astype(np.float64)) * (eps / (4 * (1 - eps)) + 2.0 ** -23) + 1e-37
    assert np.all(np.abs(y - ref) <= bound)
    assert np.max(np.abs(y - ref) / np.maximum(np.abs(x), 1e-30)) > eps / 40


@pytest.mark.parametrize("mode", [1, 2, 3])
def test_gelu_special_values(oracle, mode):
    y = oracle.gelu(np.array([0.0, 5.5, 8.0, 100.0, 3e4], np.float32), "f32", mode)
    assert y[0] == 0.0
    assert np.array_equal(y[1:], np.array([5.5, 8.0, 100.0, 3e4], np.float32))
    # very negative inputs: e overflows to +inf after the clamp, output is -0
    yn = oracle.gelu(np.array([-11.0, -50.0], np.float32), "f32", mode)
    assert np.all(yn == 0.0)


# ------------------------------ logistic / SiLU -----------------------------

@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_sigmoid_bound(oracle, mode):
    x = np.concatenate([np.linspace(-30, 30, 300001), [-80, 80, -88, 88, -100, 100]]).astype(np.float32)
    y = oracle.sigmoid(x, "f32", mode).astype(np.float64)
    ref = expit(x.astype(np.float64))
    if mode == 0:
        # rounding of the binary32 argument s = x * fl(-1/ln2) grows with |x|
        rel = 4 * 2.0 ** -24 * (1 + np.abs(x.astype(np.float64)))
        assert np.all(np.abs(y - ref) <= rel * ref + 2.0 ** -126)
    else:
        eps = EPS[mode]
        assert np.all(np.abs(y - ref) <= eps / (4 * (1 - eps)) + 2.0 ** -24)


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_silu_bound(oracle, mode):
    x = np.linspace(-40, 40, 300001).astype(np.float32)
    y = oracle.sigmoid(x, "f32", mode, silu=True).astype(np.float64)
    xd = x.astype(np.float64)
    ref = xd * expit(xd)
    eps = 4 * 2.0 ** -24 * (1 + np.abs(xd)) if mode == 0 else EPS[mode] / (4 * (1 - EPS[mode]))
    assert np.all(np.abs(y - ref) <= np.abs(xd) * (eps + 2.0 ** -24) + 2.0 ** -126)


def test_sigmoid_special_values(oracle):
    x = np.array([0.0, -np.inf, np.inf, 80.0, -80.0], np.float32)
    for mode in (0, 1, 2, 3):
        y = oracle.sigmoid(x, "f32", mode)
        assert y[1] == 0.0 and y[2] == 1.0 and y[3] == 1.0
        assert 0.0 < y[4] < 1e-33
    assert oracle.sigmoid(x, "f32", 2)[0] == 0.5           # QuAKE2 is exact at 0
    s = oracle.sigmoid(x[:1], "f32", 2, silu=True)
    assert s[0] == 0.0


# ------------------------------ e^(a x + b) ---------------------------------

@pytest.mark.parametrize("a,b", [(1.0, 0.0), (-1.0, 0.0), (0.37, 2.0), (-3.0, -1.5), (10.0, 5.0)])
@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_affine_exp_against_exact(oracle, a, b, mode):
    x = np.random.default_rng(12).uniform(-8, 8, 200000).astype(np.float32)
    y = oracle.exp(x, "f32", mode, a=a, b=b).astype(np.float64)
    ref = np.exp(np.float64(a) * x + np.float64(b))
    ok = (ref > 2.0 ** -125) & (ref < 3e38)
    rel = np.abs(y[ok] / ref[ok] - 1)
    if mode == 0:
        # binary32 rounding of the folded constants and of s, then exact exp2
        s = np.abs(np.float64(a) * x[ok] + b) / LN2
        assert np.all(rel <= 4 * 2.0 ** -24 * (1 + s * LN2) + 1e-12)
    else:
        # folded constants are rounded once; the argument keeps ~2^-17 relative spacing
        assert rel.max() <= EPS[mode] + 2e-5 * max(1.0, abs(a) * 8 + abs(b)) / 8


def test_folded_exp_equals_raw_quake(oracle):
    c = oracle.constants()
    x = np.random.default_rng(13).uniform(-87, 88, 100000).astype(np.float32)
    assert np.array_equal(oracle.exp(x, "f32", 2), oracle.quake(x, c["C0_EXP"], c["K127"], 2))
    assert np.array_equal(oracle.exp(x, "f32", 1), oracle.quake(x, c["C0_EXP"], c["C1_Q1"], 1))
    assert np.array_equal(oracle.sigmoid(x, "f32", 2),
                          (1.0 / (1.0 + oracle.quake(x, c["C0_NEG"], c["K127"], 2).astype(np.float64)))
                          .astype(np.float32))


def test_exact_mode_exponential_is_binary32(oracle):
    # reading: the comparison operators compute in single precision (Sec. II-A),
    # so their exponential overflows to +inf once 2^s exceeds the binary32 range
    # and the operator output is then exactly -0 / 0.
    g = oracle.gelu(np.array([-10.4, -9.99], np.float32), "f32", 0)
    assert g[0] == 0.0 and np.signbit(g[0])
    assert g[1] < 0 and abs(float(g[1])) > 1e-37       # 2^125.6 is still finite
    s = oracle.sigmoid(np.array([-89.0, -88.0], np.float32), "f32", 0, silu=True)
    assert s[0] == 0.0 and np.signbit(s[0])
    assert s[1] < 0


# ------------------------- unfused operators (Table IV study) ----------------

@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("t", [1.0, 0.125, 2.5])
def test_unfused_softmax_against_exact(oracle, mode, t):
    x = _rows(21, 24, 300, 3.0)
    y = oracle.softmax_unfused(x, "f32", mode, t=t).astype(np.float64)
    ref = sp_softmax(t * x.astype(np.float64), axis=1)
    big = ref > 1e-30
    rel = np.abs(y / ref - 1)[big]
    if mode == 0:
        arg = (t * (x.max(axis=1, keepdims=True) - x).astype(np.float64))[big]
        assert np.all(rel <= 4 * 2.0 ** -24 * (1 + arg) + 2e-7)
    else:
        assert rel.max() <= RATIO[mode]
    s = y.sum(axis=1)
    assert np.all(np.abs(s - 1) <= 300 * 2.0 ** -24)


def test_unfused_softmax_matches_fused_quake2(oracle):
    # folding (v - m) * t into c0, c1 changes only the binary32 rounding of l
    x = _rows(22, 16, 500, 2.0)
    for t in (1.0, 0.125, 3.0):
        a = oracle.softmax(x, "f32", 2, t=t).astype(np.float64)
        b = oracle.softmax_unfused(x, "f32", 2, t=t).astype(np.float64)
        assert np.max(np.abs(a / b - 1)) < 2e-4
        assert not np.array_equal(a, b)


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_unfused_softmax_masking(oracle, mode):
    v = _rows(23, 6, 40, 2.0)
    v[:, 5:17] = -np.inf
    v[2] = -np.inf
    y = oracle.softmax_unfused(v, "f32", mode)
    assert np.all(y[:, 5:17] == 0) and np.all(y[2] == 0)


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_unfused_gelu_against_eq4_and_fused(oracle, mode):
    x = np.linspace(-12, 12, 200001).astype(np.float32)
    y = oracle.gelu_unfused(x, "f32", mode).astype(np.float64)
    ref = _gelu_tanh(x)
    xa = np.abs(x.astype(np.float64))
    if mode == 0:
        # e^s overflows binary32 once s > 88.72 (R20), leaving at most |x| 2^-127
        assert np.all(np.abs(y - ref) <= 3e-5 * np.abs(ref) + xa * 2.0 ** -127 + 1e-40)
    else:
        eps = EPS[mode]
        assert np.all(np.abs(y - ref) <= xa * (eps / (4 * (1 - eps)) + 2.0 ** -23) + 1e-37)
        f = oracle.gelu(x, "f32", mode).astype(np.float64)
        assert np.all(np.abs(y - f) <= 1e-5 * xa + 1e-37)


# ------------------------------ implicit causal mask ------------------------

@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("period,shift", [(16, 0), (16, 3), (10, -2), (7, 100)])
def test_causal_equals_explicit_mask(oracle, mode, period, shift):
    # the implicit mask gives exactly what -inf entries give under Algorithm 2
    rows, cols = 3 * period + 1, 24
    x = _rows(30, rows, cols, 2.0)
    i = (np.arange(rows) % period)[:, None] + shift
    j = np.arange(cols)[None, :]
    xm = np.where(j > i, -np.inf, x).astype(np.float32)
    a = oracle.softmax_causal(x, period, shift, "f32", mode, t=0.7, threads=3)
    b = oracle.softmax(xm, "f32", mode, t=0.7)
    assert np.array_equal(a, b)
    # masked entries are never read: poisoning them changes nothing
    xp = np.where(j > i, np.float32(1e30), x).astype(np.float32)
    assert np.array_equal(oracle.softmax_causal(xp, period, shift, "f32", mode, t=0.7), a)


def test_causal_fully_masked_rows_are_zero(oracle):
    x = _rows(31, 8, 12, 1.0)
    y = oracle.softmax_causal(x, 4, -3, "f32", 2)
    # L = r mod 4 - 2: rows with r mod 4 in {0, 1, 2} have no live entry, r mod 4 = 3 one
    assert np.all(y[0::4] == 0) and np.all(y[1::4] == 0) and np.all(y[2::4] == 0)
    assert np.all(y[3::4, 0] == 1.0) and np.all(y[3::4, 1:] == 0)
