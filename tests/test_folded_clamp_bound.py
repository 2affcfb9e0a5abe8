"""The folded clamp of Algorithm 2's exponentials, checked in exact binary32
arithmetic on the CPU (no GPU, no library code). The softmax split-row and
attention kernels replace the clamp of l to [0, 255 * 2^23] followed by a
truncating conversion with one saturating unsigned conversion when the row
constant c1 = fma(-c0, m, 127 * 2^23) satisfies |c1| < 2^54. That is the
same integer z only if l = fma(x, c0, c1) can never exceed 255 * 2^23 for an
entry x <= m (the saturating conversion does the lower clamp). Here: that
bound over seeded random and adversarial (t, m, x), including rows whose
|c1| sits just below 2^54, and a counterexample above the threshold showing
that the condition is not vacuous."""
import math
import os
import re

import numpy as np

from fp32ref import f32, fma32

LHI = 255 * 2 ** 23
K127 = f32(127.0 * 2 ** 23)
THRESHOLD = 2.0 ** 54


def c0_of(t):
    # 2^23 t / ln 2, evaluated in double and rounded once to binary32
    return f32((t / math.log(2.0)) * 2.0 ** 23)


def z_clamped(l):
    """clamp to [0, 255 * 2^23], then truncate"""
    return int(min(max(l, 0.0), float(LHI)))


def z_saturating(l):
    """unsigned conversion that truncates and saturates (negative -> 0)"""
    if math.isnan(l) or l <= 0.0:
        return 0
    if l >= 2.0 ** 32:
        return 2 ** 32 - 1
    return int(l)


def below_f32(v):
    return float(np.nextafter(np.float32(v), np.float32(-np.inf)))


def entries(r, m, n):
    """x <= m: the max itself, its lower neighbours, random gaps, -inf"""
    xs = [m, below_f32(m), below_f32(below_f32(m)), -math.inf]
    for _ in range(n):
        gap = float(r.choice([1e-6, 1e-3, 1.0, 30.0, 1e4])) * r.random()
        xs.append(f32(m - abs(m) * gap - gap))
    return [x for x in xs if x <= m]


def check_row(t, m, r, n=6):
    c0 = c0_of(t)
    c1 = fma32(-c0, m, K127)
    if not (abs(c1) < THRESHOLD):
        return 0
    for x in entries(r, m, n):
        l = -math.inf if x == -math.inf else fma32(x, c0, c1)   # masked entry: c0 > 0
        assert l < LHI, (t, m, x, c1, l)
        assert z_saturating(l) == z_clamped(l), (t, m, x, l)
    return 1


def test_bound_holds_below_the_threshold():
    r = np.random.default_rng(2412)
    rows = 0
    for _ in range(600):
        t = float(10.0 ** r.uniform(-3, 3))
        m = f32(float(r.normal(0.0, 10.0 ** r.uniform(0, 6))))
        rows += check_row(t, m, r)
    assert rows > 500


def test_bound_holds_where_c1_is_near_the_threshold():
    # |c1| just below 2^54: c1's rounding error (half an ulp, up to 2^29) is
    # the largest the bound has to absorb
    r = np.random.default_rng(408)
    rows = 0
    for _ in range(400):
        t = float(10.0 ** r.uniform(-2, 2))
        c0 = c0_of(t)
        target = THRESHOLD * (1.0 - float(r.uniform(0.0, 2.0 ** -10)))
        m = f32(-float(r.choice([1.0, -1.0])) * target / c0)
        rows += check_row(t, m, r, n=3)
    assert rows > 300


def test_threshold_is_not_vacuous():
    # well above the threshold the rounding of c1 alone moves l past
    # 255 * 2^23 for the row max itself, so the conversion would differ
    found = False
    for t in (1.0, 0.37, 2.5):
        c0 = c0_of(t)
        for k in range(200):
            m = f32(-(2.0 ** 58) * (1.0 + k / 1024.0) / c0)
            c1 = fma32(-c0, m, K127)
            l = fma32(m, c0, c1)
            if l >= LHI:
                assert z_saturating(l) != z_clamped(l)
                found = True
                break
        if found:
            break
    assert found


def test_the_kernels_use_this_threshold():
    # the device header's check of the row constant is the bound tested above
    src = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                            "paper_2412_00408_amd", "csrc", "quake_device.hpp")).read()
    body = re.search(r"bool row_c1_below\(float c1\) \{(.*?)\n\}", src, re.S).group(1)
    lit = re.search(r"fabsf\(c1\) < (0x1p(\d+)f)", body)
    assert lit is not None and 2.0 ** int(lit.group(2)) == THRESHOLD

