"""Pins of the oracle's scalar QuAKE / QuAKE2 and of its I/O conversions.

Each test checks the oracle against something the paper or IEEE-754 fixes
independently of the oracle's own code: the closed form of Eq. 2-3 at dyadic
inputs, Algorithm 1's continuity conditions, special values, the single-fma
evaluation of Eq. 5, and library rounding routines.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from fp32ref import bits32, f32, fma32, from_bits32, mul32

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))
LN2 = math.log(2.0)


def test_constants_follow_their_definitions(oracle):
    c = oracle.constants()
    lm = GOLD["ieee_binary32"]["l_m"]
    B = GOLD["ieee_binary32"]["B"]
    beta = GOLD["schraudolph_bias"]["value"]
    assert c["C0_EXP"] == f32(2.0 ** lm / LN2)                 # 2^23 log2 e
    assert c["K127"] == float(B * 2 ** lm)                     # exact in binary32
    assert c["C1_Q1"] == f32((B - beta) * 2 ** lm)
    assert c["L_HI"] == float(255 * 2 ** lm)
    assert int(c["L_HI"]) == 0x7F800000 and from_bits32(int(c["L_HI"])) == math.inf  # z = bits of +inf
    assert c["A_GELU"] == f32(1.0 / GOLD["gelu_tanh"]["c"])
    k = 2 * 0.044715 * math.sqrt(2 / math.pi)
    assert c["C0_GELU"] == f32(-(k / LN2) * 2 ** lm)
    assert c["THIRD"] == f32(1.0 / 3.0)
    assert c["C0_NEG"] == -c["C0_EXP"]
    # bit patterns (hex) of the pinned constants
    assert bits32(c["C0_EXP"]) == 0x4B38AA3B
    assert bits32(c["K127"]) == 0x4E7E0000
    assert bits32(c["C1_Q1"]) == 0x4E7DE9AD
    assert bits32(c["C0_GELU"]) == 0xC952D3E8
    assert bits32(c["THIRD"]) == 0x3EAAAAAB


def test_softmax_c0_matches_algorithm2(oracle):
    # c0 = 2^23 t / ln 2 (Algorithm 2); EXACT mode drops the 2^23
    assert oracle.softmax_c0(1.0, oracle.Q2) == f32(2 ** 23 / LN2)
    assert bits32(oracle.softmax_c0(0.125, oracle.Q2)) == 0x49B8AA3B
    assert oracle.softmax_c0(1.0, oracle.EXACT) == f32(1 / LN2)
    for t in [0.3, 2.0, 17.5]:
        assert oracle.softmax_c0(t, oracle.Q1) == f32((t / LN2) * 2 ** 23)


BASE2 = (float(2 ** 23), float(127 * 2 ** 23))   # c0, c1 that make QuAKE compute 2^x
LOW_BINADE = (float(2 ** 23), float(2 ** 23))     # computes 2^(x - 126), l exact for x in [0, 1)


@pytest.mark.parametrize("order", ["Q1", "Q2", "Q2_DIV"])
def test_integer_powers_of_two_are_exact(oracle, order):
    # Eq. 2: the secant 1 + {x} is exact at {x} = 0; Algorithm 1's refinement
    # keeps y_m(1) = 1 (continuity condition of Sec. III-B).
    k = np.arange(-126, 128, dtype=np.float32)
    y = oracle.quake(k, *BASE2, getattr(oracle, order))
    assert np.array_equal(y, np.ldexp(np.float32(1), k.astype(np.int32)))


def test_first_order_closed_form_on_dyadic_inputs(oracle):
    # Eq. 2-3: 2^x ~ 2^floor(x) * (1 + {x}) exactly, for x = k + j/2^16
    r = np.random.default_rng(7)
    k = r.integers(-126, 128, 20000)
    j = r.integers(0, 2 ** 16, 20000)
    x = (k + j / 2.0 ** 16).astype(np.float32)
    assert np.array_equal(x.astype(np.float64), k + j / 2.0 ** 16)
    y = oracle.quake(x, *BASE2, oracle.Q1)
    want = np.ldexp(1.0 + j / 2.0 ** 16, k)
    assert np.array_equal(y.astype(np.float64), want)


def _ym_exact(am: float) -> float:
    """fl32(fl32(a_m^2 + 2) * fl32(1/3)) evaluated exactly (Eq. 6, a0=1/3, a2=2/3)."""
    return mul32(fma32(am, am, 2.0), f32(1.0 / 3.0))


def test_second_order_closed_form_on_dyadic_inputs(oracle):
    # Algorithm 1: result = 2^floor(x) * y_m(1 + {x}), the exponent of z joined
    # to the refined mantissa, for inputs where l is exact.
    r = np.random.default_rng(8)
    k = r.integers(-126, 128, 3000)
    j = r.integers(0, 2 ** 16, 3000)
    x = (k + j / 2.0 ** 16).astype(np.float32)
    y = oracle.quake(x, *BASE2, oracle.Q2)
    for xi, yi, ki, ji in zip(x, y, k, j):
        ym = _ym_exact(1.0 + ji / 2.0 ** 16)
        assert float(yi) == math.ldexp(ym, int(ki)), (xi, yi)


def test_refined_mantissa_is_continuous_and_below_two(oracle):
    # Sec. III-B: y_m = 1 at a_m = 1 and y_m -> 2 as a_m -> 2; the refinement
    # never reaches 2 (so it never carries into the exponent), and it is
    # monotone over all 2^23 mantissas.
    # c1 = 1 * 2^23 keeps l = (1 + f) 2^23 < 2^24 exact, so z takes every
    # mantissa and the result is 2^-126 * y_m(1 + f).
    f = (np.arange(2 ** 23, dtype=np.float64) / 2 ** 23).astype(np.float32)
    y = np.ldexp(oracle.quake(f, *LOW_BINADE, oracle.Q2), 126)
    assert y[0] == 1.0
    assert np.all(y >= 1.0) and np.all(y < 2.0)
    assert np.all(np.diff(y) >= 0)
    assert y[-1] >= 2.0 - 2.0 ** -21
    # deviation from 2^f stays inside the paper's 0.34 % (Sec. III-B)
    dev = y.astype(np.float64) / np.exp2(f.astype(np.float64)) - 1
    assert np.max(np.abs(dev)) < GOLD["continuity_coefficients"]["max_rel_deviation"] + 5e-5


def test_second_order_literal_division_is_within_two_ulp(oracle):
    # reading: (a_m^2 + 2)/3 is evaluated as fmaf(a_m, a_m, 2) * fl(1/3); the
    # literal division differs by at most 2 ulp and on a minority of inputs.
    f = (np.arange(2 ** 23, dtype=np.float64) / 2 ** 23).astype(np.float32)
    a = oracle.quake(f, *LOW_BINADE, oracle.Q2).view(np.int32)
    b = oracle.quake(f, *LOW_BINADE, oracle.Q2_DIV).view(np.int32)
    d = np.abs(a.astype(np.int64) - b)
    assert d.max() <= 2
    assert 0 < np.count_nonzero(d) < 2 ** 23 // 2


def test_natural_exp_special_values(oracle):
    x = np.array([0.0, -np.inf, np.inf, 89.0, -104.0, 1.0], np.float32)
    y2 = oracle.exp(x, "f32", oracle.Q2)
    y1 = oracle.exp(x, "f32", oracle.Q1)
    assert y2[0] == 1.0                       # QuAKE2 is exact at 0
    assert float(y1[0]) == float.fromhex("0x1.f4d68p-1")   # bias 0.0436 lowers e^0
    for y in (y1, y2):
        assert y[1] == 0.0 and y[2] == np.inf and y[3] == np.inf and y[4] == 0.0
    assert abs(float(y2[5]) / math.e - 1) < 0.0035


def test_affine_map_is_one_fused_multiply_add(oracle):
    # reading: l = x*c0 + c1 is a single binary32 fma (Eq. 5). Find inputs where
    # fma and multiply-then-add disagree and check that the oracle's z (the bits
    # of its first-order result) is the integer part of the fused value.
    c0, c1 = f32(2 ** 23 / LN2), float(127 * 2 ** 23)
    r = np.random.default_rng(9)
    cand = r.uniform(-80, 80, 200000).astype(np.float32)
    unfused = (cand * np.float32(c0)).astype(np.float32) + np.float32(c1)
    hits = []
    for xv, uf in zip(cand[:40000], unfused[:40000]):
        fu = fma32(float(xv), c0, c1)
        if fu != float(uf):
            hits.append((float(xv), fu))
        if len(hits) >= 200:
            break
    assert len(hits) >= 50
    xs = np.array([h[0] for h in hits], np.float32)
    z = oracle.quake(xs, c0, c1, oracle.Q1).view(np.uint32)
    want = np.array([int(h[1]) for h in hits], np.uint32)
    assert np.array_equal(z, want)


def test_l_is_binary32_so_z_is_coarse(oracle):
    # l is a binary32 value: once l >= 2^29 its spacing is >= 64, so z = 0 mod 64
    # (about 17 effective mantissa bits of the result), and z = 0 mod 32 in [2^28, 2^29).
    x = np.random.default_rng(10).uniform(-60, 80, 100000).astype(np.float32)
    z = oracle.exp(x, "f32", oracle.Q1).view(np.uint32).astype(np.int64)
    hi = z >= 2 ** 29
    assert hi.sum() > 1000 and np.all(z[hi] % 64 == 0)
    mid = (z >= 2 ** 28) & (z < 2 ** 29)
    assert mid.sum() > 100 and np.all(z[mid] % 32 == 0) and np.any(z[mid] % 64 == 32)


# ---------------------------------------------------------------------------
# I/O conversions against library routines
# ---------------------------------------------------------------------------

def _hard_doubles(n=200000, seed=11):
    r = np.random.default_rng(seed)
    v = np.concatenate([
        r.standard_normal(n) * 10.0 ** r.integers(-9, 6, n),
        r.uniform(-7e4, 7e4, n // 4),
        np.ldexp(r.integers(1, 4096, n // 4).astype(np.float64), r.integers(-40, -14, n // 4)),
        [0.0, -0.0, np.inf, -np.inf, 65504.0, 65519.99, 65520.0, 1e9, -1e9, 6.1e-5, 6e-8,
         3e-8, 2.98e-8, 1.0 + 2 ** -11, 1.0 + 3 * 2 ** -11, 1.0 + 2 ** -11 + 2 ** -40],
    ])
    return v


def test_round_to_f16_matches_numpy(oracle):
    v = _hard_doubles()
    got = oracle.round_to(v, "f16")
    want = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, want)


def test_round_to_bf16_matches_torch_on_binary32_values(oracle):
    v = _hard_doubles().astype(np.float32)
    v = np.concatenate([v, np.frombuffer(np.random.default_rng(12).bytes(4 * 200000), np.uint32)
                        .view(np.float32)])
    v = v[np.isfinite(v) | np.isinf(v)]
    v = v[~np.isnan(v)]
    got = oracle.round_to(v.astype(np.float64), "bf16")
    want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)


def test_round_to_f32_matches_cast(oracle):
    v = _hard_doubles()
    got = oracle.round_to(v, "f32")
    assert np.array_equal(got.view(np.uint32), v.astype(np.float32).view(np.uint32))


def test_decode_every_16bit_pattern(oracle):
    allb = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    f16 = oracle.decode(allb, "f16")
    ref = allb.view(np.float16).astype(np.float32)
    ok = np.isnan(ref)
    assert np.array_equal(np.isnan(f16), ok)
    assert np.array_equal(f16[~ok].view(np.uint32), ref[~ok].view(np.uint32))
    b16 = oracle.decode(allb, "bf16")
    refb = torch.from_numpy(allb.view(np.int16)).view(torch.bfloat16).float().numpy()
    okb = np.isnan(refb)
    assert np.array_equal(np.isnan(b16), okb)
    assert np.array_equal(b16[~okb].view(np.uint32), refb[~okb].view(np.uint32))


def test_16bit_outputs_are_the_binary32_result_rounded_once(oracle):
    # QuAKE results are binary32 values; a 16-bit output is that value rounded once.
    r = np.random.default_rng(13)
    x32 = (r.standard_normal(50000) * 6).astype(np.float32)
    for dt in ("f16", "bf16"):
        xb = oracle.round_to(x32.astype(np.float64), dt)
        xd = oracle.decode(xb, dt)
        for mode in (oracle.Q1, oracle.Q2):
            y16 = oracle.exp(xb, dt, mode, a=0.7, b=-0.25)
            y32 = oracle.exp(xd, "f32", mode, a=0.7, b=-0.25)
            assert np.array_equal(y16, oracle.round_to(y32.astype(np.float64), dt))
