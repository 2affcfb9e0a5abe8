"""The parity comparators themselves (CPU): they accept what the tolerance
allows and reject a single flipped output bit."""
import numpy as np
import pytest

from compare import check, check_16, check_bits, check_f32, ulp_distance


def test_ulp_distance_crosses_zero():
    a = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x3C00], np.uint16)
    b = np.array([0x8000, 0x0000, 0x8001, 0x0001, 0x3C01], np.uint16)
    assert ulp_distance(a, b, 16).tolist() == [0, 0, 2, 2, 1]


def test_bit_flip_fails_bit_exact():
    r = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    assert check_bits(r.copy(), r) is None
    g = r.copy()
    g.view(np.uint32)[1234] ^= 1
    assert check_bits(g, r) is not None


@pytest.mark.parametrize("bit", [5, 10, 22, 27, 31])   # 1e-6 admits ~8-16 ulp
def test_bit_flip_fails_f32_tolerance(bit):
    r = (np.random.default_rng(1).random(5000) + 0.5).astype(np.float32)
    assert check_f32(r.copy(), r) is None
    g = r.copy()
    g.view(np.uint32)[77] ^= (1 << bit)
    assert check_f32(g, r) is not None


def test_f32_tolerance_accepts_small_and_subnormal_differences():
    r = np.array([1.0, 1e-30, 1e-39, 0.0, np.inf], np.float32)
    g = np.array([1.0 + 2 ** -22, 1e-30 * (1 + 5e-7), 0.0, 1e-39, np.inf], np.float32)
    assert check_f32(g, r) is None
    assert check_f32(np.array([np.nan], np.float32), np.array([1.0], np.float32)) is not None


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_16bit_one_ulp(dt):
    r = np.arange(0x0400, 0x7000, dtype=np.uint16)
    assert check_16(r + 1, r, dt) is None
    assert check_16(r + 2, r, dt) is not None
    g = r.copy()
    g[100] ^= 0x0100
    assert check_16(g, r, dt) is not None


def test_check_dispatch():
    r = np.ones(8, np.float32)
    assert check(r, r, "f32", "exact_bits") is None
    g = r.copy()
    g.view(np.uint32)[0] += 3
    assert check(g, r, "f32", "exp_exact") is not None
    assert check(g, r, "f32", "op") is None      # 3 ulp of 1.0 is inside 1e-6


def test_bf16_subnormal_floor():
    # bfloat16 subnormals (below 2^-126) may flush to zero; f16 has no such floor
    r = np.array([0x001F, 0x0005, 0x807F], np.uint16)
    g = np.zeros(3, np.uint16)
    assert check_16(g, r, "bf16") is None
    assert check_16(g, np.array([0x0081, 0x0005, 0x807F], np.uint16), "bf16") is not None
    assert check_16(g, np.array([0x0003, 0, 0], np.uint16), "f16") is not None
