"""Pins of the oracle's GELU(x w^T): its matrix-product step is numpy's float64
product (a library primitive; products of bfloat16 values are exact in
float64), so the pins check the composition: with k = 1 and w = 1 it reduces
to the elementwise GELU of Eq. 7 on bfloat16 inputs (pinned on its own), with
an identity weight and no GELU it reproduces x, and its binary32 rounding of
the sums sits where it should."""
import numpy as np
import pytest

from paper_2412_00408_amd import synth


def _bf16_ones(shape):
    return np.full(shape, 0x3F80, np.uint16)


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_k1_reduces_to_elementwise_gelu(oracle, mode):
    x = synth.bits(synth.normal((4096, 1), 2.0, "bf16", 20))
    y = oracle.linear_gelu(x, _bf16_ones((1, 1)), mode)
    ref = oracle.gelu(x.reshape(-1), "bf16", mode)
    assert np.array_equal(y.reshape(-1), ref)


def test_identity_weight_reproduces_x(oracle):
    x = synth.bits(synth.normal((37, 64), 3.0, "bf16", 21))
    eye = np.where(np.eye(64, dtype=bool), 0x3F80, 0).astype(np.uint16)
    assert np.array_equal(oracle.linear_gelu(x, eye, 2, gelu=False), x)


def test_gelu_f32in_matches_gelu_for_binary32(oracle):
    v = (np.random.default_rng(22).standard_normal(100000) * 4).astype(np.float32)
    for mode in (0, 1, 2, 3):
        a = oracle.linear_gelu  # noqa: F841  (the composition below uses the same C routine)
        y = np.empty(v.size, np.float32)
        ref = oracle.gelu(v, "f32", mode)
        # GELU of binary32 inputs with binary32 output through the matrix path
        # (k = 1 cannot hold arbitrary binary32 inputs, so call the routine directly)
        lib = oracle.lib()
        assert lib.qo_gelu_f32in(v.ctypes.data, y.ctypes.data, v.size, 0, mode) == 0
        assert np.array_equal(y, ref)


def test_sums_rounded_once_to_binary32(oracle):
    # x w^T whose exact value needs more than 24 bits: 1 + 2^-30 style sums
    k = 16
    x = np.full((1, k), 0x3F80, np.uint16)                  # ones
    w = np.zeros((1, k), np.uint16)
    w[0, 0] = 0x3F80                                        # 1
    w[0, 1] = 0x3080                                        # 2^-30
    y = oracle.linear_gelu(x, w, 2, gelu=False, dt="bf16")
    assert int(y[0, 0]) == 0x3F80                           # 1 + 2^-30 rounds to 1
