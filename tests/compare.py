"""Element-by-element comparison of HIP outputs with oracle outputs.

Tolerances (the parity bar):
  * QuAKE / QuAKE2 exp: bit-exact.
  * binary32 outputs of Softmax, GELU, Logistic, SiLU (all modes), and of the
    EXACT exp: |gpu - ref| <= rel * |ref| + 2^-126, rel = 1e-6 (EXACT exp:
    at most 2 ulp apart, plus the same subnormal floor, since v_exp_f32 and
    v_rcp_f32 flush subnormal results).
  * binary16 / bfloat16 outputs: at most 1 ulp apart (distance between the
    ordered integer encodings), i.e. the two binary32 results rounded to
    neighbouring 16-bit values at most; bfloat16 shares binary32's exponent
    range, so the same 2^-126 subnormal floor applies to it.
  * NaN positions must agree; infinities must agree exactly.
"""
from __future__ import annotations

import numpy as np

ABS_FLOOR = 2.0 ** -126
REL_F32 = 1e-6


def _ordered(bits: np.ndarray, width: int) -> np.ndarray:
    b = bits.astype(np.int64) & ((1 << width) - 1)
    sign = 1 << (width - 1)
    mag = b & (sign - 1)
    return np.where(b & sign, -mag, mag)


def ulp_distance(a_bits: np.ndarray, b_bits: np.ndarray, width: int) -> np.ndarray:
    return np.abs(_ordered(a_bits, width) - _ordered(b_bits, width))


def _as_bits(a: np.ndarray) -> tuple[np.ndarray, int]:
    if a.dtype == np.float32:
        return a.view(np.uint32), 32
    if a.dtype in (np.uint16, np.float16):
        return a.view(np.uint16), 16
    if a.dtype == np.uint32:
        return a, 32
    raise TypeError(a.dtype)


def _nan_mask(bits: np.ndarray, width: int, dt: str) -> np.ndarray:
    b = bits.astype(np.int64)
    if width == 32:
        return ((b & 0x7F800000) == 0x7F800000) & ((b & 0x007FFFFF) != 0)
    if dt == "bf16":
        return ((b & 0x7F80) == 0x7F80) & ((b & 0x007F) != 0)
    return ((b & 0x7C00) == 0x7C00) & ((b & 0x03FF) != 0)


def _report(name, bad, gpu, ref, extra=""):
    idx = np.flatnonzero(bad)
    head = idx[:5]
    return "%s: %d of %d elements out of tolerance; first at %s: gpu=%s ref=%s %s" % (
        name, idx.size, bad.size, head.tolist(), np.asarray(gpu).ravel()[head].tolist(),
        np.asarray(ref).ravel()[head].tolist(), extra)


def check_bits(gpu: np.ndarray, ref: np.ndarray, name="bits", ignore=None) -> str | None:
    g, _ = _as_bits(np.ascontiguousarray(gpu).ravel())
    r, _ = _as_bits(np.ascontiguousarray(ref).ravel())
    bad = g != r
    if ignore is not None:
        bad &= ~ignore.ravel()
    return _report(name, bad, g, r) if bad.any() else None


def check_f32(gpu: np.ndarray, ref: np.ndarray, rel=REL_F32, name="f32", ignore=None) -> str | None:
    g = np.ascontiguousarray(gpu, dtype=np.float32).ravel()
    r = np.ascontiguousarray(ref, dtype=np.float32).ravel()
    gn, rn = np.isnan(g), np.isnan(r)
    with np.errstate(invalid="ignore"):
        ok = np.abs(g.astype(np.float64) - r) <= rel * np.abs(r.astype(np.float64)) + ABS_FLOOR
    ok |= (g == r)                       # infinities, signed zeros
    ok |= gn & rn
    ok &= ~(gn ^ rn)
    bad = ~ok
    if ignore is not None:
        bad &= ~ignore.ravel()
    return _report(name, bad, g, r) if bad.any() else None


def check_f32_ulp(gpu: np.ndarray, ref: np.ndarray, max_ulp=2, name="f32ulp") -> str | None:
    g = np.ascontiguousarray(gpu, dtype=np.float32).ravel()
    r = np.ascontiguousarray(ref, dtype=np.float32).ravel()
    d = ulp_distance(g.view(np.uint32), r.view(np.uint32), 32)
    gn, rn = np.isnan(g), np.isnan(r)
    with np.errstate(invalid="ignore"):
        ok = (d <= max_ulp) | (np.abs(g.astype(np.float64) - r) <= ABS_FLOOR)
    ok = np.where(gn | rn, gn & rn, ok)
    bad = ~ok
    return _report(name, bad, g, r) if bad.any() else None


def _decode16(b: np.ndarray, dt: str) -> np.ndarray:
    if dt == "bf16":
        return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return b.view(np.float16).astype(np.float64)


def check_16(gpu_bits: np.ndarray, ref_bits: np.ndarray, dt: str, max_ulp=1, name="16bit") -> str | None:
    g = np.ascontiguousarray(gpu_bits).ravel().view(np.uint16)
    r = np.ascontiguousarray(ref_bits).ravel().view(np.uint16)
    gn, rn = _nan_mask(g, 16, dt), _nan_mask(r, 16, dt)
    d = ulp_distance(g, r, 16)
    with np.errstate(invalid="ignore"):
        near = np.abs(_decode16(g, dt) - _decode16(r, dt)) <= ABS_FLOOR
    ok = np.where(gn | rn, gn & rn, (d <= max_ulp) | near)
    bad = ~ok
    return _report(name, bad, g, r) if bad.any() else None


def check(gpu: np.ndarray, ref: np.ndarray, dt: str, kind: str, name="") -> str | None:
    """kind: 'exact_bits' (QuAKE exp), 'op' (operators), 'exp_exact' (EXACT exp)."""
    if kind == "exact_bits":
        return check_bits(gpu, ref, name)
    if dt == "f32":
        return check_f32_ulp(gpu, ref, 2, name) if kind == "exp_exact" else check_f32(gpu, ref, name=name)
    return check_16(gpu, ref, dt, 1, name)
