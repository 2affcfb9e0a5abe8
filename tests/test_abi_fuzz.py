"""Seeded random checks of the C ABI's argument validation (no GPU): every
entry point is called with one to three of its arguments replaced by values
the header documents as invalid (negative or oversized sizes, strides below
the row length, NULL or misaligned pointers, unknown enum values, non-finite
or out-of-range scalars), the rest valid. The call must return the status
the header gives for one of the replaced arguments, before any HIP call (no
launch is ever reached: at least one argument is always invalid)."""
import ctypes
import math
import os

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2412_00408_amd", "libquake.so")

A = 0x10000                      # 16-byte aligned, never dereferenced
I64_MIN, I32_MAX = -(1 << 63), (1 << 31) - 1


@pytest.fixture(scope="module")
def q():
    if not os.path.exists(LIB):
        pytest.fail("libquake.so is not built; run python -m paper_2412_00408_amd.build")
    from paper_2412_00408_amd import quake
    return quake


def _neg(r):
    return int(r.choice([-1, -8, -(1 << 31), I64_MIN, -int(r.integers(1, 1 << 40))]))


def _enum_not_in(r, valid):
    while True:
        v = int(r.choice([-1, len(valid) + 3, 99, -(1 << 31), I32_MAX, int(r.integers(-1000, 1000))]))
        if v not in valid:
            return v


def _bad_positive_scalar(r, big):
    """finite > 0 is required; `big` (or larger) overflows the folded constant"""
    vals = [0.0, -0.0, -1.0, -1e-30, math.nan, math.inf, -math.inf] + ([big, 3.4e38] if big else [])
    return vals[int(r.integers(0, len(vals)))]


def _bad_affine(r):
    vals = [math.nan, math.inf, -math.inf, 3.4e38, -3.4e38]
    return vals[int(r.integers(0, len(vals)))]


def _null_or_misaligned(align):
    def gen(r):
        return None if r.random() < 0.5 else _misaligned(r, align)
    return gen


def _misaligned(r, align):
    while True:
        v = A + int(r.integers(1, 64))
        if v % align:
            return v


# For each entry point: the valid base arguments (in order) and, per argument,
# a generator of invalid values with the status it must give. Each `bad`
# entry: name -> (generator(r), status attribute).
def _specs(q):
    L = q.lib
    ew = dict(x=lambda r: None, y=lambda r: None, n=_neg,
              dt=lambda r: _enum_not_in(r, {0, 1, 2}), mode=lambda r: _enum_not_in(r, {0, 1, 2, 3}))
    ew_codes = dict(x="EINVAL", y="EINVAL", n="EINVAL", dt="EDTYPE", mode="EMODE")
    sm_base = [("x", A), ("y", A), ("rows", 4), ("cols", 8), ("ldx", 8), ("ldy", 8), ("dt", 0),
               ("mode", 2), ("t", 1.0)]
    sm_bad = dict(x=lambda r: None, y=lambda r: None, rows=_neg,
                  cols=lambda r: int(r.choice([0, -1, I64_MIN])),
                  ldx=lambda r: int(r.integers(-(1 << 20), 8)), ldy=lambda r: int(r.integers(-(1 << 20), 8)),
                  dt=lambda r: _enum_not_in(r, {0, 1, 2}), mode=lambda r: _enum_not_in(r, {0, 1, 2, 3}),
                  t=lambda r: _bad_positive_scalar(r, 1e32))
    sm_codes = dict(x="EINVAL", y="EINVAL", rows="EINVAL", cols="EINVAL", ldx="EINVAL",
                    ldy="EINVAL", dt="EDTYPE", mode="EMODE", t="EINVAL")
    unf_bad = dict(sm_bad, t=lambda r: _bad_positive_scalar(r, None))
    ws_cols = 128256
    need = ctypes.c_int64(0)
    assert L.quake_softmax_workspace_size(4, ws_cols, 0, ctypes.byref(need)) == q.OK and need.value > 0
    return {
        "quake_exp": (L.quake_exp,
                      [("x", A), ("y", A), ("n", 1000), ("dt", 0), ("mode", 2), ("a", 1.0), ("b", 0.0),
                       ("s", None)],
                      dict(ew, a=_bad_affine, b=_bad_affine), dict(ew_codes, a="EINVAL", b="EINVAL")),
        "quake_gelu": (L.quake_gelu, [("x", A), ("y", A), ("n", 1000), ("dt", 2), ("mode", 2), ("s", None)],
                       ew, ew_codes),
        "quake_gelu_unfused": (L.quake_gelu_unfused,
                               [("x", A), ("y", A), ("n", 1000), ("dt", 2), ("mode", 2), ("s", None)],
                               ew, ew_codes),
        "quake_sigmoid": (L.quake_sigmoid,
                          [("x", A), ("y", A), ("n", 1000), ("dt", 1), ("mode", 2), ("silu", 1),
                           ("s", None)], ew, ew_codes),
        "quake_exp16": (L.quake_exp16,
                        [("x", A), ("y", A), ("n", 1000), ("dt", 2), ("mode", 2), ("a", 1.0), ("b", 0.0),
                         ("s", None)],
                        dict(ew, dt=lambda r: _enum_not_in(r, {1, 2}), mode=lambda r: _enum_not_in(r, {1, 2}),
                             a=_bad_affine, b=_bad_affine),
                        dict(ew_codes, a="EINVAL", b="EINVAL")),
        "quake_softmax": (L.quake_softmax, sm_base + [("s", None)], sm_bad, sm_codes),
        "quake_softmax_unfused": (L.quake_softmax_unfused, sm_base + [("s", None)], unf_bad, sm_codes),
        "quake_softmax_noalloc": (L.quake_softmax_noalloc, sm_base + [("s", None)], sm_bad, sm_codes),
        "quake_softmax_ws": (L.quake_softmax_ws,
                             [("x", A), ("y", A), ("rows", 4), ("cols", ws_cols), ("ldx", ws_cols),
                              ("ldy", ws_cols), ("dt", 0), ("mode", 2), ("t", 1.0), ("ws", A),
                              ("ws_bytes", need.value), ("s", None)],
                             dict(sm_bad, cols=lambda r: int(r.choice([-1, I64_MIN])),
                                  ldx=lambda r: int(r.integers(-(1 << 20), ws_cols)),
                                  ldy=lambda r: int(r.integers(-(1 << 20), ws_cols)),
                                  ws=lambda r: _misaligned(r, 16),
                                  ws_bytes=lambda r: int(r.integers(I64_MIN, need.value))),
                             dict(sm_codes, ws="EINVAL", ws_bytes="EINVAL")),
        "quake_softmax_causal": (L.quake_softmax_causal,
                                 [("x", A), ("y", A), ("rows", 4), ("cols", 8), ("ldx", 8), ("ldy", 8),
                                  ("period", 8), ("shift", 0), ("wm", 1), ("dt", 0), ("mode", 2),
                                  ("t", 1.0), ("s", None)],
                                 dict(sm_bad, period=lambda r: int(r.choice([0, -1, I32_MAX + 1, I64_MIN])),
                                      shift=lambda r: int(r.choice([(1 << 40) + 1, -(1 << 40) - 1,
                                                                    I64_MIN, (1 << 62)]))),
                                 dict(sm_codes, period="EINVAL", shift="EINVAL")),
        "quake_linear_gelu": (L.quake_linear_gelu,
                              [("x", A), ("w", A), ("y", A), ("m", 256), ("n", 256), ("k", 64), ("ldx", 64),
                               ("ldw", 64), ("ldy", 256), ("dt", 2), ("mode", 2), ("gelu", 1), ("s", None)],
                              dict(x=_null_or_misaligned(16),
                                   w=_null_or_misaligned(16),
                                   y=lambda r: None, m=_neg, n=_neg,
                                   k=lambda r: int(r.choice([0, -8, 57, 63, 65, 71])),
                                   ldx=lambda r: int(r.choice([0, 56, 63, 65, 68, -64])),
                                   ldw=lambda r: int(r.choice([0, 56, 63, 65, 68, -64])),
                                   ldy=lambda r: int(r.integers(-(1 << 20), 256)),
                                   dt=lambda r: _enum_not_in(r, {1, 2}), mode=lambda r: _enum_not_in(r, {0, 1, 2, 3})),
                              dict(x="EINVAL", w="EINVAL", y="EINVAL", m="EINVAL", n="EINVAL", k="EINVAL",
                                   ldx="EINVAL", ldw="EINVAL", ldy="EINVAL", dt="EDTYPE", mode="EMODE")),
        "quake_attention": (L.quake_attention,
                            [("q", A), ("k", A), ("vt", A), ("o", A), ("heads", 4), ("seq", 128), ("dim", 64),
                             ("ldv", 128), ("dt", 2), ("mode", 2), ("t", 0.125), ("causal", 1), ("s", None)],
                            dict(q=_null_or_misaligned(16),
                                 k=_null_or_misaligned(16),
                                 vt=_null_or_misaligned(2),
                                 o=_null_or_misaligned(8),
                                 heads=_neg, seq=_neg,
                                 dim=lambda r: int(r.choice([0, 32, 63, 65, 128, -64])),
                                 ldv=lambda r: int(r.choice([0, 127, -1, I32_MAX + 1])),
                                 dt=lambda r: _enum_not_in(r, {1, 2}), mode=lambda r: _enum_not_in(r, {0, 1, 2, 3}),
                                 t=lambda r: _bad_positive_scalar(r, 3.4e38)),
                            dict(q="EINVAL", k="EINVAL", vt="EINVAL", o="EINVAL", heads="EINVAL", seq="EINVAL",
                                 dim="EINVAL", ldv="EINVAL", dt="EDTYPE", mode="EMODE", t="EINVAL")),
        "quake_stream_copy": (L.quake_stream_copy, [("x", A), ("y", A), ("bytes", 4096), ("shape", 0), ("s", None)],
                              dict(x=_null_or_misaligned(16),
                                   y=_null_or_misaligned(16),
                                   bytes=lambda r: int(r.choice([-16, 8, 4100, 16 << 31, I64_MIN])),
                                   shape=lambda r: int(r.choice([-1, 5, 99, I32_MAX]))),
                              dict(x="EINVAL", y="EINVAL", bytes="EINVAL", shape="EINVAL")),
    }


@pytest.mark.parametrize("name", ["quake_exp", "quake_gelu", "quake_gelu_unfused", "quake_sigmoid",
                                  "quake_exp16", "quake_softmax", "quake_softmax_unfused",
                                  "quake_softmax_noalloc", "quake_softmax_ws", "quake_softmax_causal",
                                  "quake_linear_gelu", "quake_attention", "quake_stream_copy"])
def test_invalid_arguments_give_their_status(q, name):
    fn, base, bad, codes = _specs(q)[name]
    names = [a for a, _ in base]
    r = np.random.default_rng(sum(map(ord, name)))
    for case in range(300):
        chosen = list(r.choice(sorted(bad), size=int(r.integers(1, min(3, len(bad)) + 1)), replace=False))
        args = dict(base)
        for c in chosen:
            args[c] = bad[c](r)
        got = fn(*[args[a] for a in names])
        want = {getattr(q, codes[c]) for c in chosen}
        assert got in want, "%s case %d: %s gave %d, expected one of %s" % (
            name, case, {c: args[c] for c in chosen}, got, sorted(want))


def test_workspace_size_query_rejects_bad_arguments(q):
    L = q.lib
    r = np.random.default_rng(2412)
    out = ctypes.c_int64(0)
    for case in range(300):
        rows, cols, dt, ptr = 64, 128256, 0, ctypes.byref(out)
        kind = int(r.integers(0, 4))
        if kind == 0:
            rows, want = _neg(r), q.EINVAL
        elif kind == 1:
            cols, want = _neg(r), q.EINVAL
        elif kind == 2:
            dt, want = _enum_not_in(r, {0, 1, 2}), q.EDTYPE
        else:
            ptr, want = None, q.EINVAL
        assert L.quake_softmax_workspace_size(rows, cols, dt, ptr) == want, (case, rows, cols, dt)
