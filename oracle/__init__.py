"""CPU oracle for QuAKE (arXiv:2412.00408) — TEST INFRASTRUCTURE.

This package wraps ``quake_oracle.c`` (plain scalar C, built with gcc,
fp-contraction off) with ctypes. Only the test suite, the smoke check and
the CPU baseline of the benchmark may import it; the HIP library and its
Python binding never do, and the two share no code.

Arrays are numpy arrays holding elements of the I/O format:
``float32`` arrays for ``"f32"``, and ``uint16`` (or ``float16``) arrays of
raw bits for ``"f16"`` and ``"bf16"``. Every function returns a new array of
the same numpy dtype as its input.

Parity notes: every function here is pinned by the ``-m "not gpu"`` tests
(closed forms of Eq. 2-3, Algorithm 1's continuity conditions, the error
bounds of Sec. III-A/III-B against exact exp over every binary32 input,
monotonicity, Algorithm 2's invariants, Eq. 4 = Eq. 7, and the rounding and
decoding routines against numpy/torch). No function is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "quake_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# A test may point the wrapper at a deliberately mutated build of the oracle
# (see tests/test_oracle_mutants.py) to show that the pins catch the mistake.
_OVERRIDE = os.environ.get("QUAKE_ORACLE_LIB")

EXACT, Q1, Q2, Q2M, Q2_DIV = 0, 1, 2, 3, 4
DTYPES = {"f32": 0, "f16": 1, "bf16": 2}

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into oracle/liboracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if _OVERRIDE:
            L = ctypes.CDLL(_OVERRIDE)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            L = ctypes.CDLL(_LIB)
        vp, i64, ci, cf = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
        L.qo_constants.argtypes = [vp]
        L.qo_softmax_c0.argtypes = [cf, ci]
        L.qo_softmax_c0.restype = cf
        L.qo_quake.argtypes = [vp, vp, i64, cf, cf, ci]
        L.qo_exp.argtypes = [vp, vp, i64, ci, ci, cf, cf]
        L.qo_sigmoid.argtypes = [vp, vp, i64, ci, ci, ci]
        L.qo_gelu.argtypes = [vp, vp, i64, ci, ci]
        L.qo_softmax.argtypes = [vp, vp, i64, i64, i64, i64, ci, ci, cf, vp]
        L.qo_softmax_unfused.argtypes = [vp, vp, i64, i64, i64, i64, ci, ci, cf, vp]
        L.qo_softmax_causal.argtypes = [vp, vp, i64, i64, i64, i64, i64, i64, ci, ci, cf, vp]
        L.qo_gelu_unfused.argtypes = [vp, vp, i64, ci, ci]
        L.qo_round.argtypes = [vp, vp, i64, ci]
        L.qo_decode.argtypes = [vp, vp, i64, ci]
        L.qo_softmax_numerators.argtypes = [vp, vp, vp, i64, i64, ci, cf]
        L.qo_softmax_numerators.restype = ci
        L.qo_gelu_f32in.argtypes = [vp, vp, i64, ci, ci]
        L.qo_gelu_f32in.restype = ci
        L.qo_exp16.argtypes = [vp, vp, i64, ci, ci, cf, cf]
        L.qo_exp16.restype = ci
        L.qo_q2m_coefficients.argtypes = [vp]
        L.qo_q2m_coefficients.restype = None
        for f in (L.qo_quake, L.qo_exp, L.qo_sigmoid, L.qo_gelu, L.qo_softmax,
                  L.qo_softmax_unfused, L.qo_gelu_unfused, L.qo_softmax_causal, L.qo_round,
                  L.qo_decode):
            f.restype = ci
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _check(rc: int):
    if rc != 0:
        raise ValueError("oracle call failed with code %d" % rc)


def _prep(x: np.ndarray, dt: str) -> np.ndarray:
    if dt not in DTYPES:
        raise ValueError(dt)
    want = np.float32 if dt == "f32" else (np.uint16, np.float16)
    if dt == "f32" and x.dtype != np.float32:
        raise TypeError("f32 oracle input must be float32")
    if dt != "f32" and x.dtype not in want:
        raise TypeError("16-bit oracle input must be uint16 or float16 bits")
    return np.ascontiguousarray(x)


def _split(n: int, threads: int):
    threads = max(1, min(threads, n))
    step = -(-n // threads)
    return [(s, min(n, s + step)) for s in range(0, n, step)]


def constants() -> dict:
    out = np.zeros(10, np.float32)
    lib().qo_constants(_ptr(out))
    names = ["C0_EXP", "K127", "C1_Q1", "L_HI", "A_GELU", "C0_GELU", "THIRD",
             "C0_NEG", "LOG2E", "C0E_GELU"]
    return dict(zip(names, out.tolist()))


def q2m_coefficients() -> dict:
    """Minimax coefficients of Eq. 6 (mode Q2M): a0, a1, a2 in double and as
    the binary32 values the approximation uses, the worst-case relative error E
    and the four equioscillation points in a_m."""
    out = np.zeros(8, np.float64)
    lib().qo_q2m_coefficients(_ptr(out))
    a = out[:3].copy()
    return dict(a=a, a_f32=a.astype(np.float32), err=float(out[3]), ref=out[4:8].copy())


def softmax_c0(t: float, mode: int) -> float:
    return float(lib().qo_softmax_c0(t, mode))


def quake(x: np.ndarray, c0: float, c1: float, order: int) -> np.ndarray:
    """Raw QuAKE (order Q1) / QuAKE2 (Q2, Q2M, Q2_DIV) of binary32 inputs."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty_like(x)
    _check(lib().qo_quake(_ptr(x), _ptr(y), x.size, c0, c1, order))
    return y


def _elementwise(fn, x, dt, extra, threads):
    x = _prep(x, dt)
    y = np.empty_like(x)
    n = x.size
    isz = x.itemsize
    xb, yb = _ptr(x), _ptr(y)

    def run(rng):
        s, e = rng
        _check(fn(xb + s * isz, yb + s * isz, e - s, DTYPES[dt], *extra))

    if threads <= 1 or n < 4096:
        if n:
            run((0, n))
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, _split(n, threads)))
    return y


def exp(x, dt="f32", mode=Q2, a=1.0, b=0.0, threads=1):
    """y = e^(a x + b) (Sec. III-A)."""
    return _elementwise(lib().qo_exp, x, dt, (mode, ctypes.c_float(a), ctypes.c_float(b)), threads)


def sigmoid(x, dt="f32", mode=Q2, silu=False, threads=1):
    """Logistic (silu=False) or SiLU (silu=True)."""
    return _elementwise(lib().qo_sigmoid, x, dt, (mode, int(bool(silu))), threads)


def gelu(x, dt="f32", mode=Q2, threads=1):
    """GELU through Eq. 7."""
    return _elementwise(lib().qo_gelu, x, dt, (mode,), threads)


def gelu_unfused(x, dt="f32", mode=Q2, threads=1):
    """GELU through Eq. 7 with the standard exponential plugged in (Table IV study)."""
    return _elementwise(lib().qo_gelu_unfused, x, dt, (mode,), threads)


def softmax_unfused(x, dt="f32", mode=Q2, t=1.0, cols=None, ldx=None, ldy=None, threads=1):
    """Row softmax with (v - m) * t computed before a standard exponential (Table IV study)."""
    return softmax(x, dt, mode, t, cols, ldx, ldy, threads, _fn="qo_softmax_unfused")


def softmax(x, dt="f32", mode=Q2, t=1.0, cols=None, ldx=None, ldy=None, threads=1, _fn="qo_softmax"):
    """Row softmax of t*x (Algorithm 2). x: 2-D array (rows, ldx) of elements.

    If cols < ldx only the first cols elements of each row are used; the
    output has shape (rows, ldy) with untouched padding set to zero.
    """
    x = _prep(x, dt)
    if x.ndim != 2:
        raise ValueError("softmax oracle wants a 2-D array")
    rows, width = x.shape
    cols = width if cols is None else cols
    ldx = width if ldx is None else ldx
    ldy = cols if ldy is None else ldy
    y = np.zeros((rows, ldy), dtype=x.dtype)
    isz = x.itemsize
    xb, yb = _ptr(x), _ptr(y)

    def run(rng):
        s, e = rng
        tmp = np.empty(max(cols, 1), np.float64)
        _check(getattr(lib(), _fn)(xb + s * ldx * isz, yb + s * ldy * isz, e - s, cols, ldx,
                                   ldy, DTYPES[dt], mode, ctypes.c_float(t), _ptr(tmp)))

    if rows == 0:
        return y
    if threads <= 1 or rows < 2:
        run((0, rows))
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, _split(rows, threads)))
    return y


def softmax_causal(x, period, shift=0, dt="f32", mode=Q2, t=1.0, threads=1):
    """Row softmax where entry (r, j) is used iff j <= r mod period + shift
    (the others are not read and give 0). x: 2-D contiguous array."""
    x = _prep(x, dt)
    rows, cols = x.shape
    y = np.zeros((rows, cols), dtype=x.dtype)
    isz = x.itemsize
    xb, yb = _ptr(x), _ptr(y)

    def run(rng):
        s, e = rng
        tmp = np.empty(max(cols, 1), np.float64)
        # chunks start at multiples of period, so r mod period is the global one
        _check(lib().qo_softmax_causal(xb + s * cols * isz, yb + s * cols * isz, e - s, cols, cols,
                                       cols, period, shift, DTYPES[dt], mode, ctypes.c_float(t),
                                       _ptr(tmp)))

    if rows == 0:
        return y
    step = period * max(1, -(-rows // (period * max(1, threads))))
    ranges = [(s0, min(rows, s0 + step)) for s0 in range(0, rows, step)]
    if threads <= 1 or len(ranges) == 1:
        for rg in ranges:
            run(rg)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, ranges))
    return y


def softmax_numerators(s: np.ndarray, mode: int, t: float = 1.0, threads: int = 1):
    """Algorithm 2 without the division, on binary32 rows: (p, sums) with p the
    binary32 exponentials against each row's max and sums their float64 sums."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    rows, cols = s.shape
    p = np.empty_like(s)
    sums = np.empty(rows, np.float64)

    def work(r):
        lo, hi = r
        _check(lib().qo_softmax_numerators(_ptr(s[lo:]), _ptr(p[lo:]), _ptr(sums[lo:]), hi - lo,
                                           cols, mode, t))

    with ThreadPoolExecutor(max(1, threads)) as ex:
        list(ex.map(work, _split(rows, threads)))
    return p, sums


def attention(q: np.ndarray, k: np.ndarray, vt: np.ndarray, mode: int, t: float,
              causal: bool = True, threads: int = 1, dt: str = "bf16") -> np.ndarray:
    """softmax(t q k^T) v per head with the softmax of Algorithm 2, for 16-bit
    (dt: "bf16" or "f16") q, k [h, s, d] and vt [h, d, >= s] (v transposed, raw
    bits; columns past s are ignored). Heads are independent and are taken a
    few at a time."""
    h, s_len, d = q.shape
    out = np.empty((h, s_len, d), np.uint16)
    for h0 in range(0, h, 4):
        out[h0:h0 + 4] = _attention_heads(q[h0:h0 + 4], k[h0:h0 + 4], vt[h0:h0 + 4], mode, t,
                                          causal, threads, dt)
    return out


def _attention_heads(q, k, vt, mode, t, causal, threads, dt="bf16"):
    """Every query of a few heads (see _attention_core)."""
    h, s_len, d = q.shape
    return _attention_core(q, k, vt, np.arange(s_len), mode, t, causal, threads, dt)


def _attention_core(q, k, vt, rows, mode, t, causal, threads, dt):
    """Queries `rows` (their indices in the sequence; q holds those queries
    only) against all keys. Scores: float64 products of the 16-bit inputs
    rounded once to binary32, causal entries (key > query) set to -inf;
    numerators and sums as softmax_numerators; the numerators rounded to the
    input format for the second product (its operands are in that format),
    that product in float64, divided by the float64 sum, rounded to the input
    format."""
    h, nr, d = q.shape
    s_len = k.shape[1]
    qd = decode(np.ascontiguousarray(q).reshape(-1), dt).astype(np.float64).reshape(h, nr, d)
    kd = decode(np.ascontiguousarray(k).reshape(-1), dt).astype(np.float64).reshape(h, s_len, d)
    vd = decode(np.ascontiguousarray(vt[:, :, :s_len]).reshape(-1), dt).astype(
        np.float64).reshape(h, d, s_len)
    scores = np.matmul(qd, np.transpose(kd, (0, 2, 1))).astype(np.float32)
    if causal:
        mask = np.arange(s_len)[None, :] > np.asarray(rows)[:, None]
        scores[:, mask] = -np.inf
    p, sums = softmax_numerators(scores.reshape(h * nr, s_len), mode, t, threads)
    pb = decode(round_to(p.astype(np.float64).reshape(-1), dt), dt).astype(np.float64)
    o = np.matmul(pb.reshape(h, nr, s_len), np.transpose(vd, (0, 2, 1)))
    with np.errstate(invalid="ignore", divide="ignore"):
        o = np.where(sums.reshape(h, nr, 1) > 0, o / sums.reshape(h, nr, 1), 0.0)
    return round_to(o.reshape(-1), dt).reshape(h, nr, d)


def attention_rows(q: np.ndarray, k: np.ndarray, vt: np.ndarray, rows, mode: int, t: float,
                   causal: bool = True, threads: int = 1, dt: str = "bf16") -> np.ndarray:
    """The outputs of `attention` for the queries `rows` only ([h, len(rows),
    d]): each query against all keys of its head (the causal mask at its own
    index), so sequences too long for the whole score matrix can be checked
    on sampled queries."""
    rows = np.asarray(rows, np.int64)
    h, s_len, d = q.shape
    if rows.size and (rows.min() < 0 or rows.max() >= s_len):
        raise ValueError("query index out of range")
    out = np.empty((h, rows.size, d), np.uint16)
    for h0 in range(0, h, 4):
        sl = slice(h0, h0 + 4)
        out[sl] = _attention_core(q[sl][:, rows], k[sl], vt[sl], rows, mode, t, causal, threads,
                                  dt)
    return out


def linear_gelu(x: np.ndarray, w: np.ndarray, mode: int, gelu: bool = True, dt: str = "bf16",
                threads: int = 1) -> np.ndarray:
    """GELU(x w^T) of 16-bit matrices x [m, k] and w [n, k] (raw bits): the
    product in float64 (every product of two bfloat16 / binary16 values is
    exact there and the sum keeps far more than binary32's precision), rounded
    once to binary32, then GELU of Eq. 7 (or nothing) and rounding to dt."""
    xd = decode(np.ascontiguousarray(x).reshape(-1), dt).astype(np.float64).reshape(x.shape)
    wd = decode(np.ascontiguousarray(w).reshape(-1), dt).astype(np.float64).reshape(w.shape)
    acc = (xd @ wd.T).astype(np.float32)
    if not gelu:
        return round_to(acc.astype(np.float64), dt)
    flat = np.ascontiguousarray(acc).reshape(-1)
    y = np.empty(flat.size, np.uint16)

    def work(r):
        lo, hi = r
        _check(lib().qo_gelu_f32in(_ptr(flat[lo:]), _ptr(y[lo:]), hi - lo, DTYPES[dt], mode))

    with ThreadPoolExecutor(max(1, threads)) as ex:
        list(ex.map(work, _split(flat.size, threads)))
    return y.reshape(acc.shape)


def exp16(x: np.ndarray, dt: str, mode: int, a: float = 1.0, b: float = 0.0,
          threads: int = 1) -> np.ndarray:
    """e^(a x + b) with QuAKE / QuAKE2 built in the 16-bit format's own layout
    (dt "f16" or "bf16"; uint16 raw bits in and out; modes Q1, Q2)."""
    if dt not in ("f16", "bf16"):
        raise ValueError(dt)
    x = _prep(x, dt)
    y = np.empty(x.shape, np.uint16)
    xf = x.reshape(-1).view(np.uint16)
    yf = y.reshape(-1)

    def work(r):
        lo, hi = r
        _check(lib().qo_exp16(_ptr(xf[lo:]), _ptr(yf[lo:]), hi - lo, DTYPES[dt], mode, a, b))

    with ThreadPoolExecutor(max(1, threads)) as ex:
        list(ex.map(work, _split(xf.size, threads)))
    return y


def round_to(v: np.ndarray, dt: str) -> np.ndarray:
    """Round float64 values once to the format dt (RNE)."""
    v = np.ascontiguousarray(v, dtype=np.float64)
    out = np.empty(v.shape, np.float32 if dt == "f32" else np.uint16)
    _check(lib().qo_round(_ptr(v), _ptr(out), v.size, DTYPES[dt]))
    return out


def decode(x: np.ndarray, dt: str) -> np.ndarray:
    """Decode elements of format dt to float32 values."""
    x = _prep(x, dt)
    out = np.empty(x.shape, np.float32)
    _check(lib().qo_decode(_ptr(x), _ptr(out), x.size, DTYPES[dt]))
    return out
