"""ctypes binding of libquake (include/quake.h) — argument marshalling only.

Every function takes CUDA (HIP) torch tensors, passes their device pointers,
sizes and torch's current stream to the C ABI of the same name, and raises
`QuakeError` on a non-OK status. No arithmetic happens here, and there is no
fallback: importing this module without a built libquake.so raises.

Build the library with ``python -m paper_2412_00408_amd.build``.
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libquake.so")

EXACT, QUAKE_1, QUAKE_2, QUAKE_2M = 0, 1, 2, 3
MODES = {"exact": EXACT, "quake1": QUAKE_1, "quake2": QUAKE_2, "quake2m": QUAKE_2M, EXACT: EXACT,
         QUAKE_1: QUAKE_1, QUAKE_2: QUAKE_2, QUAKE_2M: QUAKE_2M}
DTYPES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}
OK, EINVAL, EDTYPE, EMODE, EHIP, ENOSCRATCH = 0, 1, 2, 3, 4, 5


class QuakeError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__("%s failed: %s" % (fn, status_str(code)))
        self.code = code


def _load() -> ctypes.CDLL:
    if not os.path.exists(_LIB_PATH):
        raise ImportError("libquake.so is not built (%s); run python -m paper_2412_00408_amd.build"
                          % _LIB_PATH)
    L = ctypes.CDLL(_LIB_PATH)
    vp, i64, ci, cf = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
    L.quake_exp.argtypes = [vp, vp, i64, ci, ci, cf, cf, vp]
    L.quake_exp16.argtypes = [vp, vp, i64, ci, ci, cf, cf, vp]
    L.quake_linear_gelu.argtypes = [vp, vp, vp, i64, i64, i64, i64, i64, i64, ci, ci, ci, vp]
    L.quake_softmax.argtypes = [vp, vp, i64, i64, i64, i64, ci, ci, cf, vp]
    L.quake_softmax_ws.argtypes = [vp, vp, i64, i64, i64, i64, ci, ci, cf, vp, i64, vp]
    L.quake_softmax_noalloc.argtypes = [vp, vp, i64, i64, i64, i64, ci, ci, cf, vp]
    L.quake_softmax_workspace_size.argtypes = [i64, i64, ci, ctypes.POINTER(i64)]
    L.quake_gelu.argtypes = [vp, vp, i64, ci, ci, vp]
    L.quake_softmax_unfused.argtypes = [vp, vp, i64, i64, i64, i64, ci, ci, cf, vp]
    L.quake_gelu_unfused.argtypes = [vp, vp, i64, ci, ci, vp]
    L.quake_softmax_causal.argtypes = [vp, vp, i64, i64, i64, i64, i64, i64, ci, ci, ci, cf, vp]
    L.quake_sigmoid.argtypes = [vp, vp, i64, ci, ci, ci, vp]
    L.quake_attention.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, ci, ci, cf, ci, vp]
    L.quake_stream_copy.argtypes = [vp, vp, i64, ci, vp]
    for f in (L.quake_exp, L.quake_exp16, L.quake_linear_gelu, L.quake_softmax, L.quake_gelu,
              L.quake_softmax_ws, L.quake_softmax_workspace_size, L.quake_softmax_noalloc,
              L.quake_sigmoid, L.quake_attention, L.quake_stream_copy,
              L.quake_softmax_unfused, L.quake_gelu_unfused, L.quake_softmax_causal):
        f.restype = ci
    L.quake_status_str.argtypes = [ci]
    L.quake_status_str.restype = ctypes.c_char_p
    L.quake_abi_version.argtypes = []
    L.quake_abi_version.restype = ci
    return L


lib = _load()


def status_str(code: int) -> str:
    return lib.quake_status_str(code).decode()


def abi_version() -> int:
    return lib.quake_abi_version()


def softmax_workspace_size(rows: int, cols: int, dtype=torch.float32) -> int:
    """Bytes of workspace quake_softmax_ws uses for rows x cols (0: none)."""
    c = ctypes.c_int64(0)
    _raise("quake_softmax_workspace_size",
           lib.quake_softmax_workspace_size(rows, cols, DTYPES[dtype], ctypes.byref(c)))
    return c.value


def softmax_workspace(rows: int, cols: int, dtype=torch.float32, device="cuda:0"):
    """A zero-filled device workspace for quake_softmax_ws over rows x cols, or
    None when that shape needs none."""
    n = softmax_workspace_size(rows, cols, dtype)
    return torch.zeros(n, dtype=torch.uint8, device=device) if n else None


def _stream(t: torch.Tensor, stream) -> int:
    if stream is not None:
        return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)
    return int(torch.cuda.current_stream(t.device).cuda_stream)


def _check_io(x: torch.Tensor, y: torch.Tensor | None, contiguous=True) -> torch.Tensor:
    if not x.is_cuda:
        raise ValueError("libquake takes device tensors")
    if x.dtype not in DTYPES:
        raise TypeError("libquake takes float32, float16 or bfloat16 tensors, got %s" % x.dtype)
    if contiguous and not x.is_contiguous():
        raise ValueError("input must be contiguous")
    if y is None:
        y = torch.empty_like(x, memory_format=torch.contiguous_format)
    if y.dtype != x.dtype or y.device != x.device or y.shape != x.shape:
        raise ValueError("output must match the input's dtype, device and shape")
    if contiguous and not y.is_contiguous():
        raise ValueError("output must be contiguous")
    return y


def _raise(fn, rc):
    if rc != OK:
        raise QuakeError(fn, rc)


def quake_exp(x, y=None, mode=QUAKE_2, a=1.0, b=0.0, stream=None):
    """y = e^(a x + b) elementwise."""
    y = _check_io(x, y)
    _raise("quake_exp", lib.quake_exp(x.data_ptr(), y.data_ptr(), x.numel(), DTYPES[x.dtype],
                                      MODES[mode], a, b, _stream(x, stream)))
    return y


def quake_exp16(x, y=None, mode=QUAKE_2, a=1.0, b=0.0, stream=None):
    """y = e^(a x + b) with the approximation built in x's own 16-bit layout."""
    y = _check_io(x, y)
    _raise("quake_exp16", lib.quake_exp16(x.data_ptr(), y.data_ptr(), x.numel(), DTYPES[x.dtype],
                                          MODES[mode], a, b, _stream(x, stream)))
    return y


def quake_gelu(x, y=None, mode=QUAKE_2, stream=None):
    """tanh-form GELU through Eq. 7."""
    y = _check_io(x, y)
    _raise("quake_gelu", lib.quake_gelu(x.data_ptr(), y.data_ptr(), x.numel(), DTYPES[x.dtype],
                                        MODES[mode], _stream(x, stream)))
    return y


def quake_gelu_unfused(x, y=None, mode=QUAKE_2, stream=None):
    """GELU with the standard exponential plugged in (fusion study, Table IV)."""
    y = _check_io(x, y)
    _raise("quake_gelu_unfused", lib.quake_gelu_unfused(x.data_ptr(), y.data_ptr(), x.numel(),
                                                        DTYPES[x.dtype], MODES[mode],
                                                        _stream(x, stream)))
    return y


def quake_sigmoid(x, y=None, mode=QUAKE_2, silu=False, stream=None):
    """Logistic sigma(x), or SiLU x*sigma(x) with silu=True."""
    y = _check_io(x, y)
    _raise("quake_sigmoid", lib.quake_sigmoid(x.data_ptr(), y.data_ptr(), x.numel(),
                                              DTYPES[x.dtype], MODES[mode], int(bool(silu)),
                                              _stream(x, stream)))
    return y


def _rows_view(t: torch.Tensor, what: str):
    """(rows, cols, row stride) of a contiguous tensor, or of a 2-D tensor with a
    contiguous last dimension (a slice of a wider matrix)."""
    cols = t.shape[-1]
    if t.is_contiguous():
        return t.numel() // max(cols, 1) if cols else 0, cols, cols
    if t.dim() == 2 and (t.stride(1) == 1 or cols == 1):
        return t.shape[0], cols, t.stride(0)
    raise ValueError("%s must be contiguous, or 2-D with a contiguous last dimension" % what)


def quake_linear_gelu(x, w, y=None, mode=QUAKE_2, gelu=True, stream=None):
    """y = GELU(x w^T) (or x w^T with gelu=False): bfloat16 or float16 x [m, k]
    and w [n, k] with contiguous rows, binary32 accumulation, y [m, n] in the
    same format."""
    if not (x.is_cuda and w.is_cuda):
        raise ValueError("libquake takes device tensors")
    if x.dim() != 2 or w.dim() != 2 or x.shape[1] != w.shape[1]:
        raise ValueError("x [m, k] and w [n, k] with the same k")
    m, k = x.shape
    n = w.shape[0]
    for t, what in ((x, "x"), (w, "w")):
        if t.dtype not in DTYPES:
            raise TypeError("libquake takes float32, float16 or bfloat16 tensors, got %s" % t.dtype)
        if t.stride(1) != 1:
            raise ValueError("%s must have a contiguous last dimension" % what)
    if y is None:
        y = torch.empty((m, n), dtype=x.dtype, device=x.device)
    if y.shape != (m, n) or y.dtype != x.dtype or y.stride(1) != 1:
        raise ValueError("y must be [m, n] of x's dtype with a contiguous last dimension")
    _raise("quake_linear_gelu", lib.quake_linear_gelu(
        x.data_ptr(), w.data_ptr(), y.data_ptr(), m, n, k, x.stride(0), w.stride(0), y.stride(0),
        DTYPES[x.dtype], MODES[mode], int(bool(gelu)), _stream(x, stream)))
    return y


def _span(t: torch.Tensor):
    """[first, last + 1) byte addresses a tensor view touches (empty: (0, 0))."""
    if t.numel() == 0:
        return 0, 0
    last = sum((n - 1) * st for n, st in zip(t.shape, t.stride()))
    return t.data_ptr(), t.data_ptr() + (last + 1) * t.element_size()


def _vt_row_stride(shape, strides) -> int:
    """Row stride (ldv) of v^T [..., dim, seq]: the last dimension contiguous,
    rows ldv apart, heads dim * ldv apart one after another."""
    dim, seq = shape[-2], shape[-1]
    if seq > 1 and strides[-1] != 1:
        raise ValueError("vt must have a contiguous last dimension")
    ldv = strides[-2] if dim > 1 else seq
    want = [ldv, 1]
    for i in range(len(shape) - 3, -1, -1):
        want.insert(0, want[0] * shape[i + 1])
    if any(n > 1 and st != w for n, st, w in zip(shape, strides, want)):
        raise ValueError("vt must be [..., dim, seq] with a contiguous last dimension and "
                         "rows (possibly padded) packed head after head")
    return ldv


def quake_attention(q, k, vt, o=None, mode=QUAKE_2, t=None, causal=True, stream=None):
    """softmax(t q k^T) v per head with Algorithm 2's softmax: bfloat16 or
    float16 q, k [..., seq, 64] and vt = v transposed [..., 64, seq] (or a view
    of wider, padded rows with a contiguous last dimension); returns o
    [..., seq, 64] in the same format. t defaults to 1/sqrt(64)."""
    for a, what in ((q, "q"), (k, "k"), (vt, "vt")):
        if not a.is_cuda:
            raise ValueError("libquake takes device tensors")
        if a.dtype not in DTYPES:
            raise TypeError("libquake takes float32, float16 or bfloat16 tensors, got %s" % a.dtype)
        if a.dim() < 2:
            raise ValueError("%s needs [..., rows, cols]" % what)
    if not (q.is_contiguous() and k.is_contiguous()) or q.shape != k.shape:
        raise ValueError("q and k must be contiguous and of the same shape")
    if k.dtype != q.dtype or vt.dtype != q.dtype:
        raise TypeError("q, k and vt must have the same dtype")
    seq, dim = q.shape[-2], q.shape[-1]
    heads = q.numel() // max(seq * dim, 1)
    if tuple(vt.shape[:-2]) != tuple(q.shape[:-2]) or tuple(vt.shape[-2:]) != (dim, seq):
        raise ValueError("vt must be [..., dim, seq]")
    ldv = _vt_row_stride(tuple(vt.shape), tuple(vt.stride()))
    if o is None:
        o = torch.empty_like(q)
    if o.shape != q.shape or o.dtype != q.dtype or not o.is_contiguous():
        raise ValueError("o must be contiguous and shaped like q")
    o0, o1 = _span(o)
    for a, what in ((q, "q"), (k, "k"), (vt, "vt")):
        a0, a1 = _span(a)
        if o0 < a1 and a0 < o1:
            raise ValueError("o must not overlap %s" % what)
    t = 1.0 / dim ** 0.5 if t is None else t
    _raise("quake_attention", lib.quake_attention(
        q.data_ptr(), k.data_ptr(), vt.data_ptr(), o.data_ptr(), heads, seq, dim, ldv,
        DTYPES[q.dtype], MODES[mode], t, int(bool(causal)), _stream(q, stream)))
    return o


def quake_softmax_unfused(x, y=None, mode=QUAKE_2, t=1.0, stream=None):
    """Softmax with (x - m) * t computed before a standard exponential (Table IV)."""
    return quake_softmax(x, y, mode, t, stream, _fn="quake_softmax_unfused")


def quake_softmax(x, y=None, mode=QUAKE_2, t=1.0, stream=None, workspace=None,
                  _fn="quake_softmax"):
    """Softmax of t*x over the last dimension (Algorithm 2). With `workspace`
    (a zero-filled uint8 device tensor of softmax_workspace_size bytes, e.g.
    from softmax_workspace) rows longer than 16384 elements are split over
    workgroups that exchange their maxima and sums (quake_softmax_ws)."""
    if x.dim() == 0:
        raise ValueError("softmax needs at least one dimension")
    _check_io(x, None, contiguous=False)
    if y is None:
        y = torch.empty_like(x, memory_format=torch.contiguous_format)
    if y.dtype != x.dtype or y.device != x.device or y.shape != x.shape:
        raise ValueError("output must match the input's dtype, device and shape")
    rows, cols, ldx = _rows_view(x, "input")
    _, _, ldy = _rows_view(y, "output")
    args = (x.data_ptr(), y.data_ptr(), rows, cols, ldx, ldy, DTYPES[x.dtype], MODES[mode], t)
    if workspace is not None:
        if _fn != "quake_softmax":
            raise ValueError("%s takes no workspace" % _fn)
        if not workspace.is_cuda or workspace.device != x.device or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on x's device")
        nbytes = workspace.numel() * workspace.element_size()
        _raise("quake_softmax_ws", lib.quake_softmax_ws(*args, workspace.data_ptr(), nbytes,
                                                        _stream(x, stream)))
    else:
        _raise(_fn, getattr(lib, _fn)(*args, _stream(x, stream)))
    return y


def quake_softmax_noalloc(x, y=None, mode=QUAKE_2, t=1.0, stream=None):
    """quake_softmax_ws with the library's fixed device scratch instead of a
    workspace (no allocation; calls must not overlap on one GPU)."""
    return quake_softmax(x, y, mode, t, stream, _fn="quake_softmax_noalloc")


def quake_softmax_causal(x, y=None, period=None, shift=0, mode=QUAKE_2, t=1.0, write_masked=True,
                         stream=None):
    """Softmax of t*x over the last dimension where entry (r, j) is used iff
    j <= r mod period + shift (default period: the row length); masked
    entries are not read and give 0 (left unwritten where a whole 16-byte
    vector is masked, if write_masked is False)."""
    if x.dim() == 0:
        raise ValueError("softmax needs at least one dimension")
    _check_io(x, None, contiguous=False)
    if y is None:
        y = torch.empty_like(x, memory_format=torch.contiguous_format)
    if y.dtype != x.dtype or y.device != x.device or y.shape != x.shape:
        raise ValueError("output must match the input's dtype, device and shape")
    rows, cols, ldx = _rows_view(x, "input")
    _, _, ldy = _rows_view(y, "output")
    period = cols if period is None else period
    _raise("quake_softmax_causal", lib.quake_softmax_causal(
        x.data_ptr(), y.data_ptr(), rows, cols, ldx, ldy, period, shift, int(bool(write_masked)),
        DTYPES[x.dtype], MODES[mode], t, _stream(x, stream)))
    return y
