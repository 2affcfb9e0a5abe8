"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function include/quake.h declares, and rejects bad arguments with the
documented status before any HIP call is made."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "quake.h")
LIB = os.path.join(ROOT, "paper_2412_00408_amd", "libquake.so")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(quake_\w+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def q():
    if not os.path.exists(LIB):
        pytest.fail("libquake.so is not built; run python -m paper_2412_00408_amd.build")
    from paper_2412_00408_amd import quake
    return quake


def test_header_declares_the_entry_points():
    names = declared_functions()
    for f in ["quake_exp", "quake_softmax", "quake_gelu", "quake_sigmoid", "quake_status_str",
              "quake_abi_version"]:
        assert f in names


def test_library_exports_every_declared_symbol(q):
    lib = ctypes.CDLL(LIB)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_binding_declares_every_argument_list(q):
    # ctypes passes an undeclared argument as a C int: a 64-bit device pointer
    # or stream handle would be cut to 32 bits. Every entry point the header
    # declares must have its argument types (and return type) set.
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    for name in declared_functions():
        decl = re.search(r"\b%s\s*\(([^)]*)\)" % name, src).group(1).strip()
        nargs = 0 if decl in ("", "void") else decl.count(",") + 1
        fn = getattr(q.lib, name)
        assert fn.argtypes is not None and len(fn.argtypes) == nargs, name
        assert fn.restype is not None, name


def test_version_and_status_strings(q):
    src = open(HEADER).read()
    ver = int(re.search(r"#define QUAKE_ABI_VERSION (\d+)", src).group(1))
    assert q.abi_version() == ver
    for code, tag in [(0, "QUAKE_OK"), (1, "QUAKE_EINVAL"), (2, "QUAKE_EDTYPE"), (3, "QUAKE_EMODE"),
                      (4, "QUAKE_EHIP"), (5, "QUAKE_ENOSCRATCH")]:
        assert q.status_str(code).startswith(tag)
    assert q.status_str(99).startswith("QUAKE_?")


FAKE = 0x1000  # never dereferenced: every call below returns before touching memory


def test_elementwise_validation(q):
    L = q.lib
    for fn, extra in [(L.quake_exp, (1.0, 0.0)), (L.quake_gelu, ()), (L.quake_sigmoid, (0,))]:
        def call(x, y, n, dt, mode, ex=extra):
            return fn(x, y, n, dt, mode, *ex, None)
        assert call(FAKE, FAKE, 0, 0, 2) == q.OK            # empty: no launch
        assert call(None, None, 0, 0, 2) == q.OK
        assert call(FAKE, FAKE, -1, 0, 2) == q.EINVAL
        assert call(None, FAKE, 10, 0, 2) == q.EINVAL
        assert call(FAKE, None, 10, 0, 2) == q.EINVAL
        assert call(FAKE, FAKE, 10, 3, 2) == q.EDTYPE
        assert call(FAKE, FAKE, 10, -1, 2) == q.EDTYPE
        assert call(FAKE, FAKE, 10, 0, 4) == q.EMODE
        assert call(FAKE, FAKE, 10, 0, -1) == q.EMODE
        assert call(FAKE, FAKE, 0, 7, 2) == q.EDTYPE        # enums are checked first
    nan, inf = float("nan"), float("inf")
    assert L.quake_exp(FAKE, FAKE, 10, 0, 2, nan, 0.0, None) == q.EINVAL
    assert L.quake_exp(FAKE, FAKE, 10, 0, 2, 1.0, inf, None) == q.EINVAL
    assert L.quake_exp(FAKE, FAKE, 10, 0, 2, 3e38, 0.0, None) == q.EINVAL   # c0 overflows
    assert L.quake_exp(FAKE, FAKE, 10, 0, 1, -2.9e31, 0.0, None) == q.EINVAL  # 2^23 a / ln2 > max
    assert L.quake_exp(FAKE, FAKE, 10, 0, 2, 1.0, 2.9e31, None) == q.EINVAL   # c1 overflows
    assert L.quake_exp(FAKE, FAKE, 10, 0, 0, 1.0, 2.4e38, None) == q.EINVAL   # b / ln2 > max


def test_softmax_validation(q):
    f = q.lib.quake_softmax
    ok = dict(x=FAKE, y=FAKE, rows=4, cols=8, ldx=8, ldy=8, dt=0, mode=2, t=1.0)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["x"], a["y"], a["rows"], a["cols"], a["ldx"], a["ldy"], a["dt"], a["mode"],
                 a["t"], None)

    assert call(rows=0) == q.OK
    assert call(rows=0, x=None, y=None) == q.OK
    assert call(rows=-1) == q.EINVAL
    assert call(cols=-1) == q.EINVAL
    assert call(cols=0) == q.EINVAL
    assert call(ldx=7) == q.EINVAL
    assert call(ldy=7) == q.EINVAL
    assert call(x=None) == q.EINVAL
    assert call(y=None) == q.EINVAL
    assert call(t=0.0) == q.EINVAL
    assert call(t=-1.0) == q.EINVAL
    assert call(t=float("inf")) == q.EINVAL
    assert call(t=float("nan")) == q.EINVAL
    assert call(t=1e38) == q.EINVAL            # c0 = 2^23 t / ln2 overflows
    assert call(dt=5) == q.EDTYPE
    assert call(mode=9) == q.EMODE


def test_softmax_workspace_size_and_validation(q):
    import ctypes
    L = q.lib

    def size(rows, cols, dt=0):
        c = ctypes.c_int64(-1)
        rc = L.quake_softmax_workspace_size(rows, cols, dt, ctypes.byref(c))
        return rc, c.value
    # rows that fit one workgroup (<= 16384 elements) or need more than 256
    # chunks take no workspace
    assert size(64, 16384) == (q.OK, 0)
    assert size(0, 128256) == (q.OK, 0)
    assert size(64, (1 << 22) + 1) == (q.OK, 0)
    # 64 x 128256: 8 chunks per row, 256 + 12 * 512 + 4 * 64 bytes
    assert size(64, 128256) == (q.OK, 6656)
    assert size(64, 128256, 2) == (q.OK, 6656)             # independent of the format
    assert size(5000, 20000)[1] == ((256 + 12 * 2 * 1024 + 4 * 1024 + 255) // 256) * 256
    assert size(-1, 10)[0] == q.EINVAL and size(1, -1)[0] == q.EINVAL
    assert size(1, 10, 7)[0] == q.EDTYPE
    assert L.quake_softmax_workspace_size(1, 10, 0, None) == q.EINVAL

    A = 0x10000   # 16-byte aligned, never dereferenced

    def call(ws=A, nbytes=6656, rows=64, cols=128256):
        return L.quake_softmax_ws(A, A, rows, cols, cols, cols, 0, 2, 1.0, ws, nbytes, None)
    assert call(nbytes=6655) == q.EINVAL                   # smaller than the size query
    assert call(ws=A + 8) == q.EINVAL                      # not 16-byte aligned
    assert call(nbytes=-1) == q.EINVAL
    assert call(rows=0) == q.OK                            # empty: nothing launched


def test_binding_rejects_host_tensors(q):
    import torch
    with pytest.raises(ValueError):
        q.quake_gelu(torch.zeros(4))
    with pytest.raises(ValueError):
        q.quake_softmax(torch.zeros(2, 4))


def test_causal_and_unfused_validation(q):
    L = q.lib
    # quake_softmax_causal(x, y, rows, cols, ldx, ldy, period, shift, write_masked, dt, mode, t, s)
    assert L.quake_softmax_causal(FAKE, FAKE, 0, 8, 8, 8, 4, 0, 1, 0, 2, 1.0, None) == q.OK
    assert L.quake_softmax_causal(FAKE, FAKE, 4, 8, 8, 8, 0, 0, 1, 0, 2, 1.0, None) == q.EINVAL
    assert L.quake_softmax_causal(FAKE, FAKE, 4, 8, 8, 8, -3, 0, 1, 0, 2, 1.0, None) == q.EINVAL
    assert L.quake_softmax_causal(FAKE, FAKE, 4, 8, 8, 8, 1 << 31, 0, 1, 0, 2, 1.0, None) == q.EINVAL
    assert L.quake_softmax_causal(FAKE, FAKE, 4, 8, 8, 8, 4, 1 << 41, 1, 0, 2, 1.0, None) == q.EINVAL
    assert L.quake_softmax_causal(FAKE, FAKE, 4, 8, 7, 8, 4, 0, 1, 0, 2, 1.0, None) == q.EINVAL
    assert L.quake_softmax_causal(FAKE, FAKE, 4, 8, 8, 8, 4, 0, 1, 9, 2, 1.0, None) == q.EDTYPE
    assert L.quake_softmax_unfused(FAKE, FAKE, 4, 8, 8, 8, 0, 2, 0.0, None) == q.EINVAL
    assert L.quake_softmax_unfused(FAKE, FAKE, 0, 8, 8, 8, 0, 2, 1.0, None) == q.OK
    assert L.quake_gelu_unfused(FAKE, FAKE, -1, 0, 2, None) == q.EINVAL
    assert L.quake_gelu_unfused(FAKE, FAKE, 10, 0, 5, None) == q.EMODE


def test_exp16_validation(q):
    L = q.lib
    # quake_exp16(x, y, n, dtype, mode, a, b, stream)
    assert L.quake_exp16(FAKE, FAKE, 0, 1, 2, 1.0, 0.0, None) == q.OK
    assert L.quake_exp16(None, None, 0, 2, 1, 1.0, 0.0, None) == q.OK
    assert L.quake_exp16(FAKE, FAKE, 10, 0, 2, 1.0, 0.0, None) == q.EDTYPE     # binary32
    assert L.quake_exp16(FAKE, FAKE, 10, 3, 2, 1.0, 0.0, None) == q.EDTYPE
    assert L.quake_exp16(FAKE, FAKE, 10, 1, 0, 1.0, 0.0, None) == q.EMODE      # EXACT
    assert L.quake_exp16(FAKE, FAKE, 10, 1, 3, 1.0, 0.0, None) == q.EMODE      # QUAKE_2M
    assert L.quake_exp16(FAKE, FAKE, -1, 1, 2, 1.0, 0.0, None) == q.EINVAL
    assert L.quake_exp16(None, FAKE, 10, 1, 2, 1.0, 0.0, None) == q.EINVAL
    assert L.quake_exp16(FAKE, FAKE, 10, 1, 2, float("inf"), 0.0, None) == q.EINVAL
    assert L.quake_exp16(FAKE, FAKE, 10, 2, 2, 1.0, float("nan"), None) == q.EINVAL
    assert L.quake_exp16(FAKE, FAKE, 10, 1, 2, 3e38, 0.0, None) == q.EINVAL      # c0 overflows


def test_linear_gelu_validation(q):
    L = q.lib
    A = 0x10000   # 16-byte aligned, never dereferenced

    def call(m=256, n=256, k=64, ldx=64, ldw=64, ldy=256, dt=2, mode=2, x=A, w=A, y=A):
        return L.quake_linear_gelu(x, w, y, m, n, k, ldx, ldw, ldy, dt, mode, 1, None)
    assert call(m=0) == q.OK and call(n=0) == q.OK
    assert call(dt=0) == q.EDTYPE and call(dt=3) == q.EDTYPE   # binary32, unknown
    assert call(mode=7) == q.EMODE
    assert call(k=0) == q.EINVAL
    assert call(k=60, ldx=64, ldw=64) == q.EINVAL         # k not a multiple of 8
    assert call(ldx=32) == q.EINVAL                        # ldx < k
    assert call(ldx=68) == q.EINVAL                        # ldx not a multiple of 8
    assert call(ldy=255) == q.EINVAL
    assert call(x=A + 2) == q.EINVAL                       # misaligned x
    assert call(w=A + 8) == q.EINVAL
    assert call(y=0) == q.EINVAL
    assert call(m=-1) == q.EINVAL
    big = (1 << 31) - 128                                  # within two slabs of 2^31
    assert call(k=big, ldx=big, ldw=big) == q.EINVAL


def test_attention_validation(q):
    L = q.lib
    A = 0x10000   # 16-byte aligned, never dereferenced

    def call(h=4, s=128, d=64, ldv=128, dt=2, mode=2, t=0.125, qp=A, kp=A, vp=A, op=A):
        return L.quake_attention(qp, kp, vp, op, h, s, d, ldv, dt, mode, t, 1, None)
    assert call(h=0) == q.OK and call(s=0, ldv=0) == q.OK
    assert call(h=0, qp=None, kp=None, vp=None, op=None) == q.OK
    assert call(dt=0) == q.EDTYPE and call(dt=3) == q.EDTYPE   # binary32, unknown
    assert call(mode=9) == q.EMODE
    assert call(d=128) == q.EINVAL                         # head dimension 64 only
    assert call(s=131073, ldv=131080) == q.EINVAL          # longer than 131072
    assert call(s=130, ldv=128) == q.EINVAL                # ldv < seq
    assert call(t=0.0) == q.EINVAL and call(t=float("nan")) == q.EINVAL
    assert call(t=1e38) == q.EINVAL                        # c0 overflows
    assert call(qp=A + 8) == q.EINVAL and call(vp=A + 1) == q.EINVAL
    assert call(op=A + 2) == q.EINVAL
    assert call(kp=None) == q.EINVAL
    assert call(h=-1) == q.EINVAL


def test_attention_vt_row_stride(q):
    import torch
    f = q._vt_row_stride
    vt = torch.empty((2, 3, 64, 40))
    assert f(tuple(vt.shape), vt.stride()) == 40
    padded = torch.empty((2, 3, 64, 48))[..., :40]
    assert f(tuple(padded.shape), padded.stride()) == 48
    with pytest.raises(ValueError):
        t = torch.empty((2, 3, 40, 64)).transpose(-1, -2)       # v, not v^T, in memory
        f(tuple(t.shape), t.stride())
    with pytest.raises(ValueError):
        t = torch.empty((3, 2, 64, 40)).transpose(0, 1)         # heads out of order
        f(tuple(t.shape), t.stride())


def test_span_of_views(q):
    import torch
    t = torch.empty((4, 10))
    assert q._span(t) == (t.data_ptr(), t.data_ptr() + 160)
    v = t[:, 2:5]
    assert q._span(v) == (t.data_ptr() + 8, t.data_ptr() + 4 * (3 * 10 + 5))
    assert q._span(torch.empty(0)) == (0, 0)
