"""Seeded random sweeps of shapes, masks, modes and formats for the fused
attention, the softmax, the elementwise operators and the fused linear+GELU,
against the oracle under the same bars as their own test modules:
combinations the hand-picked cases do not cover (head counts and sequence
lengths on both sides of every kernel choice, ragged tails, padded v^T rows,
split rows with and without a workspace, strides, vector lengths across the
launch shapes, GEMM tiles with ragged edges).
Every case is drawn from a fixed seed, so a failure names a reproducible
case; sizes are bounded so that the oracle finishes each in seconds."""
import numpy as np
import pytest
import torch

import test_gpu_attention as ta
import test_gpu_linear as tl
import test_gpu_softmax as ts
from gpu_util import assert_parity, kind_of, run_elementwise, say
from paper_2412_00408_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def q():
    assert torch.cuda.is_available(), "GPU tests need cuda:0"
    from paper_2412_00408_amd import quake
    return quake


def _attention_cases(n, seed):
    """(heads, seq, causal, mode, dt, ldv, seed): lengths around the one-pass
    limits (512, 1024) and the two-pass range, head counts from one to the
    two-group tile counts, at most 40 M query-key pairs per case."""
    rng = np.random.default_rng(seed)
    anchors = [1, 31, 32, 33, 63, 64, 65, 511, 512, 513, 1023, 1024, 1025, 1088, 1100, 1500,
               2047, 2049]
    out = []
    while len(out) < n:
        seq = int(rng.choice(anchors)) if rng.random() < 0.5 else int(rng.integers(1, 2200))
        hmax = max(1, min(64, 40_000_000 // (seq * seq)))
        heads = int(rng.integers(1, hmax + 1))
        causal = bool(rng.random() < 0.5)
        mode = int(rng.integers(0, 4))
        dt = "bf16" if rng.random() < 0.7 else "f16"
        pad = int(rng.choice([0, 0, 0, 3, 8]))
        out.append((heads, seq, causal, mode, dt, seq + pad if pad else None,
                    int(rng.integers(0, 1 << 20))))
    return out


ATTENTION_CASES = _attention_cases(40, 2412)


@pytest.mark.parametrize("heads,seq,causal,mode,dt,ldv,seed", ATTENTION_CASES)
def test_random_attention(q, heads, seq, causal, mode, dt, ldv, seed):
    g, r, ins = ta._run(q, heads, seq, mode, causal, seed, ldv=ldv,
                        pad=float("nan") if ldv else 0.0, dt=dt)
    ta._check(g, r, ins, seq, causal,
              "random attention %s h%d s%d c%d m%d ldv%s seed%d" % (dt, heads, seq, causal, mode,
                                                                    ldv, seed), dt=dt)


def _softmax_cases(n, seed):
    """(rows, cols, dt, mode, t, ld_pad, ws, seed): row lengths across the
    wave-per-row, workgroup-per-row and split kernels (split rows with and
    without a workspace), with and without a row stride, at most 2.5 M
    elements per case."""
    rng = np.random.default_rng(seed)
    anchors = [1, 7, 64, 127, 128, 129, 512, 1000, 4096, 8191, 8192, 16384, 16385, 40000, 128256]
    out = []
    while len(out) < n:
        cols = int(rng.choice(anchors)) if rng.random() < 0.5 else int(rng.integers(1, 140000))
        rows = int(rng.integers(1, max(2, min(300, 2_500_000 // cols)) + 1))
        dt = str(rng.choice(["f32", "bf16", "f16"]))
        mode = int(rng.integers(0, 4))
        t = float(rng.choice([0.125, 0.7, 1.0, 2.5]))
        ld_pad = int(rng.choice([0, 0, 5, 64]))
        ws = bool(cols > 16384 and rng.random() < 0.6)
        out.append((rows, cols, dt, mode, t, ld_pad, ws, int(rng.integers(0, 1 << 20))))
    return out


SOFTMAX_CASES = _softmax_cases(40, 408)


@pytest.mark.parametrize("rows,cols,dt,mode,t,ld_pad,ws,seed", SOFTMAX_CASES)
def test_random_softmax(q, rows, cols, dt, mode, t, ld_pad, ws, seed):
    say("random softmax", dt, rows, cols, mode, t, ld_pad, "workspace" if ws else "", seed)
    x = synth.normal((rows, cols), 3.0, dt, seed)
    g, r, d = ts._run(q, x, mode, t, ld_pad=ld_pad, ws=ws)
    assert_parity(g, r, d, "op", "random softmax %s %dx%d m%d t%g pad%d ws%d seed%d" % (
        dt, rows, cols, mode, t, ld_pad, ws, seed))


def _offset_cases(n, seed):
    """(rows, cols, dt, mode, ld_pad, offset, ws, seed): x and y both a few
    elements past a 16-byte boundary, with ragged lengths and strides, so rows
    start at every offset (the shifted-row kernels and, past their lengths,
    the scalar kernel)."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        cols = int(rng.integers(1, 140000)) if rng.random() < 0.7 else int(rng.integers(1, 600))
        rows = int(rng.integers(1, max(2, min(200, 1_500_000 // cols)) + 1))
        dt = str(rng.choice(["f32", "bf16", "f16"]))
        out.append((rows, cols, dt, int(rng.integers(0, 4)), int(rng.choice([0, 1, 3, 8])),
                    int(rng.integers(1, 8)), bool(cols > 16384 and rng.random() < 0.5),
                    int(rng.integers(0, 1 << 20))))
    return out


@pytest.mark.parametrize("rows,cols,dt,mode,ld_pad,offset,ws,seed", _offset_cases(24, 1001))
def test_random_softmax_offsets(q, rows, cols, dt, mode, ld_pad, offset, ws, seed):
    say("random softmax offsets", dt, rows, cols, mode, ld_pad, offset, "workspace" if ws else "", seed)
    x = synth.normal((rows, cols), 3.0, dt, seed)
    g, r, d = ts._run(q, x, mode, 0.9, ld_pad=ld_pad, offset=offset, ws=ws)
    assert_parity(g, r, d, "op", "random softmax offsets %s %dx%d m%d pad%d off%d ws%d seed%d" % (
        dt, rows, cols, mode, ld_pad, offset, ws, seed))


def _causal_cases(n, seed):
    """(rows, cols, dt, mode, period, shift, seed): implicit causal masks over
    ragged and aligned lengths, square and rectangular periods, shifts that
    leave rows empty or full."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        cols = int(rng.integers(1, 20000)) if rng.random() < 0.6 else int(rng.integers(1, 1100))
        rows = int(rng.integers(1, max(2, min(400, 1_500_000 // cols)) + 1))
        dt = str(rng.choice(["f32", "bf16", "f16"]))
        kind = int(rng.integers(0, 3))
        period = cols if kind == 0 else int(rng.integers(1, 2 * cols + 2))
        shift = 0 if kind == 0 else int(rng.integers(-cols, cols + 1))
        out.append((rows, cols, dt, int(rng.integers(0, 4)), period, shift, int(rng.integers(0, 1 << 20))))
    return out


@pytest.mark.parametrize("rows,cols,dt,mode,period,shift,seed", _causal_cases(24, 2025))
def test_random_causal(q, rows, cols, dt, mode, period, shift, seed):
    say("random causal", dt, rows, cols, mode, period, shift, seed)
    x = synth.normal((rows, cols), 2.0, dt, seed)
    g, r, d = ts._run_causal(q, x, mode, 0.6, period, shift)
    assert_parity(g, r, d, "op", "random causal %s %dx%d m%d p%d s%d seed%d" % (
        dt, rows, cols, mode, period, shift, seed))


def _elementwise_cases(n, seed):
    """(op, n, dt, mode, a, b, seed): lengths from one element to past the
    resident-grid limit of 16-bit vectors (2^25 elements), ragged tails, and
    random affine maps for e^(a x + b)."""
    rng = np.random.default_rng(seed)
    anchors = [1, 7, 8, 9, 4095, 4096, 4104, 1 << 20, (1 << 25) - 8, (1 << 25) + 8]
    out = []
    while len(out) < n:
        ne = int(rng.choice(anchors)) if rng.random() < 0.4 else int(rng.integers(1, 3_000_000))
        op = str(rng.choice(["exp", "gelu", "sigmoid", "silu", "gelu_unfused"]))
        dt = str(rng.choice(["f32", "f16", "bf16"]))
        mode = int(rng.integers(0, 4))
        a = float(rng.choice([1.0, -1.0, 0.37, -2.5]))
        b = float(rng.choice([0.0, 1.5, -3.0]))
        if op != "exp":
            a, b = 1.0, 0.0
        out.append((op, ne, dt, mode, a, b, int(rng.integers(0, 1 << 20))))
    return out


ELEMENTWISE_CASES = _elementwise_cases(30, 2024)


@pytest.mark.parametrize("op,n,dt,mode,a,b,seed", ELEMENTWISE_CASES)
def test_random_elementwise(q, op, n, dt, mode, a, b, seed):
    say("random elementwise", op, n, dt, mode, a, b, seed)
    x = synth.uniform_with_outliers(n, -14.0, 14.0, 0.01, 80.0, dt, seed)
    g, r, d = run_elementwise(q, op, x, mode, a=a, b=b)
    assert_parity(g, r, d, kind_of(op, mode), "random %s %s n%d m%d a%g b%g seed%d" % (
        op, dt, n, mode, a, b, seed))


def _elementwise_offset_cases(n, seed):
    """(op, n, dt, xoff, yoff, seed): x and y views at random element offsets
    (the same or different offsets from 16 bytes), random lengths."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        op = str(rng.choice(["exp", "gelu", "sigmoid", "silu", "gelu_unfused"]))
        ne = int(rng.integers(1, 2_000_000)) if rng.random() < 0.7 else int(rng.integers(1, 64))
        out.append((op, ne, str(rng.choice(["f32", "bf16", "f16"])), int(rng.integers(0, 8)),
                    int(rng.integers(0, 8)), int(rng.integers(0, 1 << 20))))
    return out


@pytest.mark.parametrize("op,n,dt,xoff,yoff,seed", _elementwise_offset_cases(24, 77))
def test_random_elementwise_offsets(q, op, n, dt, xoff, yoff, seed):
    import oracle
    from gpu_util import THREADS, host_bits
    say("random elementwise offsets", op, n, dt, xoff, yoff, seed)
    x = synth.uniform_with_outliers(n + 8, -14.0, 14.0, 0.01, 80.0, dt, seed)
    xb = host_bits(x)[xoff:xoff + n].copy()
    xg = x.to("cuda:0")
    yfull = torch.full((n + 8,), 5.0, dtype=x.dtype, device="cuda:0")
    src, dst = xg[xoff:xoff + n], yfull[yoff:yoff + n]
    if op == "exp":
        q.quake_exp(src, dst, mode=2)
        ref = oracle.exp(xb, dt, 2, threads=THREADS)
    elif op == "gelu":
        q.quake_gelu(src, dst, mode=2)
        ref = oracle.gelu(xb, dt, 2, threads=THREADS)
    elif op == "gelu_unfused":
        q.quake_gelu_unfused(src, dst, mode=2)
        ref = oracle.gelu_unfused(xb, dt, 2, threads=THREADS)
    else:
        q.quake_sigmoid(src, dst, mode=2, silu=(op == "silu"))
        ref = oracle.sigmoid(xb, dt, 2, silu=(op == "silu"), threads=THREADS)
    torch.cuda.synchronize()
    out = host_bits(yfull)
    assert_parity(out[yoff:yoff + n].copy(), ref, dt, kind_of(op, 2),
                  "random offsets %s %s n%d x+%d y+%d seed%d" % (op, dt, n, xoff, yoff, seed))
    pad = np.concatenate([out[:yoff], out[yoff + n:]])
    assert np.all(oracle.decode(pad, dt) == 5.0), "write outside y"


def _linear_cases(n, seed):
    """(m, n, k, mode, dt, gelu, pad, seed): output widths around multiples
    of 128 and 192 (grids this small take the 128-wide tile), ragged m and n,
    k a multiple of 8 from one slab to several with a tail, operand rows
    padded to a longer stride."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        m = int(rng.choice([1, 127, 128, 129, 256])) if rng.random() < 0.4 else int(rng.integers(1, 520))
        nn = int(rng.choice([1, 191, 192, 193, 384, 576, 128, 129])) if rng.random() < 0.5 else \
            int(rng.integers(1, 700))
        k = 8 * int(rng.integers(1, 65))
        out.append((m, nn, k, int(rng.integers(0, 4)), str(rng.choice(["bf16", "f16"])),
                    bool(rng.random() < 0.75), int(rng.choice([0, 0, 8, 24])),
                    int(rng.integers(0, 1 << 20))))
    return out


LINEAR_CASES = _linear_cases(30, 768)


@pytest.mark.parametrize("m,n,k,mode,dt,gelu,pad,seed", LINEAR_CASES)
def test_random_linear_gelu(q, m, n, k, mode, dt, gelu, pad, seed):
    say("random linear", dt, m, n, k, mode, gelu, pad, seed)
    g, r, xb, wb = tl._run(q, m, n, k, mode, gelu, seed, pad=pad, dt=dt)
    tl._check(g, r, xb, wb, k, 2.0 if gelu else 1.0, "random linear %s %dx%dx%d m%d gelu%d pad%d seed%d"
              % (dt, m, n, k, mode, gelu, pad, seed), dt)
