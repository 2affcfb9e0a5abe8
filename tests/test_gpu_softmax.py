"""GPU parity of quake_softmax (Algorithm 2) against the oracle, through the C
ABI, on cuda:0: every kernel family (wave per row, workgroup per row, split
rows, generic), ragged lengths, strides, masking, temperatures, modes and the
three workload shapes."""
import numpy as np
import pytest
import torch

import oracle
from compare import check_bits
from gpu_util import THREADS, assert_parity, host_bits, say
from paper_2412_00408_amd import synth

pytestmark = pytest.mark.gpu

MODES = [0, 1, 2, 3]


@pytest.fixture(scope="module")
def q():
    assert torch.cuda.is_available(), "GPU tests need cuda:0"
    from paper_2412_00408_amd import quake
    return quake


def _run(q, x_cpu, mode, t, ld_pad=0, offset=0, fused=True, ws=False):
    """Softmax of a [rows, cols] CPU tensor on the GPU and in the oracle.

    ld_pad > 0 stores rows with stride cols + ld_pad (input and output);
    offset > 0 shifts both base pointers by that many elements; ws passes a
    fresh zero-filled workspace (quake_softmax_ws), whose slots must be zero
    again afterwards."""
    dt = {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[x_cpu.dtype]
    rows, cols = x_cpu.shape
    ld = cols + ld_pad
    xb = host_bits(x_cpu)
    wsb = q.softmax_workspace(rows, cols, x_cpu.dtype) if ws else None
    kw = {"workspace": wsb} if wsb is not None else {}
    if ld_pad or offset:
        big = torch.zeros(rows * ld + offset + 8, dtype=x_cpu.dtype)
        view = big[offset:offset + rows * ld].view(rows, ld)[:, :cols]
        view.copy_(x_cpu)
        gx = big.to("cuda:0")
        xg = gx[offset:offset + rows * ld].view(rows, ld)[:, :cols]
        gy = torch.full_like(gx, 7.0)
        yg = gy[offset:offset + rows * ld].view(rows, ld)[:, :cols]
        (q.quake_softmax if fused else q.quake_softmax_unfused)(xg, yg, mode=mode, t=t, **kw)
        torch.cuda.synchronize()
        out = gy.cpu()
        # padding around the rows must be untouched
        pad = torch.ones_like(out, dtype=torch.bool)
        pad[offset:offset + rows * ld].view(rows, ld)[:, :cols] = False
        assert torch.all(out[pad] == 7.0)
        g = host_bits(out[offset:offset + rows * ld].view(rows, ld)[:, :cols].contiguous())
    else:
        xg = x_cpu.to("cuda:0")
        yg = (q.quake_softmax if fused else q.quake_softmax_unfused)(xg, mode=mode, t=t, **kw)
        torch.cuda.synchronize()
        g = host_bits(yg)
    if wsb is not None:
        assert int(wsb[256:].count_nonzero()) == 0, "workspace slots not returned to zero"
        assert int(wsb[4:8].view(torch.int32)[0]) == 0, "an exchange wait gave up on an idle GPU"
    fn = oracle.softmax if fused else oracle.softmax_unfused
    ref = fn(xb.reshape(rows, cols), dt, mode, t=t, threads=THREADS)
    return g, ref, dt


def _paths(cols):
    """Rows longer than one workgroup's registers run twice: without a
    workspace (one workgroup per row) and split over exchanging workgroups."""
    return (False, True) if cols > 16384 else (False,)


COLS_F32 = [1, 2, 3, 4, 100, 128, 252, 256, 260, 512, 1000, 1024, 2048, 4096, 8188, 8192, 8196,
            10000, 16384, 16388, 65536, 128256, 200000]
COLS_16 = [1, 8, 24, 512, 1000, 1024, 2048, 4096, 8192, 16384, 16392, 32768, 128256]


@pytest.mark.parametrize("cols", COLS_F32)
@pytest.mark.parametrize("mode", MODES)
def test_lengths_f32(q, cols, mode):
    rows = 5 if cols >= 65536 else 37
    x = synth.normal((rows, cols), 3.0, "f32", 200 + cols % 97)
    for ws in _paths(cols):
        say("softmax f32", rows, cols, mode, "workspace" if ws else "")
        g, r, dt = _run(q, x, mode, 1.0, ws=ws)
        assert_parity(g, r, dt, "op", "softmax f32 %dx%d mode %d ws %d" % (rows, cols, mode, ws))


@pytest.mark.parametrize("cols", COLS_16)
@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("mode", MODES)
def test_lengths_16bit(q, cols, dt, mode):
    rows = 5 if cols >= 32768 else 29
    x = synth.normal((rows, cols), 2.0, dt, 300 + cols % 89)
    for ws in _paths(cols):
        say("softmax", dt, rows, cols, mode, "workspace" if ws else "")
        g, r, d = _run(q, x, mode, 0.7, ws=ws)
        assert_parity(g, r, d, "op", "softmax %s %dx%d mode %d ws %d" % (dt, rows, cols, mode, ws))


@pytest.mark.parametrize("cols", [128, 512, 3000, 8192, 50000])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_strides_and_misalignment(q, cols, dt):
    x = synth.normal((9, cols), 2.0, dt, 400)
    for pad, off in [(8, 0), (3, 0), (0, 1), (5, 3)]:
        for ws in _paths(cols):
            say("softmax strided", dt, cols, pad, off, "workspace" if ws else "")
            g, r, d = _run(q, x, 2, 1.0, ld_pad=pad, offset=off, ws=ws)
            assert_parity(g, r, d, "op", "softmax %s cols %d pad %d off %d ws %d"
                          % (dt, cols, pad, off, ws))


@pytest.mark.parametrize("cols", [64, 512, 1001, 4096, 20480, 50257, 65536, 128256])
@pytest.mark.parametrize("mode", MODES)
def test_masked_rows(q, cols, mode):
    r = np.random.default_rng(7)
    v = r.standard_normal((12, cols)).astype(np.float32) * 3
    v[r.random((12, cols)) < 0.7] = -np.inf
    v[3] = -np.inf                       # fully masked row -> zeros
    v[5, :] = -np.inf
    v[5, cols - 1] = 1.5                 # only the last entry is live -> one-hot
    for dt in ("f32", "bf16"):
        x = synth.to_format(v, dt)
        for ws in _paths(cols):
            say("softmax masked", dt, cols, mode, "workspace" if ws else "")
            g, ref, d = _run(q, x, mode, 1.0, ws=ws)
            assert_parity(g, ref, d, "op", "masked %s cols %d mode %d ws %d" % (dt, cols, mode, ws))
            gv = oracle.decode(g.reshape(-1), d).reshape(12, cols)
            assert np.all(gv[3] == 0.0)
            assert abs(float(gv[5, cols - 1]) - 1.0) <= 2.0 ** -23 and np.all(gv[5, :-1] == 0.0)


# Rows without a workspace too long for the register-row kernels: the
# row-resident kernel in each of its three shapes (registers at two workgroups
# per CU; registers at one; registers plus an LDS part), at both ends of each,
# then the first length past it (three-pass kernel).
RESIDENT_COLS = {"f32": [16388, 16900, 49152, 49156, 90112, 90116, 129024, 129028],
                 "bf16": [16392, 20000, 49152, 49160, 94208, 94216, 131072, 131080],
                 "f16": [16392, 49152, 49160, 94216, 131072, 131080]}


@pytest.mark.parametrize("dt,cols", [(d, c) for d, cs in RESIDENT_COLS.items() for c in cs])
@pytest.mark.parametrize("mode", MODES)
def test_resident_row_shapes(q, dt, cols, mode):
    x = synth.normal((3, cols), 3.0 if dt == "f32" else 2.0, dt, 1300 + cols % 101)
    say("softmax resident", dt, cols, mode)
    g, r, d = _run(q, x, mode, 0.8)
    assert_parity(g, r, d, "op", "resident %s cols %d mode %d" % (dt, cols, mode))
    if mode == 2:
        say("softmax resident strided", dt, cols)
        g, r, d = _run(q, x, mode, 0.8, ld_pad=8)
        assert_parity(g, r, d, "op", "resident strided %s cols %d" % (dt, cols))


def _shifted_cols(dt):
    """Ragged lengths at both ends of every class of the shifted-row path: a
    row of cols elements covers at most (cols + 2V - 2) // V aligned vectors,
    so a class of Nv vectors takes cols <= (Nv - 1) V + 1. The last length is
    one past the row-resident kernel's capacity: the generic kernel."""
    V = 4 if dt == "f32" else 8
    limits = [64, 128, 256, 512, 1024, 2048] + ([4096] if dt == "f32" else [])
    limits += [24 * 512, 44 * 512, 63 * 512] if dt == "f32" else [12 * 512, 23 * 512, 32 * 512]
    out = [1, 2, 3, V + 1]
    for n in limits:
        out += [(n - 1) * V + 1, (n - 1) * V + 2]
    return out


SHIFTED = [(dt, c) for dt in ("f32", "bf16", "f16") for c in _shifted_cols(dt)]


# Rows whose start is not 16-byte aligned: consecutive rows of a ragged length
# start at every offset in turn; the shifted-row kernels read the aligned
# vectors around each row (and the first length past them the generic kernel).
@pytest.mark.parametrize("dt,cols", SHIFTED)
@pytest.mark.parametrize("mode", MODES)
def test_shifted_rows(q, dt, cols, mode):
    rows = 9 if cols < 40000 else 5
    x = synth.normal((rows, cols), 3.0 if dt == "f32" else 2.0, dt, 1500 + cols % 113)
    for ws in _paths(cols):
        say("softmax shifted", dt, rows, cols, mode, "workspace" if ws else "")
        g, r, d = _run(q, x, mode, 0.9, ws=ws)
        assert_parity(g, r, d, "op", "shifted %s %dx%d mode %d ws %d" % (dt, rows, cols, mode, ws))


@pytest.mark.parametrize("cols", [7, 1001, 5000, 50257])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_shifted_offsets_and_strides(q, cols, dt):
    """Aligned lengths behind an offset base, ragged strides, and x and y at
    different offsets (the generic kernel)."""
    x = synth.normal((6, cols), 2.0, dt, 1600 + cols)
    for pad, off in [(0, 1), (0, 3), (1, 0), (5, 2), (3, 7)]:
        say("softmax shifted offsets", dt, cols, pad, off)
        g, r, d = _run(q, x, 2, 1.0, ld_pad=pad, offset=off)
        assert_parity(g, r, d, "op", "shifted %s cols %d pad %d off %d" % (dt, cols, pad, off))
    tdt = x.dtype
    big = torch.zeros(6 * cols + 1, dtype=tdt)
    big[1:].view(6, cols).copy_(x)
    xg = big.to("cuda:0")[1:].view(6, cols)            # x one element past 16 bytes
    yg = q.quake_softmax(xg, mode=2, t=1.0)            # y aligned: offsets differ
    torch.cuda.synchronize()
    g = host_bits(yg)
    r = oracle.softmax(host_bits(x).reshape(6, cols), dt, 2, t=1.0, threads=THREADS)
    assert_parity(g, r, dt, "op", "x and y at different offsets %s cols %d" % (dt, cols))


@pytest.mark.parametrize("t", [0.125, 0.5, 1.0, 3.0, 20.0])
@pytest.mark.parametrize("cols", [512, 128256])
def test_temperatures(q, t, cols):
    x = synth.normal((6, cols), 2.0, "f32", 500)
    for mode in MODES:
        for ws in _paths(cols):
            say("softmax t", t, cols, mode, "workspace" if ws else "")
            g, r, d = _run(q, x, mode, t, ws=ws)
            assert_parity(g, r, d, "op", "t %g cols %d mode %d ws %d" % (t, cols, mode, ws))


def test_many_rows_split_path_multiple_launches(q):
    # 1100 rows of 100000 fp32 with a workspace: two launches (1024 rows each
    # at most) of 7 chunks per row, each launch many times the workgroups the
    # device holds at once
    x = synth.normal((1100, 100000), 3.0, "f32", 600)
    say("softmax split 1100x100000")
    g, r, d = _run(q, x, 2, 1.0, ws=True)
    assert_parity(g, r, d, "op", "split 1100x100000")


def test_inplace_and_determinism(q):
    for cols in (512, 4096, 128256, 1001):
        x = synth.normal((7, cols), 3.0, "bf16", 700).to("cuda:0")
        for ws in _paths(cols):
            w = q.softmax_workspace(7, cols, x.dtype) if ws else None
            a = q.quake_softmax(x, mode=2, workspace=w)
            b = q.quake_softmax(x, mode=2, workspace=w)
            z = x.clone()
            q.quake_softmax(z, z, mode=2, workspace=w)
            torch.cuda.synchronize()
            say("softmax inplace/determinism", cols, "workspace" if ws else "")
            assert check_bits(host_bits(a), host_bits(b)) is None
            assert check_bits(host_bits(a), host_bits(z)) is None


def test_split_path_on_two_streams(q):
    # two split launches at once, one workspace per stream: together they ask
    # for more workgroups than the device holds, which only changes the speed
    x = synth.normal((64, 128256), 3.0, "f32", 800).to("cuda:0")
    w0 = q.softmax_workspace(64, 128256)
    ref = q.quake_softmax(x, mode=2, workspace=w0)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    ws = {s1: q.softmax_workspace(64, 128256), s2: q.softmax_workspace(64, 128256)}
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    outs = []
    for s in (s1, s2, s1, s2):
        with torch.cuda.stream(s):
            outs.append(q.quake_softmax(x, mode=2, workspace=ws[s]))
    torch.cuda.synchronize()
    for o in outs:
        assert check_bits(host_bits(o), host_bits(ref)) is None
    for w in ws.values():
        assert int(w[256:].count_nonzero()) == 0


# ---------------------------------------------------------------- workloads

@pytest.mark.parametrize("mode", MODES)
def test_workload_softmax_f32_64x128(q, mode):
    w = synth.WORKLOADS["softmax_f32_64x128"]
    say(w.name, mode)
    g, r, d = _run(q, w.make(), mode, w.t)
    assert_parity(g, r, d, "op", "%s mode %d" % (w.name, mode))
    s = oracle.decode(g, "f32").reshape(w.rows, w.cols).astype(np.float64).sum(axis=1)
    assert np.all(np.abs(s - 1) < 1e-5)


@pytest.mark.parametrize("mode", MODES)
def test_workload_attn_softmax_bf16_causal(q, mode):
    w = synth.WORKLOADS["attn_softmax_bf16_causal"]
    say(w.name, mode)
    x = w.make()
    g, r, d = _run(q, x, mode, w.t)
    assert_parity(g, r, d, "op", "%s mode %d" % (w.name, mode))
    # masked region is exactly zero
    gv = g.reshape(w.rows, w.cols)
    i = (np.arange(w.rows) % w.cols)[:, None]
    j = np.arange(w.cols)[None, :]
    assert np.all(gv[np.broadcast_to(j > i, gv.shape)] == 0)


@pytest.mark.parametrize("mode", MODES)
def test_workload_lmhead_softmax_f32_64x128256(q, mode):
    w = synth.WORKLOADS["lmhead_softmax_f32_64x128256"]
    x = w.make()
    for ws in (False, True):
        say(w.name, mode, "workspace" if ws else "")
        g, r, d = _run(q, x, mode, w.t, ws=ws)
        assert_parity(g, r, d, "op", "%s mode %d ws %d" % (w.name, mode, ws))


# ------------------------------------------- unfused form (Table IV study)

@pytest.mark.parametrize("cols,dt", [(128, "f32"), (512, "bf16"), (1001, "f32"), (4096, "f32"),
                                     (16384, "f32"), (16384, "bf16"), (128256, "f32"),
                                     (50000, "f16"), (30000, "bf16"), (70000, "f32")])
@pytest.mark.parametrize("mode", MODES)
def test_unfused(q, cols, dt, mode):
    rows = 6 if cols > 20000 else 33
    x = synth.normal((rows, cols), 2.5, dt, 900 + cols % 83)
    for t in (1.0, 0.125):
        say("softmax unfused", dt, rows, cols, mode, t)
        g, r, d = _run(q, x, mode, t, fused=False)
        assert_parity(g, r, d, "op", "unfused %s %dx%d mode %d t %g" % (dt, rows, cols, mode, t))


def test_unfused_masked_and_strided(q):
    r = np.random.default_rng(11)
    v = r.standard_normal((10, 3000)).astype(np.float32)
    v[r.random((10, 3000)) < 0.5] = -np.inf
    v[4] = -np.inf
    x = synth.to_format(v, "bf16")
    for mode in MODES:
        say("softmax unfused masked", mode)
        g, ref, d = _run(q, x, mode, 0.5, fused=False)
        assert_parity(g, ref, d, "op", "unfused masked mode %d" % mode)
        g, ref, d = _run(q, x, mode, 0.5, ld_pad=5, offset=1, fused=False)
        assert_parity(g, ref, d, "op", "unfused masked strided mode %d" % mode)


@pytest.mark.parametrize("fused,mode", [(True, 0), (True, 1), (True, 2), (False, 0), (False, 2)])
def test_workload_table4_softmax_f32_16384x16384(q, fused, mode):
    w = synth.TABLE4_WORKLOADS["softmax_f32_16384x16384"]
    say(w.name, "fused" if fused else "unfused", mode)
    g, r, d = _run(q, w.make(), mode, w.t, fused=fused)
    assert_parity(g, r, d, "op", "%s fused=%s mode %d" % (w.name, fused, mode))


# ------------------------------------------------------- implicit causal mask

def _run_causal(q, x_cpu, mode, t, period, shift):
    dt = {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[x_cpu.dtype]
    xg = x_cpu.to("cuda:0")
    yg = q.quake_softmax_causal(xg, period=period, shift=shift, mode=mode, t=t)
    torch.cuda.synchronize()
    ref = oracle.softmax_causal(host_bits(x_cpu), period, shift, dt, mode, t=t, threads=THREADS)
    return host_bits(yg), ref, dt


# ragged lengths (rows start at every offset from 16 bytes): the shifted
# register-row kernels up to 4096 (binary32) / 2048 (16-bit) covered vectors,
# then the scalar kernel (16383 f32, 16378 bf16)
@pytest.mark.parametrize("cols,dt", [(64, "f32"), (512, "bf16"), (1000, "bf16"), (4096, "f32"),
                                     (16384, "f32"), (40000, "f32"), (32768, "bf16"),
                                     (1, "f32"), (3, "bf16"), (63, "f32"), (1001, "bf16"),
                                     (4095, "f32"), (2047, "f16"), (16381, "f32"), (16383, "f32"),
                                     (16377, "bf16"), (16378, "bf16")])
@pytest.mark.parametrize("mode", MODES)
def test_causal(q, cols, dt, mode):
    rows = min(2 * cols, 96) if cols <= 4096 else 9
    x = synth.normal((rows, cols), 2.0, dt, 1000 + cols % 71)
    for period, shift in [(cols, 0), (rows, cols - rows), (7, 3), (5, -2)]:
        say("softmax causal", dt, rows, cols, mode, period, shift)
        g, r, d = _run_causal(q, x, mode, 0.6, period, shift)
        assert_parity(g, r, d, "op", "causal %s %dx%d mode %d p %d s %d" % (dt, rows, cols, mode,
                                                                            period, shift))


@pytest.mark.parametrize("mode", MODES)
def test_workload_attn_implicit_causal(q, mode):
    """The attention workload with the mask implied instead of read: equal to
    the oracle, and bit-identical to the explicit -inf input on the GPU; poison
    in the masked half changes nothing."""
    w = synth.WORKLOADS["attn_softmax_bf16_causal"]
    x = w.make()
    say(w.name, "implicit", mode)
    g, r, d = _run_causal(q, x, mode, w.t, w.cols, 0)
    assert_parity(g, r, d, "op", "implicit causal mode %d" % mode)
    xg = x.to("cuda:0")
    explicit = q.quake_softmax(xg, mode=mode, t=w.t)
    poisoned = xg.clone()
    i = (torch.arange(w.rows, device="cuda:0") % w.cols)[:, None]
    j = torch.arange(w.cols, device="cuda:0")[None, :]
    poisoned[j > i] = float("nan")
    implicit = q.quake_softmax_causal(poisoned, period=w.cols, shift=0, mode=mode, t=w.t)
    torch.cuda.synchronize()
    assert check_bits(host_bits(implicit), host_bits(explicit)) is None


@pytest.mark.parametrize("cols,dt", [(512, "bf16"), (4096, "f32"), (40000, "f32"), (1000, "bf16"),
                                     (1001, "bf16"), (333, "f32"), (20001, "f32")])
def test_causal_without_masked_writes(q, cols, dt):
    rows = 64 if cols <= 4096 else 6
    x = synth.normal((rows, cols), 2.0, dt, 1100 + cols % 61)
    ref = oracle.softmax_causal(host_bits(x), cols, 0, dt, 2, t=1.0, threads=THREADS)
    xg = x.to("cuda:0")
    y = torch.full_like(xg, 7.0)
    say("softmax causal no masked writes", dt, rows, cols)
    q.quake_softmax_causal(xg, y, period=cols, shift=0, mode=2, write_masked=False)
    torch.cuda.synchronize()
    g = host_bits(y)
    vec = 4 if dt == "f32" else 8
    i = np.arange(rows)[:, None] % cols
    j = np.arange(cols)[None, :]
    live = j <= i
    # vector kernels write whole 16-byte vectors that hold a live entry: row r
    # starts s = r * cols mod vec elements past a 16-byte boundary (the
    # shifted-row kernels up to 4096 / 2048 vectors); the scalar kernel
    # writes the live entries only
    s = (np.arange(rows)[:, None] * cols) % vec
    vector_path = cols % vec == 0 or (cols + 2 * vec - 2) // vec <= (4096 if dt == "f32" else 2048)
    written = ((s + j) // vec) <= ((s + i) // vec) if vector_path else live
    # live outputs match the oracle; untouched outputs keep their old value
    assert_parity(g[live], ref[live], dt, "op", "causal no-writes %s %d" % (dt, cols))
    gv = oracle.decode(g.reshape(-1), dt).reshape(rows, cols)
    assert np.all(gv[~written] == 7.0)
    assert np.all(gv[written & ~live] == 0.0)


# Square causal blocks (period = cols, shift = 0, at most 64 vectors per row)
# take the paired-row kernel: two rows per wave, r and M - 1 - r. Shapes cover
# K = 0 and K > 0 (P above 63 vectors), odd M, one-vector rows, a trailing
# partial block (handled by the one-row kernel) and padded row strides.
@pytest.mark.parametrize("P,dt,rows,pad", [(512, "bf16", 2 * 512 + 37, 0), (504, "bf16", 504, 8),
                                           (256, "f32", 2 * 256 + 3, 0), (252, "f32", 252, 4),
                                           (200, "f16", 401, 0), (8, "bf16", 40, 0),
                                           (4, "f32", 13, 4), (72, "bf16", 3 * 72, 0)])
@pytest.mark.parametrize("mode", MODES)
def test_causal_paired_rows(q, P, dt, rows, pad, mode):
    ld = P + pad
    x = synth.normal((rows, ld), 2.0, dt, 1200 + P)
    xg = x.to("cuda:0")[:, :P]
    say("softmax causal paired", dt, rows, P, pad, mode)
    for wm in (True, False):
        y = torch.full((rows, ld), 5.0, dtype=xg.dtype, device="cuda:0")[:, :P]
        q.quake_softmax_causal(xg, y, period=P, shift=0, mode=mode, t=0.7, write_masked=wm)
        torch.cuda.synchronize()
        g = host_bits(y)
        ref = oracle.softmax_causal(host_bits(x[:, :P]), P, 0, dt, mode, t=0.7, threads=THREADS)
        i = np.arange(rows)[:, None] % P
        j = np.arange(P)[None, :]
        live = j <= i
        vec = 4 if dt == "f32" else 8
        written = live | ((j // vec) <= (i // vec)) if not wm else np.ones_like(live)
        assert_parity(g[written], ref[written], dt, "op", "paired %s P %d wm %d" % (dt, P, wm))
        if not wm:
            gv = oracle.decode(g.reshape(-1), dt).reshape(rows, P)
            assert np.all(gv[~written] == 5.0)
        # bit-identical to the one-row kernel reading explicit -inf entries
        xm = xg.clone()
        xm[torch.from_numpy(~live).to("cuda:0")] = float("-inf")
        e = q.quake_softmax(xm, mode=mode, t=0.7)
        torch.cuda.synchronize()
        eb = host_bits(e)
        assert check_bits(g[written], eb[written]) is None
