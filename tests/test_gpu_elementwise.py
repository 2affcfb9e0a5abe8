"""GPU parity of quake_exp, quake_gelu and quake_sigmoid against the oracle,
through the C ABI, on cuda:0."""
import numpy as np
import pytest
import torch

import oracle
from compare import check_bits, check_f32_ulp
from gpu_util import THREADS, assert_parity, host_bits, kind_of, run_elementwise, say
from paper_2412_00408_amd import synth

pytestmark = pytest.mark.gpu

MODES = [0, 1, 2, 3]
DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


@pytest.fixture(scope="module")
def q():
    assert torch.cuda.is_available(), "GPU tests need cuda:0"
    from paper_2412_00408_amd import quake
    return quake


@pytest.mark.parametrize("mode", [1, 2, 3])
def test_exp_f32_bit_exact_every_input(q, mode):
    """QuAKE / QuAKE2 exp of every binary32 bit pattern (NaN inputs excluded)."""
    chunk = 1 << 26
    bad = 0
    first = None
    for lo in range(0, 1 << 32, chunk):
        if lo % (1 << 30) == 0:
            say("exp f32 mode", mode, "patterns from", hex(lo))
        u = torch.arange(lo, lo + chunk, dtype=torch.int64, device="cuda:0")
        u = torch.where(u >= (1 << 31), u - (1 << 32), u).to(torch.int32)
        xg = u.view(torch.float32)
        yg = q.quake_exp(xg, mode=mode)
        xb = xg.cpu().numpy()
        yb = yg.cpu().numpy()
        ref = oracle.exp(xb, "f32", mode, threads=THREADS)
        nan_in = np.isnan(xb)
        mism = (yb.view(np.uint32) != ref.view(np.uint32)) & ~nan_in
        n = int(mism.sum())
        if n and first is None:
            i = int(np.flatnonzero(mism)[0])
            first = (hex(int(xb.view(np.uint32)[i])), float(yb[i]), float(ref[i]))
        bad += n
    assert bad == 0, "%d mismatches, first %s" % (bad, first)


def test_exp_f32_exact_mode_sampled(q):
    """EXACT exp (hardware v_exp_f32) on every 61st binary32 pattern: <= 2 ulp."""
    u = torch.arange(0, 1 << 32, 61, dtype=torch.int64, device="cuda:0")
    u = torch.where(u >= (1 << 31), u - (1 << 32), u).to(torch.int32)
    xg = u.view(torch.float32)
    yg = q.quake_exp(xg, mode=0)
    xb = xg.cpu().numpy()
    ref = oracle.exp(xb, "f32", 0, threads=THREADS)
    keep = ~np.isnan(xb)
    msg = check_f32_ulp(yg.cpu().numpy()[keep], ref[keep], 2, "exp exact")
    assert msg is None, msg


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("ab", [(1.0, 0.0), (-1.0, 0.0), (0.37, 2.0), (-3.0, -1.5), (10.0, 5.0)])
def test_exp_affine(q, dt, mode, ab):
    x = synth.normal((300_001,), 6.0, dt, 100)
    say("exp", dt, mode, ab)
    g, r, d = run_elementwise(q, "exp", x, mode, a=ab[0], b=ab[1])
    assert_parity(g, r, d, kind_of("exp", mode), "exp %s %s %s" % (dt, mode, ab))


@pytest.mark.parametrize("op", ["gelu", "sigmoid", "silu", "gelu_unfused"])
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("mode", MODES)
def test_operators_random(q, op, dt, mode):
    x = synth.uniform_with_outliers(1_000_003, -14.0, 14.0, 0.01, 80.0, dt, 101)
    say(op, dt, mode)
    g, r, d = run_elementwise(q, op, x, mode)
    assert_parity(g, r, d, "op", "%s %s %s" % (op, dt, mode))


@pytest.mark.parametrize("op", ["exp", "gelu", "sigmoid", "silu", "gelu_unfused"])
@pytest.mark.parametrize("mode", MODES)
def test_special_values(q, op, mode):
    vals = [0.0, -0.0, 1e-40, -1e-40, 1e-30, 5.0, -5.0, 10.0, -9.99, -10.2, -10.5, 20.0, -20.0,
            80.0, -80.0, 87.0, -87.0, 88.7, 89.0, -104.0, 1e4, -1e4, 3e38, -3e38]
    if not op.startswith("gelu"):
        vals += [np.inf, -np.inf]
    x = torch.tensor(vals, dtype=torch.float32)
    say("special", op, mode)
    g, r, d = run_elementwise(q, op, x, mode)
    assert_parity(g, r, d, kind_of(op, mode), "special %s %s" % (op, mode))


@pytest.mark.parametrize("n", [1, 3, 7, 8, 9, 15, 17, 255, 4096 + 5, 4096 * 3 + 1, 1_000_003])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_ragged_lengths(q, n, dt):
    x = synth.normal((n,), 3.0, dt, 102)
    for op in ("exp", "gelu", "sigmoid", "silu", "gelu_unfused"):
        say("ragged", op, dt, n)
        g, r, d = run_elementwise(q, op, x, 2)
        assert_parity(g, r, d, kind_of(op, 2), "ragged %s %s %d" % (op, dt, n))


# x and y at the same offset from a 16-byte boundary: the elements before the
# first boundary take the scalar kernel, the rest the vector kernels; lengths
# shorter than, equal to and just past that head. x and y at different
# offsets: each aligned vector of y assembled from two aligned vectors of x
# (every byte shift), scalar head and tail. Padding around y must stay
# untouched.
OFFSETS = [(1, 1), (2, 2), (3, 3), (5, 5), (7, 7), (1, 0), (0, 3), (2, 5), (3, 1), (7, 2), (5, 0),
           (0, 1), (6, 7), (4, 0)]


# (a nonzero offset of a whole 16-byte vector, 4 binary32 elements, is left out)
@pytest.mark.parametrize("dt,xoff,yoff", [(dt, a, b) for dt in ("f32", "f16", "bf16") for a, b in OFFSETS
                                          if dt != "f32" or not any(o and o % 4 == 0 for o in (a, b))])
def test_offsets(q, dt, xoff, yoff):
    V = 4 if dt == "f32" else 8
    esz = 4 if dt == "f32" else 2
    head = ((16 - (yoff * esz) % 16) % 16) // esz
    for n in sorted({1, max(1, head - 1), max(1, head), head + 1, head + V + 1, 2 * V - 1, 2 * V,
                     2 * V + 1, 5000, 1_000_003}):
        x = synth.normal((n + 8,), 3.0, dt, 110 + n % 31 + xoff)
        xb = host_bits(x)[xoff:xoff + n].copy()
        xg = x.to("cuda:0")
        yfull = torch.full((n + 8,), 5.0, dtype=x.dtype, device="cuda:0")
        src, dst = xg[xoff:xoff + n], yfull[yoff:yoff + n]
        for op in ("exp", "gelu", "sigmoid", "silu"):
            say("offsets", op, dt, n, xoff, yoff)
            if op == "exp":
                q.quake_exp(src, dst, mode=2)
                ref = oracle.exp(xb, dt, 2, threads=THREADS)
            elif op == "gelu":
                q.quake_gelu(src, dst, mode=2)
                ref = oracle.gelu(xb, dt, 2, threads=THREADS)
            else:
                q.quake_sigmoid(src, dst, mode=2, silu=(op == "silu"))
                ref = oracle.sigmoid(xb, dt, 2, silu=(op == "silu"), threads=THREADS)
            torch.cuda.synchronize()
            out = host_bits(yfull)
            assert_parity(out[yoff:yoff + n].copy(), ref, dt, kind_of(op, 2),
                          "offsets %s %s n %d x+%d y+%d" % (op, dt, n, xoff, yoff))
            pad = np.concatenate([out[:yoff], out[yoff + n:]])
            assert np.all(oracle.decode(pad, dt) == 5.0), "write outside y"


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_misaligned_and_inplace(q, dt):
    x = synth.normal((100_003,), 3.0, dt, 103)
    xb = host_bits(x)
    for op in ("exp", "gelu", "sigmoid", "silu"):
        say("misaligned/inplace", op, dt)
        xg = x.to("cuda:0")
        # input and output both shifted by one element: not 16-byte aligned
        src = xg[1:]
        dst = torch.empty(100_004, dtype=x.dtype, device="cuda:0")[1:-1]
        if op == "exp":
            y = q.quake_exp(src, dst, mode=2)
            ref = oracle.exp(xb[1:].copy(), dt, 2, threads=THREADS)
        elif op == "gelu":
            y = q.quake_gelu(src, dst, mode=2)
            ref = oracle.gelu(xb[1:].copy(), dt, 2, threads=THREADS)
        else:
            y = q.quake_sigmoid(src, dst, mode=2, silu=(op == "silu"))
            ref = oracle.sigmoid(xb[1:].copy(), dt, 2, silu=(op == "silu"), threads=THREADS)
        assert_parity(host_bits(y), ref, dt, kind_of(op, 2), "misaligned %s %s" % (op, dt))
        # in place, aligned
        z = xg.clone()
        if op == "exp":
            q.quake_exp(z, z, mode=2)
            ref = oracle.exp(xb, dt, 2, threads=THREADS)
        elif op == "gelu":
            q.quake_gelu(z, z, mode=2)
            ref = oracle.gelu(xb, dt, 2, threads=THREADS)
        else:
            q.quake_sigmoid(z, z, mode=2, silu=(op == "silu"))
            ref = oracle.sigmoid(xb, dt, 2, silu=(op == "silu"), threads=THREADS)
        assert_parity(host_bits(z), ref, dt, kind_of(op, 2), "inplace %s %s" % (op, dt))


def test_empty_is_a_no_op(q):
    x = torch.empty(0, device="cuda:0")
    y = q.quake_gelu(x)
    assert y.numel() == 0
    z = torch.full((4,), 7.0, device="cuda:0")
    q.lib.quake_exp(z.data_ptr(), z.data_ptr(), 0, 0, 2, 1.0, 0.0, None)
    torch.cuda.synchronize()
    assert z.cpu().tolist() == [7.0] * 4


def test_more_than_2_pow_31_elements(q):
    """fp16 sigmoid over 2^31 + 77 elements (split into several launches);
    sampled outputs around every launch boundary are checked one by one."""
    n = (1 << 31) + 77
    say("2^31+77 fp16 sigmoid")
    g = torch.Generator(device="cuda:0")
    g.manual_seed(synth.SEED_BASE + 104)
    x = (torch.rand(n, generator=g, device="cuda:0", dtype=torch.float16) - 0.5) * 24
    y = q.quake_sigmoid(x, mode=2)
    torch.cuda.synchronize()
    pos = set()
    for b in (0, 1 << 30, 1 << 31):
        pos.update(range(max(0, b - 40), min(n, b + 40)))
    pos.update(range(n - 100, n))
    pos.update(np.random.default_rng(5).integers(0, n, 20000).tolist())
    idx = torch.tensor(sorted(pos), dtype=torch.int64, device="cuda:0")
    xs = host_bits(x[idx])
    ys = host_bits(y[idx])
    del x, y
    ref = oracle.sigmoid(xs, "f16", 2)
    assert_parity(ys, ref, "f16", "op", "2^31+77")


@pytest.mark.parametrize("mode", MODES)
def test_workload_gelu_bf16_4096x3072(q, mode):
    w = synth.WORKLOADS["gelu_bf16_4096x3072"]
    say(w.name, mode)
    g, r, d = run_elementwise(q, "gelu", w.make(), mode)
    assert_parity(g, r, d, "op", "%s mode %d" % (w.name, mode))


@pytest.mark.parametrize("op", ["sigmoid", "silu"])
@pytest.mark.parametrize("mode", MODES)
def test_workload_logistic_f16_2p28(q, op, mode):
    w = synth.WORKLOADS["sigmoid_f16_2p28"]
    say(w.name, op, mode)
    g, r, d = run_elementwise(q, op, w.make(), mode)
    assert_parity(g, r, d, "op", "%s %s mode %d" % (w.name, op, mode))


def test_streams(q):
    x = synth.normal((200_000,), 2.0, "bf16", 105).to("cuda:0")
    ref = q.quake_gelu(x, mode=2)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        y = q.quake_gelu(x, mode=2)
    s.synchronize()
    torch.cuda.synchronize()
    assert check_bits(host_bits(y), host_bits(ref)) is None


@pytest.mark.parametrize("op", ["gelu", "gelu_unfused"])
@pytest.mark.parametrize("mode", MODES)
def test_workload_table4_gelu_f32_260k(q, op, mode):
    w = synth.TABLE4_WORKLOADS["gelu_f32_260k"]
    say(w.name, op, mode)
    g, r, d = run_elementwise(q, op, w.make(), mode)
    assert_parity(g, r, d, "op", "%s %s mode %d" % (w.name, op, mode))
