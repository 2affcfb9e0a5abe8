"""GPU parity of quake_exp16 (QuAKE built in the binary16 / bfloat16 layout)
against the oracle, through the C ABI, on cuda:0: every 16-bit input pattern,
several affine maps, long and ragged arrays, misaligned buffers, in place."""
import numpy as np
import pytest
import torch

import oracle
from compare import check_bits
from gpu_util import THREADS, host_bits, say
from paper_2412_00408_amd import synth

pytestmark = pytest.mark.gpu

TD = {"f16": torch.float16, "bf16": torch.bfloat16}
AB = [(1.0, 0.0), (-1.0, 0.0), (0.6931471805599453, 0.0), (2.5, -1.25), (-0.37, 3.0), (40.0, 7.0)]


@pytest.fixture(scope="module")
def q():
    assert torch.cuda.is_available(), "GPU tests need cuda:0"
    from paper_2412_00408_amd import quake
    return quake


def _all_patterns(dt):
    u = torch.arange(0, 1 << 16, dtype=torch.int32).to(torch.int16)
    return u.view(TD[dt])


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("mode", [1, 2])
def test_every_pattern_bit_exact(q, dt, mode):
    x = _all_patterns(dt)
    xb = host_bits(x)
    xg = x.to("cuda:0")
    for a, b in AB:
        say("exp16 all patterns", dt, mode, a, b)
        y = q.quake_exp16(xg, mode=mode, a=a, b=b)
        torch.cuda.synchronize()
        ref = oracle.exp16(xb, dt, mode, a=a, b=b, threads=THREADS)
        g = host_bits(y)
        nan_in = np.isnan(oracle.decode(xb, dt))
        msg = check_bits(g, ref, "exp16 %s mode %d a %g b %g" % (dt, mode, a, b), ignore=nan_in)
        assert msg is None, msg


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("n,off", [(1, 0), (7, 0), (8, 0), (1000, 0), (1000, 1), (3 << 20, 0),
                                   ((1 << 22) + 13, 0), ((1 << 20) + 5, 3), (1, 5), (2, 7),
                                   (3, 5), (4, 5), (9, 1), (100_001, 6), (1 << 22, 2)])
def test_lengths_and_alignment(q, dt, n, off):
    x = synth.uniform((n + off,), -12.0, 12.0, dt, 1300 + n % 97)
    xb = host_bits(x)[off:]
    xg = x.to("cuda:0")[off:]
    y = torch.full((n + off,), 3.0, dtype=TD[dt], device="cuda:0")
    say("exp16 length", dt, n, off)
    q.quake_exp16(xg, y[off:], mode=2)
    torch.cuda.synchronize()
    out = host_bits(y)
    ref = oracle.exp16(xb, dt, 2, threads=THREADS)
    assert check_bits(out[off:], ref, "exp16 %s n %d off %d" % (dt, n, off)) is None
    if off:
        assert np.all(oracle.decode(out[:off], dt) == 3.0)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("n,xoff,yoff", [(15, 1, 0), (16, 1, 0), (17, 0, 3), (1000, 3, 6),
                                         (100_003, 7, 2), ((1 << 20) + 5, 5, 1), (33, 6, 6)])
def test_offsets_differ(q, dt, n, xoff, yoff):
    # x and y at different offsets from 16 bytes: each aligned vector of y
    # assembled from two aligned vectors of x; padding around y untouched
    x = synth.uniform((n + 8,), -12.0, 12.0, dt, 1350 + n % 83)
    xb = host_bits(x)[xoff:xoff + n].copy()
    xg = x.to("cuda:0")
    y = torch.full((n + 8,), 3.0, dtype=TD[dt], device="cuda:0")
    say("exp16 offsets", dt, n, xoff, yoff)
    q.quake_exp16(xg[xoff:xoff + n], y[yoff:yoff + n], mode=2)
    torch.cuda.synchronize()
    out = host_bits(y)
    ref = oracle.exp16(xb, dt, 2, threads=THREADS)
    assert check_bits(out[yoff:yoff + n].copy(), ref, "exp16 %s n %d x+%d y+%d" % (dt, n, xoff, yoff)) is None
    assert np.all(oracle.decode(np.concatenate([out[:yoff], out[yoff + n:]]), dt) == 3.0)


def test_in_place_and_stream(q):
    x = synth.uniform((1 << 20,), -9.0, 9.0, "f16", 1400).to("cuda:0")
    ref = q.quake_exp16(x, mode=1)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    z = x.clone()
    with torch.cuda.stream(s):
        q.quake_exp16(z, z, mode=1)
    s.synchronize()
    assert check_bits(host_bits(z), host_bits(ref)) is None


def test_close_to_the_binary32_path(q):
    # both approximate e^x; the 16-bit construction carries l_m mantissa bits
    x = synth.uniform((1 << 16,), -8.0, 8.0, "f16", 1500).to("cuda:0")
    a = q.quake_exp16(x, mode=2).float()
    b = q.quake_exp(x, mode=2).float()
    rel = ((a - b).abs() / b).max().item()
    assert rel < 0.004
