"""GPU parity of quake_linear_gelu (matrix-core product with the GELU of Eq. 7
in its epilogue) against the oracle's float64 product rounded to binary32
followed by the oracle's GELU.

Tolerance per element (derived, written here): the GPU sums in binary32 in
its own order, so its accumulator differs from the binary32-rounded exact sum
by at most k * 2^-24 * sum_i |x_i w_i| (plus that rounding); GELU with any of
the exponentials here changes by at most 2x a change of its argument (slope of
x * sigma(.) at most 1.13, QuAKE's piecewise slope at most 1.44 times e^x's),
and each side rounds once to the 16-bit format: |gpu - ref| <= ulp(ref) +
2 * (k + 1) * 2^-24 * sum|x||w| + floor, with ulp and floor of that format
(bfloat16: 8 significant bits, floor 2^-126; binary16: 11 bits, outputs below
2^-14 spaced 2^-24 apart)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import THREADS, host_bits, say
from paper_2412_00408_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def q():
    assert torch.cuda.is_available(), "GPU tests need cuda:0"
    from paper_2412_00408_amd import quake
    return quake


def _ulp(v, dt):
    a = np.abs(v)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    if dt == "bf16":
        return np.where(a >= 2.0 ** -126, np.ldexp(1.0, (e - 7).astype(int)), 2.0 ** -133)
    return np.where(a >= 2.0 ** -14, np.ldexp(1.0, (e - 10).astype(int)), 2.0 ** -24)


def _check(g_bits, r_bits, xb, wb, k, lip, name, dt="bf16"):
    g = oracle.decode(g_bits.reshape(-1), dt).astype(np.float64)
    r = oracle.decode(r_bits.reshape(-1), dt).astype(np.float64)
    xa = np.abs(oracle.decode(xb.reshape(-1), dt).astype(np.float64)).reshape(xb.shape)
    wa = np.abs(oracle.decode(wb.reshape(-1), dt).astype(np.float64)).reshape(wb.shape)
    s = (xa @ wa.T).reshape(-1)
    floor = 2.0 ** -126 if dt == "bf16" else 2.0 ** -25
    bound = _ulp(r, dt) + lip * (k + 1) * 2.0 ** -24 * s + floor
    err = np.abs(g - r)
    bad = ~(err <= bound)
    assert not bad.any(), "%s: %d of %d outside the bound, worst at %d: gpu %r ref %r bound %r" % (
        name, int(bad.sum()), bad.size, int(np.argmax(err - bound)), g[np.argmax(err - bound)],
        r[np.argmax(err - bound)], bound[np.argmax(err - bound)])
    return err


def _run(q, m, n, k, mode, gelu, seed, pad=0, dt="bf16"):
    x = synth.normal((m, k + pad), 1.0, dt, seed)
    w = synth.normal((n, k + pad), 0.05, dt, seed + 1)
    xg, wg = x.to("cuda:0"), w.to("cuda:0")
    y = q.quake_linear_gelu(xg[:, :k], wg[:, :k], mode=mode, gelu=gelu)
    torch.cuda.synchronize()
    xb, wb = host_bits(x)[:, :k].copy(), host_bits(w)[:, :k].copy()
    ref = oracle.linear_gelu(xb, wb, mode, gelu=gelu, dt=dt, threads=THREADS)
    return host_bits(y), ref, xb, wb


# grids below one 128 x 192 tile per CU (256 CUs) take the 128 x 128 tile,
# whatever n; the wide tile is tested below
@pytest.mark.parametrize("m,n,k", [(128, 128, 64), (256, 384, 768), (200, 130, 72), (1, 1, 8),
                                   (129, 257, 136), (64, 1000, 32), (200, 192, 72),
                                   (129, 576, 136), (1, 192, 8)])
@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_shapes_and_modes(q, m, n, k, mode, dt):
    for gelu in (True, False):
        say("linear gelu", dt, m, n, k, mode, gelu)
        g, r, xb, wb = _run(q, m, n, k, mode, gelu, 1600 + m % 7 + n % 5, dt=dt)
        _check(g, r, xb, wb, k, 2.0 if gelu else 1.0,
               "linear %s %dx%dx%d mode %d gelu %d" % (dt, m, n, k, mode, gelu), dt)


# a grid of at most one tile per CU over k >= 1024 loads every slab two slabs
# ahead into a second register set: odd and even slab counts, a k tail,
# ragged m and n, both tile widths
@pytest.mark.parametrize("m,n,k", [(128, 192, 1024), (200, 130, 1032), (1, 1, 2056),
                                   (129, 576, 1096), (300, 384, 4096)])
@pytest.mark.parametrize("mode", [0, 2])
@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_long_k_two_slabs_ahead(q, m, n, k, mode, dt):
    for gelu in (True, False):
        say("linear gelu long k", dt, m, n, k, mode, gelu)
        g, r, xb, wb = _run(q, m, n, k, mode, gelu, 1650 + m % 7 + n % 5, dt=dt)
        _check(g, r, xb, wb, k, 2.0 if gelu else 1.0,
               "linear long k %s %dx%dx%d mode %d gelu %d" % (dt, m, n, k, mode, gelu), dt)


# n a multiple of 192 with at least one 128 x 192 tile per CU takes the wide
# tile: a ragged last tile row and a k tail, and exactly 256 tiles over
# k >= 1024 (the wide tile with slabs two ahead)
@pytest.mark.parametrize("m,n,k,mode,dt", [(2043, 3072, 72, 2, "bf16"), (2043, 3072, 72, 0, "f16"),
                                           (2048, 3072, 1032, 2, "bf16"), (2048, 3072, 1032, 3, "f16")])
def test_wide_tile_grid(q, m, n, k, mode, dt):
    for gelu in (True, False):
        say("linear gelu wide tiles", dt, m, n, k, mode, gelu)
        g, r, xb, wb = _run(q, m, n, k, mode, gelu, 1670 + m % 7, dt=dt)
        _check(g, r, xb, wb, k, 2.0 if gelu else 1.0,
               "linear wide %s %dx%dx%d mode %d gelu %d" % (dt, m, n, k, mode, gelu), dt)


def test_strided_rows(q):
    say("linear gelu strided")
    g, r, xb, wb = _run(q, 256, 256, 768, 2, True, 1700, pad=24)
    _check(g, r, xb, wb, 768, 2.0, "strided")


# output views of a wider buffer: (column offset, row stride) with 8-byte
# aligned rows (vector stores) and without (element stores)
@pytest.mark.parametrize("off,ldy", [(0, 200), (4, 196), (1, 200), (2, 194)])
@pytest.mark.parametrize("n", [192, 130])
def test_output_views_keep_their_padding(q, off, ldy, n):
    m, k = 130, 72
    say("linear gelu into a view: n %d offset %d ldy %d" % (n, off, ldy))
    x = synth.normal((m, k), 1.0, "bf16", 1750)
    w = synth.normal((n, k), 0.05, "bf16", 1751)
    big = torch.full((m, ldy), 0x7FC1, dtype=torch.int16, device="cuda:0")   # a NaN pattern
    y = big.view(torch.bfloat16)[:, off:off + n]
    q.quake_linear_gelu(x.to("cuda:0"), w.to("cuda:0"), y=y, mode=2)
    torch.cuda.synchronize()
    got = big.cpu().numpy().view(np.uint16)
    keep = np.ones(ldy, bool)
    keep[off:off + n] = False
    assert (got[:, keep] == 0x7FC1).all(), "writes outside the view"
    xb, wb = host_bits(x), host_bits(w)
    ref = oracle.linear_gelu(xb, wb, 2, gelu=True, dt="bf16", threads=THREADS)
    _check(np.ascontiguousarray(got[:, off:off + n]), ref, xb, wb, k, 2.0,
           "view n %d off %d ldy %d" % (n, off, ldy))


@pytest.mark.parametrize("mode,dt", [(0, "bf16"), (2, "bf16"), (2, "f16")])
def test_bert_mlp_shape(q, mode, dt):
    """The up-projection of a BERT-base MLP over 4096 tokens, [4096, 768] x [3072, 768]^T,
    the producer of the GELU workload's input."""
    say("linear gelu 4096x3072x768", mode, dt)
    g, r, xb, wb = _run(q, 4096, 3072, 768, mode, True, 1800, dt=dt)
    err = _check(g, r, xb, wb, 768, 2.0, "bert mlp mode %d %s" % (mode, dt), dt)
    # most outputs are the oracle's 16-bit value itself (binary16 has 3 more
    # bits, so more of them differ by the accumulation order)
    assert np.count_nonzero(err == 0) > (0.95 if dt == "bf16" else 0.75) * err.size


def test_bert_down_projection_shape(q):
    """The down-projection of a BERT-base MLP over 4096 tokens, [4096, 3072] x
    [768, 3072]^T, the product alone: 192 tiles of 128 x 128 (the wide tile
    would leave half the CUs idle) over k = 3072, so the slabs go two ahead."""
    say("linear 4096x768x3072")
    g, r, xb, wb = _run(q, 4096, 768, 3072, 2, False, 1850)
    err = _check(g, r, xb, wb, 3072, 1.0, "bert down projection")
    assert np.count_nonzero(err == 0) > 0.9 * err.size
