"""quake_softmax_noalloc (the split-row softmax on the library's fixed device
scratch, for callers that cannot allocate) against quake_softmax_ws (the same
kernels on a caller workspace), through the C ABI on cuda:0: calls in a row,
the later ones on smaller inputs (the last with rows that are not 16-byte
aligned), bit for bit; the first also against the oracle; a shape beyond the
scratch is refused before any launch."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from compare import check_bits
from gpu_util import THREADS, assert_parity, host_bits, say
from paper_2412_00408_amd import synth

pytestmark = pytest.mark.gpu

SCRATCH = 262144


@pytest.fixture(scope="module")
def q():
    assert torch.cuda.is_available(), "GPU tests need cuda:0"
    from paper_2412_00408_amd import quake
    return quake


def _noalloc(q, x, y, mode=2, t=1.0):
    rows, cols = x.shape
    s = int(torch.cuda.current_stream().cuda_stream)
    return q.lib.quake_softmax_noalloc(x.data_ptr(), y.data_ptr(), rows, cols, cols, cols,
                                       q.DTYPES[x.dtype], mode, t, s)


def test_noalloc_matches_the_workspace_entry_point(q):
    w = synth.WORKLOADS["lmhead_softmax_f32_64x128256"]
    cases = [(w.make(), "f32 64x128256"),
             (synth.normal((24, 40000), 3.0, "bf16", 1400), "bf16 24x40000"),
             # rows starting at every offset from 16 bytes: the shifted split form
             (synth.normal((16, 50257), 3.0, "f32", 1402), "f32 16x50257")]
    for i, (xc, name) in enumerate(cases):
        x = xc.to("cuda:0")
        rows, cols = x.shape
        assert 0 < q.softmax_workspace_size(rows, cols, x.dtype) <= SCRATCH
        ws = q.softmax_workspace(rows, cols, x.dtype)
        ref = q.quake_softmax(x, mode=2, workspace=ws)
        y = torch.full_like(x, 5.0)
        say("noalloc call", i, name)
        assert _noalloc(q, x, y) == q.OK
        torch.cuda.synchronize()
        msg = check_bits(host_bits(y), host_bits(ref), name="noalloc vs ws %s" % name)
        assert msg is None, msg
        if i == 0:
            r = oracle.softmax(host_bits(xc), "f32", 2, threads=THREADS)
            assert_parity(host_bits(y), r, "f32", "op", "noalloc vs oracle %s" % name)


def test_noalloc_refuses_shapes_beyond_its_scratch(q):
    x = torch.zeros((8, 16), device="cuda:0")
    y = torch.empty_like(x)
    s = int(torch.cuda.current_stream().cuda_stream)
    big_rows, big_cols = 1024, 21 * 16384          # 12 * 1024 * 21 + 4 * 1024 + 256 > 262144 bytes
    assert q.softmax_workspace_size(big_rows, big_cols) > SCRATCH
    # refused before anything is launched (the pointers are never dereferenced)
    assert q.lib.quake_softmax_noalloc(x.data_ptr(), y.data_ptr(), big_rows, big_cols, big_cols,
                                       big_cols, 0, 2, 1.0, s) == q.ENOSCRATCH
    assert q.softmax_workspace_size(1024, 20 * 16384) <= SCRATCH
    # rows that need no exchange run as quake_softmax
    xs = synth.normal((3, 1000), 2.0, "f32", 1401).to("cuda:0")
    ys = torch.empty_like(xs)
    assert _noalloc(q, xs, ys) == q.OK
    torch.cuda.synchronize()
    assert check_bits(host_bits(ys), host_bits(q.quake_softmax(xs, mode=2))) is None
