"""GPU robustness: HIP-graph replay of every kernel family (elementwise,
softmax, the 16-bit construction, linear+GELU, fused attention), a first-ever
split-row softmax call made under graph capture, and the split-row exchange
told not to wait at all (the wait-limit word of the caller's workspace), so
that every workgroup recomputes its peers' values, which must give the same
bits."""
import numpy as np
import pytest
import torch

import oracle
from compare import check_bits
from gpu_util import THREADS, assert_parity, host_bits, say
from paper_2412_00408_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def q():
    assert torch.cuda.is_available(), "GPU tests need cuda:0"
    from paper_2412_00408_amd import quake
    return quake


def _ops(q, bufs):
    """One call of each kernel family on preallocated buffers."""
    q.quake_gelu(bufs["gelu_x"], bufs["gelu_y"], mode=2)                       # pipelined stride
    q.quake_sigmoid(bufs["sig_x"], bufs["sig_y"], mode=2, silu=True)           # one-shot
    q.quake_softmax(bufs["attn_x"], bufs["attn_y"], mode=2, t=0.125)           # wave per row
    q.quake_softmax(bufs["lm_x"], bufs["lm_y"], mode=2, workspace=bufs["lm_ws"])  # split rows
    q.quake_softmax(bufs["lm_x"], bufs["lm2_y"], mode=2)                       # long rows
    q.quake_softmax_causal(bufs["attn_x"], bufs["causal_y"], period=512, mode=2, t=0.125)
    q.quake_softmax(bufs["gen_x"], bufs["gen_y"], mode=1)                      # generic
    q.quake_exp16(bufs["e16_x"], bufs["e16_y"], mode=2)                        # 16-bit layout
    q.quake_linear_gelu(bufs["lin_x"], bufs["lin_w"], bufs["lin_y"], mode=2)   # matrix cores
    q.quake_attention(bufs["att_q"], bufs["att_k"], bufs["att_vt"], bufs["att_y"], mode=2,
                      t=0.125, causal=True)                                    # fused attention
    q.quake_attention(bufs["att8_q"], bufs["att8_k"], bufs["att8_vt"], bufs["att8_y"], mode=2,
                      t=0.125, causal=False)                                   # eight waves
    q.quake_attention(bufs["att2p_q"], bufs["att2p_k"], bufs["att2p_vt"], bufs["att2p_y"],
                      mode=2, t=0.125, causal=True)                            # two passes


def quake_ws(rows, cols):
    from paper_2412_00408_amd import quake
    return quake.softmax_workspace(rows, cols)


def _bufs():
    b = {
        "gelu_x": synth.WORKLOADS["gelu_bf16_4096x3072"].make(n=1 << 22).to("cuda:0"),
        "sig_x": synth.WORKLOADS["silu_f16_2p28"].make(n=1 << 26).to("cuda:0"),
        "attn_x": synth.WORKLOADS["attn_softmax_bf16_causal"].make(rows=4096).to("cuda:0"),
        "lm_x": synth.WORKLOADS["lmhead_softmax_f32_64x128256"].make(rows=16).to("cuda:0"),
        "gen_x": synth.normal((37, 1001), 2.0, "f32", 1200).to("cuda:0"),
    }
    b["e16_x"] = synth.WORKLOADS["sigmoid_f16_2p28"].make(n=1 << 20).to("cuda:0")
    b["lin_x"] = synth.normal((256, 768), 1.0, "bf16", 1201).to("cuda:0")
    b["lin_w"] = synth.normal((512, 768), 0.05, "bf16", 1202).to("cuda:0")
    for name, heads, seq, seed in (("att", 4, 512, 1203), ("att8", 2, 700, 1204),
                                   ("att2p", 1, 1100, 1205)):
        qa, ka, va = synth.attention_inputs(heads, seq, seed)
        b[name + "_q"], b[name + "_k"], b[name + "_vt"] = (qa.to("cuda:0"), ka.to("cuda:0"),
                                                           va.to("cuda:0"))
        b[name + "_y"] = torch.empty_like(b[name + "_q"])
    for k in ("gelu", "sig", "attn", "lm", "gen", "e16"):
        b[k + "_y"] = torch.empty_like(b[k + "_x"])
    b["causal_y"] = torch.empty_like(b["attn_x"])
    b["lm2_y"] = torch.empty_like(b["lm_x"])
    b["lm_ws"] = quake_ws(16, 128256)
    b["lin_y"] = torch.empty((256, 512), dtype=torch.bfloat16, device="cuda:0")
    return b


def test_graph_replay_matches_eager(q):
    bufs = _bufs()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):          # eager reference
        _ops(q, bufs)
    s.synchronize()
    ref = {k: v.clone() for k, v in bufs.items() if k.endswith("_y")}
    g = torch.cuda.CUDAGraph()
    for k in ref:
        bufs[k].zero_()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        _ops(q, bufs)
    torch.cuda.synchronize()
    scratch = torch.zeros(1 << 20, device="cuda:0")
    for rep in range(5):
        say("graph replay", rep)
        for k in ref:
            bufs[k].fill_(7.0)
        scratch.add_(1.0)                       # the program's own eager work between replays
        _ = q.quake_gelu(bufs["gelu_x"], mode=0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            msg = check_bits(host_bits(bufs[k]), host_bits(v), name="replay %d %s" % (rep, k))
            assert msg is None, msg
    assert int(bufs["lm_ws"][256:].count_nonzero()) == 0


def test_first_split_call_inside_graph_capture(q):
    # the workspace is the caller's and starts zero-filled, so the very first
    # split-row call may be captured: nothing is allocated or initialised
    w = synth.WORKLOADS["lmhead_softmax_f32_64x128256"]
    x = w.make(rows=24).to("cuda:0")
    ws = q.softmax_workspace(24, 128256)
    y = torch.empty_like(x)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        q.quake_softmax(x, y, mode=2, workspace=ws)
    torch.cuda.synchronize()
    ws_ref = q.softmax_workspace(24, 128256)
    ref = q.quake_softmax(x, mode=2, workspace=ws_ref)
    torch.cuda.synchronize()
    oref = oracle.softmax(host_bits(x), "f32", 2, threads=THREADS)
    assert_parity(host_bits(ref), oref, "f32", "op", "eager split")
    for rep in range(4):
        say("first split call captured, replay", rep)
        y.fill_(3.0)
        _ = q.quake_softmax(x, mode=1, workspace=ws_ref)     # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        msg = check_bits(host_bits(y), host_bits(ref), name="captured split replay %d" % rep)
        assert msg is None, msg
        assert int(ws[256:].count_nonzero()) == 0


def test_split_waits_given_up_give_the_same_bits(q):
    # word 0 of the workspace is the wait limit; 0xFFFFFFFF means no waiting:
    # every workgroup computes every chunk max and sum of its row from x
    # itself, with the owners' loads and summation order, so the bits must be
    # those of the exchange (and the workspace is left zeroed all the same)
    w = synth.WORKLOADS["lmhead_softmax_f32_64x128256"]
    for rows, cols, seed in ((8, 128256, 0), (40, 50000, 1)):
        x = w.make(rows=rows).to("cuda:0") if cols == 128256 else \
            synth.normal((rows, cols), 3.0, "f32", 1300 + seed).to("cuda:0")
        G = (cols + 16383) // 16384
        ref_ws = q.softmax_workspace(rows, cols)
        ref = q.quake_softmax(x, mode=2, workspace=ref_ws)
        ws = q.softmax_workspace(rows, cols)
        ws[0:4].view(torch.int32).fill_(-1)
        say("split waits given up", rows, cols)
        y = q.quake_softmax(x, mode=2, workspace=ws)
        torch.cuda.synchronize()
        assert int(ws[4:8].view(torch.int32)[0]) == rows * G   # every workgroup recomputed
        assert int(ws[256:].count_nonzero()) == 0
        msg = check_bits(host_bits(y), host_bits(ref), name="no-wait %dx%d" % (rows, cols))
        assert msg is None, msg
        # the same workspace back on the default limit: the same bits again
        ws[0:4].view(torch.int32).fill_(0)
        y2 = q.quake_softmax(x, mode=2, workspace=ws)
        torch.cuda.synchronize()
        assert check_bits(host_bits(y2), host_bits(ref)) is None
    oref = oracle.softmax(host_bits(x), "f32", 2, threads=THREADS)
    assert_parity(host_bits(y), oref, "f32", "op", "no-wait vs the oracle")


@pytest.mark.parametrize("rows,cols,dt", [(24, 50257, "f32"), (9, 100001, "bf16"), (8, 131065, "f16"),
                                          (16, 16389, "f32"), (8, 32767, "f32")])
def test_split_waits_given_up_on_shifted_rows(q, rows, cols, dt):
    # rows whose start is not 16-byte aligned take the split kernel's shifted
    # form: the recomputation from x masks the same elements as the owners.
    # When cols' chunk count does not cover the most vectors such a row can
    # span (32767 f32), the one-workgroup kernel runs and the workspace is
    # not touched.
    x = synth.normal((rows, cols), 3.0, dt, 1400 + cols % 89).to("cuda:0")
    V = 4 if dt == "f32" else 8
    nvm = (cols + 2 * V - 2) // V
    split = (nvm * V + 16383) // 16384 == (cols + 16383) // 16384
    G = (cols + 16383) // 16384 if split else 0
    ref = q.quake_softmax(x, mode=2, workspace=q.softmax_workspace(rows, cols))
    ws = q.softmax_workspace(rows, cols)
    ws[0:4].view(torch.int32).fill_(-1)
    say("split waits given up, shifted rows", dt, rows, cols)
    y = q.quake_softmax(x, mode=2, workspace=ws)
    torch.cuda.synchronize()
    assert int(ws[4:8].view(torch.int32)[0]) == rows * G
    assert int(ws[256:].count_nonzero()) == 0
    assert check_bits(host_bits(y), host_bits(ref), name="no-wait shifted %dx%d" % (rows, cols)) is None
    oref = oracle.softmax(host_bits(x.cpu()), dt, 2, threads=THREADS)
    assert_parity(host_bits(y), oref, dt, "op", "no-wait shifted vs the oracle")
