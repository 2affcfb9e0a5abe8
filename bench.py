#!/usr/bin/env python3
"""Benchmark of the QuAKE hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--mode quake2]

A step is one launch of the operator over the whole workload (every step of
the fused path: load + widen, (row max), affine map, clamp, convert, QuAKE2
refinement, consumer, narrow + store). The default workload is the GELU of a
BERT-base MLP activation, bf16 [4096, 3072]. Inputs are seeded synthetic data
resident in HBM before the timed region; the timed launches rotate over
enough input/output buffer pairs (>= 1 GiB) that the 256 MB Infinity Cache
cannot serve them. Launch sequences are captured in a HIP graph (eager
launches if capture is not possible) and timed with HIP events on the
launching stream. Before the first measurement the kernel runs untimed for
--prewarm seconds (an idle MI355X takes a few hundred milliseconds to reach
its steady clocks). The same kernel with the hardware exp2 (EXACT), with
first-order QuAKE and with the minimax-coefficient QuAKE2 is timed in the same
process for the speedup.

Prints ONE JSON line. The oracle (CPU, plain C) is timed on the host cores on
the same workload as `cpu_baseline`.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0       # MI355X HBM3E, AMD published peak
MODE_IDS = {"exact": 0, "quake1": 1, "quake2": 2, "quake2m": 3}
KERNEL_SOURCES = ["paper_2412_00408_amd/csrc/elementwise.hip",
                  "paper_2412_00408_amd/csrc/softmax.hip",
                  "paper_2412_00408_amd/csrc/quake_device.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.md")


def source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="gelu_bf16_4096x3072")
    ap.add_argument("--mode", default="quake2", choices=sorted(MODE_IDS))
    ap.add_argument("--launch", default="graph", choices=["graph", "eager"])
    ap.add_argument("--only", action="store_true",
                    help="time only --workload in --mode (for profiler passes)")
    ap.add_argument("--section", choices=["attention", "linear_gelu"],
                    help="time only the fused attention (quake_attention) or the fused "
                         "linear+GELU (quake_linear_gelu) and print its JSON (for profiler passes)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-table4", action="store_true",
                    help="skip the fused-vs-unfused study (the paper's Table IV, on this GPU)")
    ap.add_argument("--mall-resident", action="store_true",
                    help="also time the headline kernel on one reused buffer pair (warm)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="also run torch copies of MIB MiB (reference kernel for counters)")
    ap.add_argument("--prewarm", type=float, default=1.0, metavar="SECONDS",
                    help="untimed back-to-back launches before the first measurement")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU work (thread-seconds) spent timing the oracle")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# GPU side
# ---------------------------------------------------------------------------

def make_launcher(q, w, mode, xs, ys, fused=True):
    """Returns f(i) that launches the operator on buffer pair i (raw C ABI)."""
    import torch
    L = q.lib
    dt = q.DTYPES[xs[0].dtype]
    n = xs[0].numel()
    stream = lambda: int(torch.cuda.current_stream().cuda_stream)  # noqa: E731
    xp = [x.data_ptr() for x in xs]
    yp = [y.data_ptr() for y in ys]
    if w.op == "gelu":
        g = L.quake_gelu if fused else L.quake_gelu_unfused

        def f(i):
            return g(xp[i], yp[i], n, dt, mode, stream())
    elif w.op in ("sigmoid", "silu"):
        silu = int(w.op == "silu")

        def f(i):
            return L.quake_sigmoid(xp[i], yp[i], n, dt, mode, silu, stream())
    elif w.op in ("exp", "exp16"):
        e = L.quake_exp16 if w.op == "exp16" else L.quake_exp

        def f(i):
            return e(xp[i], yp[i], n, dt, mode, 1.0, 0.0, stream())
    elif w.op == "softmax":
        rows, cols = w.rows, w.cols
        sm = L.quake_softmax if fused else L.quake_softmax_unfused

        def f(i):
            return sm(xp[i], yp[i], rows, cols, cols, cols, dt, mode, w.t, stream())
    else:
        raise KeyError(w.op)
    return f


def prewarm(q, w, x_host, seconds, launch_kind):
    """Untimed: run the workload's kernel back to back for about `seconds`, in
    the same way as a measurement (rotating buffers, same launch kind), so the
    GPU leaves its idle clock state before anything is measured (the first few
    hundred milliseconds of work on an idle MI355X run several percent slower)."""
    steps = max(1, int(seconds * 5e12 / w.algo_bytes))     # at about 5 TB/s
    time_workload(q, w, MODE_IDS["quake2"], x_host, steps, 0, launch_kind)


def time_workload(q, w, mode, x_host, steps, warmup, launch_kind, fused=True, pairs=None):
    """ms per launch over `steps` launches, nbuf per graph replay, rotating
    over `pairs` input/output buffer pairs (default nbuf: enough for >= 1 GiB,
    beyond the 256 MB Infinity Cache)."""
    import torch
    nbuf = min(64, max(2, math.ceil((1 << 30) / w.algo_bytes)))
    pairs = nbuf if pairs is None else pairs
    xs, ys = [], []
    x0 = x_host.to("cuda:0")
    for _ in range(pairs):
        xs.append(x0.clone())
        ys.append(torch.empty_like(x0))
    del x0
    f0 = make_launcher(q, w, mode, xs, ys, fused)

    def f(i):
        return f0(i % pairs)
    for i in range(max(warmup, nbuf)):
        rc = f(i % nbuf)
        if rc != 0:
            raise RuntimeError("launch failed: %s" % q.status_str(rc))
    torch.cuda.synchronize()

    kind = launch_kind
    graph = None
    if kind == "graph":
        try:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):        # per-stream workspaces exist before capture
                for i in range(nbuf):
                    f(i)
            s.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.stream(s):
                with torch.cuda.graph(graph, stream=s):
                    for i in range(nbuf):
                        rc = f(i)
                        if rc != 0:
                            raise RuntimeError(q.status_str(rc))
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
        except Exception as e:  # cooperative launches may not be capturable
            graph = None
            kind = "eager (graph capture failed: %s)" % str(e).splitlines()[0][:80]
            torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    if graph is not None:
        # exactly `steps` launches: whole replays of the nbuf-launch graph, then
        # the remainder launched directly on the same stream
        reps, rem = divmod(steps, nbuf)
        launches = steps
        graph.replay()
        torch.cuda.synchronize()
        start.record(stream)
        for _ in range(reps):
            graph.replay()
        for i in range(rem):
            f(i)
        end.record(stream)
    else:
        launches = steps
        start.record(stream)
        for i in range(steps):
            f(i % nbuf)
        end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / launches
    out = ys[(launches - 1) % pairs]
    del xs
    return ms, launches, pairs, kind, out


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, on the host cores
# ---------------------------------------------------------------------------

def copy_ceiling(w, reps):
    """A plain copy of the workload's input bytes (read numel elements, write
    numel elements: the same algorithmic bytes as the operator) with torch's
    copy kernel, over >= 1 GiB of rotating buffer pairs, graph-captured: the
    bandwidth a kernel moving these bytes reaches on this machine."""
    import torch
    from paper_2412_00408_amd import synth
    nb = min(64, max(2, math.ceil((1 << 30) / w.algo_bytes)))
    n = w.numel * synth.ELEM_BYTES[w.dt] // 4
    srcs = [torch.ones(n, dtype=torch.float32, device="cuda:0") for _ in range(nb)]
    dsts = [torch.empty_like(srcs[0]) for _ in range(nb)]

    def f(i, stream):
        dsts[i].copy_(srcs[i])
    ms = graph_ms(f, nb, max(10, reps // nb))
    del srcs, dsts
    return {"ms": ms, "gbps": round(w.algo_bytes / (ms * 1e-3) / 1e9, 2),
            "kernel": "torch copy_ of %d bytes" % (n * 4)}


def cpu_baseline(w, x_host, cpu_seconds):
    import oracle
    from paper_2412_00408_amd import synth
    try:
        threads = len(os.sched_getaffinity(0))
    except AttributeError:
        threads = os.cpu_count() or 1
    threads = max(1, min(threads, 16))
    xb = synth.bits(x_host)
    mode = oracle.Q2

    def run(th, sample):
        xs = xb[:sample] if w.op != "softmax" else xb[:sample]
        if w.op == "gelu":
            oracle.gelu(xs, w.dt, mode, threads=th)
        elif w.op in ("sigmoid", "silu"):
            oracle.sigmoid(xs, w.dt, mode, silu=(w.op == "silu"), threads=th)
        else:
            oracle.softmax(xs.reshape(-1, w.cols), w.dt, mode, t=w.t, threads=th)

    # size the sample so one pass is ~0.5 s of CPU work on one thread
    unit = w.cols if w.op == "softmax" else 1
    total_units = w.numel // unit
    probe = max(1, min(total_units, (1 << 20) // unit))
    t0 = time.perf_counter()
    run(1, probe * unit if w.op != "softmax" else probe)
    per_unit = (time.perf_counter() - t0) / probe
    sample_units = int(min(total_units, max(1, 0.5 * threads / max(per_unit, 1e-12))))
    sample = sample_units * unit if w.op != "softmax" else sample_units
    elems = sample_units * unit
    reps, wall = 0, 0.0
    while wall * threads < cpu_seconds and reps < 1000:
        t0 = time.perf_counter()
        run(threads, sample)
        wall += time.perf_counter() - t0
        reps += 1
    gbps = (2 * synth.ELEM_BYTES[w.dt] * elems * reps) / wall / 1e9
    # single thread, as the paper's protocol (one pass)
    t0 = time.perf_counter()
    run(1, sample)
    one = (2 * synth.ELEM_BYTES[w.dt] * elems) / (time.perf_counter() - t0) / 1e9
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    cpu = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {
        "value": round(gbps, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
        "cpu_model": cpu,
        "sample": "%d of %d elements of %s, quake2, %d passes over %.1f s wall" % (
            elems, w.numel, w.name, reps, wall),
        "single_thread_value": round(one, 3),
        "single_thread_mode_ratios": cpu_mode_ratios(w, xb),
    }


def cpu_mode_ratios(w, xb):
    """The oracle's own operators timed on one host core (the paper's protocol:
    single thread, scalar code) in every mode, on the first 2^20 elements (or
    the rows holding them), median of three passes: the host-CPU counterpart
    of the QuAKE-versus-exp comparison. EXACT here is the oracle's reference
    exponential (binary32 result of a double exp2), the plug-in exp of the
    unfused operator is the 'vanilla' form of the fusion study."""
    import oracle
    n = min(xb.size, 1 << 20)
    xs = xb.reshape(-1)[:n] if w.op != "softmax" else xb[:max(1, n // w.cols)]

    def op(mode, fused=True):
        if w.op == "gelu":
            (oracle.gelu if fused else oracle.gelu_unfused)(xs, w.dt, mode, threads=1)
        elif w.op in ("sigmoid", "silu"):
            oracle.sigmoid(xs, w.dt, mode, silu=(w.op == "silu"), threads=1)
        else:
            (oracle.softmax if fused else oracle.softmax_unfused)(
                xs.reshape(-1, w.cols), w.dt, mode, t=w.t, threads=1)

    def med(fn):
        ts = []
        for _ in range(3):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return sorted(ts)[1]

    t = {m: med(lambda m=m: op(MODE_IDS[m])) for m in ("exact", "quake1", "quake2", "quake2m")}
    out = {"elements": int(xs.size), "ns_per_element": {m: round(v / xs.size * 1e9, 2)
                                                       for m, v in t.items()},
           "speedup_vs_exact": {m: round(t["exact"] / v, 3) for m, v in t.items() if m != "exact"}}
    if w.op in ("gelu", "softmax"):
        van = med(lambda: op(0, fused=False))
        out["speedup_vs_unfused_exact"] = {m: round(van / t[m], 3)
                                           for m in ("quake1", "quake2", "quake2m")}
    return out


def native16(q, synth, a):
    """e^x over 2^28 binary16 elements: the binary32 path (quake_exp: binary32
    arithmetic, result narrowed) against the construction in binary16's own
    layout (quake_exp16), QuAKE and QuAKE2; both read and write 2 bytes per
    element."""
    import dataclasses
    w = synth.EXTRA_WORKLOADS["exp_f16_2p28"]
    xh = w.make()
    steps = max(100, min(a.steps, int(1e12 / w.algo_bytes)))
    out = {"algo_bytes": w.algo_bytes}
    for path, wop in (("binary32_path", w), ("native16", dataclasses.replace(w, op="exp16"))):
        for m in ("quake1", "quake2"):
            ms = time_workload(q, wop, MODE_IDS[m], xh, steps, a.warmup, a.launch)[0]
            out["%s_%s_ms" % (path, m)] = ms
            out["%s_%s_gbps" % (path, m)] = round(w.algo_bytes / (ms * 1e-3) / 1e9, 2)
    out["native16_speedup"] = {m: round(out["binary32_path_%s_ms" % m] / out["native16_%s_ms" % m], 4)
                               for m in ("quake1", "quake2")}
    return out


PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix-core peak


def graph_ms(f, nb, reps):
    """Average ms per launch of f(i, stream) for i = 0 .. nb-1 (one launch on
    operand set i, enqueued on `stream`), captured once in a HIP graph and
    replayed `reps` times: the Python cost of a launch stays out of the timed
    region."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for i in range(nb):
            f(i, s.cuda_stream)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(nb):
                rc = f(i, s.cuda_stream)
                if rc not in (0, None):
                    raise RuntimeError("launch failed: %d" % rc)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for _ in range(reps):
        g.replay()
    e1.record(st)
    torch.cuda.synchronize()
    del g
    return e0.elapsed_time(e1) / (reps * nb)


def linear_gelu(q, synth, a):
    """GELU(x w^T) for the up-projection of a BERT-base MLP over 4096 tokens
    (x [4096, 768], w [3072, 768], bf16): the fused kernel in every mode, the
    same product without the GELU, the product followed by quake_gelu, and
    torch.matmul (the vendor BLAS) for context. Eight rotating operand sets
    (about 290 MB) keep the timed launches out of the 256 MB Infinity Cache;
    each variant is captured in a HIP graph over the eight sets and replayed."""
    import torch
    m, n, k = 4096, 3072, 768
    nb = 8
    xs = [synth.normal((m, k), 1.0, "bf16", 1900 + i).to("cuda:0") for i in range(nb)]
    ws = [synth.normal((n, k), 0.05, "bf16", 1950 + i).to("cuda:0") for i in range(nb)]
    ys = [torch.empty((m, n), dtype=torch.bfloat16, device="cuda:0") for _ in range(nb)]
    wts = [w.t().contiguous() for w in ws]
    flop = 2.0 * m * n * k
    reps = max(10, min(a.steps, 2000) // nb)
    L = q.lib

    def lin(mode, gelu):
        def f(i, stream):
            return L.quake_linear_gelu(xs[i].data_ptr(), ws[i].data_ptr(), ys[i].data_ptr(), m, n, k,
                                       k, k, n, 2, mode, gelu, stream)
        return f

    def gelu_only(i, stream):
        return L.quake_gelu(ys[i].data_ptr(), ys[i].data_ptr(), m * n, 2, 2, stream)

    def vendor(i, stream):
        torch.matmul(xs[i], wts[i], out=ys[i])

    out = {"shape_mnk": [m, n, k], "flop": flop, "peak_tflops": PEAK_BF16_TFLOPS,
           "launch": "graph (%d launches per replay)" % nb}
    for mname in ("exact", "quake1", "quake2", "quake2m"):
        out["fused_%s_ms" % mname] = graph_ms(lin(MODE_IDS[mname], 1), nb, reps)
    ms0 = graph_ms(lin(2, 0), nb, reps)
    msg = graph_ms(gelu_only, nb, reps)
    mst = graph_ms(vendor, nb, reps)
    out.update({"product_only_ms": ms0, "quake_gelu_ms": msg, "torch_matmul_ms": mst})
    out["fused_quake2_tflops"] = round(flop / (out["fused_quake2_ms"] * 1e-3) / 1e12, 1)
    out["product_only_tflops"] = round(flop / (ms0 * 1e-3) / 1e12, 1)
    out["product_only_frac_of_peak"] = round(out["product_only_tflops"] / PEAK_BF16_TFLOPS, 4)
    out["fused_vs_product_then_gelu"] = round((ms0 + msg) / out["fused_quake2_ms"], 4)
    out["epilogue_ms_over_product"] = {mm: round(out["fused_%s_ms" % mm] - ms0, 5)
                                       for mm in ("exact", "quake1", "quake2", "quake2m")}
    del xs, ws, ys, wts
    return out


def torch_sdpa_ms(sets, vs, causal, t, n):
    """ms per call of torch.nn.functional.scaled_dot_product_attention on the
    given (q, k, v^T, o) sets (v passed as vs, [heads, seq, d]) with only the
    flash and memory-efficient backends allowed (no fallback to the math
    path), launched eagerly back to back; None where neither is available."""
    import torch
    from torch.nn.attention import SDPBackend, sdpa_kernel
    try:
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
            def f(i):
                qg, kg, _, _ = sets[i % len(sets)]
                return torch.nn.functional.scaled_dot_product_attention(
                    qg[None], kg[None], vs[i % len(vs)][None], is_causal=bool(causal), scale=t)
            for i in range(10):
                f(i)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(n):
                f(i)
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / n
    except RuntimeError:
        return None


def fused_attention(q, synth, a, heads=96, seq=512):
    """softmax(t q k^T) v over the attention workload's heads (8 x 12 heads,
    512 tokens, head dimension 64, bf16, t = 1/8; or another heads x seq) in one kernel
    (quake_attention), causal and not, in every mode, against the explicit
    path on the same inputs: the score product (torch.bmm, the vendor BLAS),
    quake_softmax_causal / quake_softmax over the bf16 scores, and the second
    product (torch.bmm). Algorithmic bytes: q, k and v read once, o written
    once; useful flops: 4 d per (query, live key) pair. The fused launches are
    captured in a HIP graph over 12 rotating operand sets (about 300 MB, more
    than the Infinity Cache holds) and replayed; the explicit path is captured
    the same way over two sets. For context, torch's own fused attention
    (scaled_dot_product_attention restricted to its flash / memory-efficient
    kernels, exact exponential, so other numbers) is timed over the same 12
    rotating sets with eager launches."""
    import torch
    d, t, nb = 64, 0.125, 12
    sets = []
    for i in range(nb):
        qc, kc, vtc = synth.attention_inputs(heads, seq, 2000 + i)
        sets.append((qc.to("cuda:0"), kc.to("cuda:0"), vtc.to("cuda:0"),
                     torch.empty((heads, seq, d), dtype=torch.bfloat16, device="cuda:0")))
    L = q.lib
    algo = 4 * heads * seq * d * 2
    pairs = {1: heads * seq * (seq + 1) // 2, 0: heads * seq * seq}
    # about the same GPU time per configuration at every length
    reps = max(10, min(a.steps, 20000) // nb * 512 * 512 // (seq * seq))

    out = {"heads": heads, "seq": seq, "head_dim": d, "t": t, "algo_bytes": algo,
           "launch": "graph (%d launches per replay)" % nb}
    scores = torch.empty((heads, seq, seq), dtype=torch.bfloat16, device="cuda:0")
    probs = torch.empty_like(scores)
    kts = [kk.transpose(1, 2).contiguous() for _, kk, _, _ in sets[:2]]
    vs = [vt.transpose(1, 2).contiguous() for _, _, vt, _ in sets[:2]]
    vs_all = vs + [vt.transpose(1, 2).contiguous() for _, _, vt, _ in sets[2:]]
    for causal, name in ((1, "causal"), (0, "noncausal")):
        r = {}
        for mname, mid in MODE_IDS.items():
            def f(i, stream, mid=mid, causal=causal):
                qg, kg, vg, og = sets[i]
                return L.quake_attention(qg.data_ptr(), kg.data_ptr(), vg.data_ptr(),
                                         og.data_ptr(), heads, seq, d, seq, 2, mid, t, causal,
                                         stream)
            r[mname] = graph_ms(f, nb, reps)
        flop = 4.0 * d * pairs[causal]

        def explicit(i, stream):
            qg, _, _, og = sets[i]
            torch.bmm(qg, kts[i], out=scores)
            if causal:
                rc = L.quake_softmax_causal(scores.data_ptr(), probs.data_ptr(), heads * seq, seq,
                                            seq, seq, seq, 0, 1, 2, 2, t, stream)
            else:
                rc = L.quake_softmax(scores.data_ptr(), probs.data_ptr(), heads * seq, seq, seq,
                                     seq, 2, 2, t, stream)
            if rc != 0:
                raise RuntimeError(q.status_str(rc))
            torch.bmm(probs, vs[i], out=og)
        ms_ex = graph_ms(explicit, 2, 100)
        ms_sdpa = torch_sdpa_ms(sets, vs_all, causal, t, max(24, reps // 10))
        ms = r["quake2"]
        out[name] = {
            "fused_ms": {m: round(v, 6) for m, v in r.items()},
            "speedup_vs_exact": {m: round(r["exact"] / v, 4) for m, v in r.items() if m != "exact"},
            "useful_flop": flop,
            "quake2_gbps": round(algo / (ms * 1e-3) / 1e9, 2),
            "quake2_frac_of_hbm_peak": round(algo / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
            "quake2_tflops": round(flop / (ms * 1e-3) / 1e12, 2),
            "quake2_frac_of_bf16_peak": round(flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "explicit_quake2_ms": round(ms_ex, 6),
            "fused_speedup_vs_explicit": round(ms_ex / ms, 3),
            "torch_sdpa_ms": None if ms_sdpa is None else round(ms_sdpa, 6),
            "fused_speedup_vs_torch_sdpa": None if ms_sdpa is None else round(ms_sdpa / ms, 3),
        }
    del sets, scores, probs, kts, vs, vs_all
    return out


def implicit_causal(q, synth, a):
    """The attention workload with the causal mask implied (quake_softmax_causal):
    only live entries are read, so its algorithmic bytes are the live inputs
    plus every output."""
    import torch
    w = synth.WORKLOADS["attn_softmax_bf16_causal"]
    xh = w.make()
    nbuf = 12
    xs = [xh.to("cuda:0") for _ in range(nbuf)]
    ys = [torch.empty_like(xs[0]) for _ in range(nbuf)]
    L = q.lib
    res = {}
    for mode, wm in ((0, 1), (2, 1), (2, 0)):
        def f(i, mode=mode, wm=wm):
            return L.quake_softmax_causal(xs[i].data_ptr(), ys[i].data_ptr(), w.rows, w.cols, w.cols,
                                          w.cols, w.cols, 0, wm, 2, mode, w.t,
                                          int(torch.cuda.current_stream().cuda_stream))
        for i in range(nbuf):
            f(i)
        torch.cuda.synchronize()
        st = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        steps = 960
        e0.record(st)
        for i in range(steps):
            f(i % nbuf)
        e1.record(st)
        torch.cuda.synchronize()
        res[(mode, wm)] = e0.elapsed_time(e1) / steps
    heads = w.shape[0] * w.shape[1]
    live = heads * (w.cols * (w.cols + 1) // 2)
    algo = 2 * live + 2 * w.numel
    ms = res[(2, 1)]
    # outputs stored without masked writes: whole 16-byte vectors holding a live entry
    vecs = heads * sum((i // 8 + 1) for i in range(w.cols))
    algo_nw = 2 * live + 16 * vecs
    ms_nw = res[(2, 0)]
    return {"quake2_ms": ms, "algo_bytes": algo, "quake2_gbps": round(algo / (ms * 1e-3) / 1e9, 2),
            "frac_of_peak": round(algo / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
            "speedup_vs_exact": round(res[(0, 1)] / ms, 4),
            "no_masked_writes": {"quake2_ms": ms_nw, "algo_bytes": algo_nw,
                                 "quake2_gbps": round(algo_nw / (ms_nw * 1e-3) / 1e9, 2),
                                 "speedup_vs_explicit_mask_input": None},
            "launch": "eager"}


def table4(q, synth, w_head, x_head, a):
    """The paper's fusion study (Sec. V-A, Table IV) on this GPU: the vanilla
    operator (unfused, exact exp), QuAKE plugged in without folding, and the
    fused QuAKE operators, on the paper's op-level shapes and on two workloads
    above. Ratios are time(vanilla)/time(unfused QuAKE) ("without fusion") and
    time(unfused)/time(fused) ("additional from fusion")."""
    out = {}
    cases = list(synth.TABLE4_WORKLOADS.values()) + [synth.WORKLOADS["gelu_bf16_4096x3072"],
                                                     synth.WORKLOADS["attn_softmax_bf16_causal"]]
    for w in cases:
        xh = x_head if w.name == w_head.name else w.make()
        steps = max(50, min(a.steps, int(1e12 / w.algo_bytes)))    # about 0.2 s per variant
        t = {}
        for key, mode, fused in (("vanilla", 0, False), ("unfused_quake1", 1, False),
                                 ("unfused_quake2", 2, False), ("fused_exact", 0, True),
                                 ("fused_quake1", 1, True), ("fused_quake2", 2, True)):
            t[key] = time_workload(q, w, mode, xh, steps, 10, a.launch, fused)[0]
        out[w.name] = {
            "ms": {k: round(v, 6) for k, v in t.items()},
            "speedup_without_fusion": {"quake1": round(t["vanilla"] / t["unfused_quake1"], 4),
                                       "quake2": round(t["vanilla"] / t["unfused_quake2"], 4)},
            "additional_speedup_from_fusion": {
                "quake1": round(t["unfused_quake1"] / t["fused_quake1"], 4),
                "quake2": round(t["unfused_quake2"] / t["fused_quake2"], 4)},
            "fused_quake2_gbps": round(w.algo_bytes / (t["fused_quake2"] * 1e-3) / 1e9, 2),
        }
        del xh
    return out


def traffic_for(name, hash_now):
    """HBM bytes per launch measured by rocprofv3 FETCH_SIZE / WRITE_SIZE passes
    (profiles/traffic.md), or None if absent or taken on other kernel sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    hashes = [ln.split(":", 1)[1].strip() for ln in text.splitlines() if ln.startswith("source_hash:")]
    if not hashes or hashes[-1] != hash_now:
        return None
    for ln in text.splitlines():
        cells = [c.strip() for c in ln.strip().strip("|").split("|")]
        if len(cells) == 8 and cells[0] == name:
            return int(cells[5])
    return None


def main():
    a = parse()
    if a.gpus != 1:
        print("bench.py measures one GPU only: libquake's hot path runs on a single MI355X and "
              "has no multi-GPU mode (asked for --gpus %d)" % a.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2412_00408_amd import quake as q, synth

    assert torch.cuda.is_available(), "bench.py needs cuda:0"
    if a.calibrate_copy:
        nb = a.calibrate_copy << 20
        src = torch.empty(nb // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
    if a.section == "attention":
        if a.prewarm > 0:
            qc, kc, vtc = synth.attention_inputs(96, 512, 1)
            qg, kg, vg = qc.to("cuda:0"), kc.to("cuda:0"), vtc.to("cuda:0")
            t_end = time.time() + a.prewarm
            while time.time() < t_end:
                q.quake_attention(qg, kg, vg, mode=MODE_IDS[a.mode], t=0.125)
            torch.cuda.synchronize()
            del qg, kg, vg
        print(json.dumps({"attention_bf16_96x512x64": fused_attention(q, synth, a),
                          "attention_bf16_64x1024x64": fused_attention(q, synth, a, 64, 1024),
                          "attention_bf16_32x2048x64": fused_attention(q, synth, a, 32, 2048)}),
              flush=True)
        return
    if a.section == "linear_gelu":
        if a.prewarm > 0:
            xg = synth.normal((4096, 768), 1.0, "bf16", 1900).to("cuda:0")
            wg = synth.normal((3072, 768), 0.05, "bf16", 1950).to("cuda:0")
            t_end = time.time() + a.prewarm
            while time.time() < t_end:
                q.quake_linear_gelu(xg, wg, mode=MODE_IDS[a.mode])
            torch.cuda.synchronize()
            del xg, wg
        print(json.dumps({"linear_gelu_bf16_4096x3072x768": linear_gelu(q, synth, a)}), flush=True)
        return
    w = synth.WORKLOADS[a.workload]
    x_host = w.make()

    if a.prewarm > 0:
        prewarm(q, w, x_host, a.prewarm, a.launch)
    modes = [a.mode] if a.only else ["exact", "quake1", "quake2", "quake2m"]
    res = {}
    for m in modes:
        ms, launches, nbuf, kind, _ = time_workload(q, w, MODE_IDS[m], x_host, a.steps, a.warmup,
                                                    a.launch)
        res[m] = dict(ms=ms, gbps=w.algo_bytes / (ms * 1e-3) / 1e9, launches=launches, nbuf=nbuf,
                      launch=kind)
    head = res[a.mode]
    hnow = source_hash()
    tb = traffic_for(w.name + ":" + a.mode, hnow)
    line = {
        # value: GB/s of algorithmic HBM traffic (input read once + output
        # written once); roofline.frac: the fraction of the HBM peak;
        # speedup_vs_exact: against the same kernel with the exact exponential
        "metric": "softmax/GELU GB/s and % of HBM roofline on 1 MI355X; speedup vs exact-exp kernel",
        "value": round(head["gbps"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": head["launches"],
        "warmup": a.warmup,
        "ms_per_step": head["ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded, %s)" % w.name,
        "config": {"workload": w.name, "op": w.op, "io_dtype": w.dt, "shape": list(w.shape),
                   "mode": a.mode, "elements": w.numel, "algo_bytes": w.algo_bytes,
                   "launch": head["launch"], "rotating_buffer_pairs": head["nbuf"]},
        "roofline": {"bound": "hbm", "achieved": round(head["gbps"], 2), "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(head["gbps"] / PEAK_HBM_GBPS, 4),
                     "traffic": tb},
        "modes": {m: {"ms_per_launch": r["ms"], "gbps": round(r["gbps"], 2),
                      "elements_per_s": w.numel / (r["ms"] * 1e-3)} for m, r in res.items()},
    }
    if not a.only:
        cc = copy_ceiling(w, a.steps)
        line["copy_ceiling"] = dict(cc, frac=round(cc["gbps"] / PEAK_HBM_GBPS, 4),
                                    value_over_copy=round(head["gbps"] / cc["gbps"], 4))
    if "exact" in res:
        line["speedup_vs_exact"] = {m: round(res["exact"]["ms"] / r["ms"], 4)
                                    for m, r in res.items() if m != "exact"}
    if not a.no_cpu_baseline and not a.only:
        line["cpu_baseline"] = cpu_baseline(w, x_host, a.cpu_seconds)
    if not a.no_secondary and not a.only:
        sec = {}
        for name, w2 in synth.WORKLOADS.items():
            if name == w.name:
                continue
            xh = w2.make()
            r2 = {}
            # about 0.2 s of GPU time per mode at ~5 TB/s, at most --steps launches
            sec_steps = max(100, min(a.steps, int(1e12 / w2.algo_bytes)))
            for m in ("exact", "quake1", "quake2", "quake2m"):
                ms, launches, nbuf, kind, _ = time_workload(q, w2, MODE_IDS[m], xh,
                                                            sec_steps, a.warmup, a.launch)
                r2[m] = (ms, kind)
            ms2 = r2["quake2"][0]
            gb = w2.algo_bytes / (ms2 * 1e-3) / 1e9
            sec[name] = {"quake2_ms": ms2, "quake2_gbps": round(gb, 2),
                         "frac_of_peak": round(gb / PEAK_HBM_GBPS, 4),
                         "speedup_vs_exact": round(r2["exact"][0] / ms2, 4),
                         "quake1_speedup_vs_exact": round(r2["exact"][0] / r2["quake1"][0], 4),
                         "quake2m_speedup_vs_exact": round(r2["exact"][0] / r2["quake2m"][0], 4),
                         "launch": r2["quake2"][1]}
            del xh
        sec["exp_f16_2p28"] = native16(q, synth, a)
        sec["linear_gelu_bf16_4096x3072x768"] = linear_gelu(q, synth, a)
        sec["attention_bf16_96x512x64"] = fused_attention(q, synth, a)
        sec["attention_bf16_64x1024x64"] = fused_attention(q, synth, a, 64, 1024)
        sec["attention_bf16_32x2048x64"] = fused_attention(q, synth, a, 32, 2048)
        imp = implicit_causal(q, synth, a)
        imp["no_masked_writes"]["speedup_vs_explicit_mask_input"] = round(
            sec["attn_softmax_bf16_causal"]["quake2_ms"] / imp["no_masked_writes"]["quake2_ms"], 4)
        sec["attn_softmax_bf16_causal_implicit"] = imp
        line["secondary"] = sec
    if not a.no_table4 and not a.only:
        line["table4"] = table4(q, synth, w, x_host, a)
    if a.mall_resident and not a.only:
        # the same kernel on one input/output pair reused launch after launch, so
        # that the Infinity Cache (256 MB) serves much of it: context, not the
        # metric (opt-in, so that a kernel trace of the default command averages
        # cold launches only)
        ms_w, _, _, kind_w, _ = time_workload(q, w, MODE_IDS[a.mode], x_host, a.steps, a.warmup,
                                              a.launch, pairs=1)
        line["mall_resident"] = {"ms_per_launch": ms_w,
                                 "gbps": round(w.algo_bytes / (ms_w * 1e-3) / 1e9, 2),
                                 "rotating_buffer_pairs": 1, "launch": kind_w,
                                 "note": "one buffer pair reused (warm, MALL-resident); "
                                         "not the metric"}
    line["kernel_source_hash"] = hnow
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
