"""Helpers for the GPU parity tests: move seeded inputs to cuda:0, run the HIP
path through the C ABI binding, run the oracle on the same host bytes, and
compare with the tolerances of compare.py."""
from __future__ import annotations

import os
import sys

import numpy as np
import torch

import oracle
from compare import check
from paper_2412_00408_amd import synth

THREADS = max(1, min(16, os.cpu_count() or 1))
DTS = {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}


def say(*a):
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def host_bits(t: torch.Tensor) -> np.ndarray:
    return synth.bits(t.detach().to("cpu"))


def run_elementwise(q, op: str, x_cpu: torch.Tensor, mode: int, **kw):
    """Returns (gpu_bits, oracle_bits, dt) for one elementwise operator."""
    dt = DTS[x_cpu.dtype]
    xb = host_bits(x_cpu)
    xg = x_cpu.to("cuda:0")
    if op == "exp":
        yg = q.quake_exp(xg, mode=mode, a=kw.get("a", 1.0), b=kw.get("b", 0.0))
        ref = oracle.exp(xb, dt, mode, a=kw.get("a", 1.0), b=kw.get("b", 0.0), threads=THREADS)
    elif op == "gelu":
        yg = q.quake_gelu(xg, mode=mode)
        ref = oracle.gelu(xb, dt, mode, threads=THREADS)
    elif op == "gelu_unfused":
        yg = q.quake_gelu_unfused(xg, mode=mode)
        ref = oracle.gelu_unfused(xb, dt, mode, threads=THREADS)
    elif op in ("sigmoid", "silu"):
        yg = q.quake_sigmoid(xg, mode=mode, silu=(op == "silu"))
        ref = oracle.sigmoid(xb, dt, mode, silu=(op == "silu"), threads=THREADS)
    else:
        raise KeyError(op)
    torch.cuda.synchronize()
    return host_bits(yg), ref, dt


def kind_of(op: str, mode: int) -> str:
    if op == "exp":
        return "exact_bits" if mode != 0 else "exp_exact"
    return "op"


def assert_parity(gpu, ref, dt, kind, name):
    msg = check(gpu, ref, dt, kind, name)
    assert msg is None, msg
