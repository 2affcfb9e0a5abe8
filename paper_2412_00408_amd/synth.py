"""Seeded synthetic inputs with the shapes and value distributions of the
operator workloads QuAKE targets (Softmax rows, GELU and Logistic vectors).

This module draws random numbers and rounds them to the I/O format; it holds
none of the method's arithmetic. Both the HIP path and the CPU oracle receive
exactly the tensors produced here.

Workloads (name -> operator, I/O format, shape, distribution):
  softmax_f32_64x128        softmax, f32, [64,128], 4*N(0,1), t = 1
  gelu_bf16_4096x3072       GELU, bf16, [4096,3072] (BERT-base MLP width), N(0, 1.5^2)
  attn_softmax_bf16_causal  softmax, bf16, [8,12,512,512] viewed as 49152 rows of
                            512, N(0,1) scores with -inf at column j > row i of
                            each 512x512 block, t = 1/8 (= 1/sqrt(64))
  sigmoid_f16_2p28          Logistic and SiLU, f16, 2^28 elements, U[-12,12] with
                            Bernoulli(0.01) positions set to +-80 (sign p = 1/2)
  lmhead_softmax_f32_64x128256  softmax, f32, [64,128256], 3*N(0,1) with 16
                            distinct random columns per row set to +20
and the two op-level shapes of the fusion study (TABLE4_WORKLOADS):
  softmax_f32_16384x16384   softmax, f32, [16384,16384], 4*N(0,1), t = 1
  gelu_f32_260k             GELU, f32, [260000], N(0, 1.5^2)

Every generator is numpy PCG64 seeded with SEED_BASE + k, so a given call is
reproducible across machines. `rows`/`n` arguments shrink a workload to a
prefix of the same distribution (used for oracle-sized parity cases).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

SEED_BASE = 2412_00408

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
ELEM_BYTES = {"f32": 4, "f16": 2, "bf16": 2}


def rng(k: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(SEED_BASE + k))


def to_format(v: np.ndarray, dt: str) -> torch.Tensor:
    """float32 numpy values -> CPU tensor of format dt (round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32))
    return t.to(TORCH_DT[dt])


def bits(t: torch.Tensor) -> np.ndarray:
    """Raw element bits of a CPU tensor as numpy (float32, or uint16 for 16-bit)."""
    t = t.contiguous()
    if t.dtype == torch.float32:
        return t.numpy()
    return t.view(torch.int16).numpy().view(np.uint16)


def from_bits(a: np.ndarray, dt: str) -> torch.Tensor:
    if dt == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(TORCH_DT[dt])


# --------------------------------------------------------------------------
# Distribution building blocks
# --------------------------------------------------------------------------

def normal(shape, std: float, dt: str, k: int) -> torch.Tensor:
    v = rng(k).standard_normal(shape, dtype=np.float32) * np.float32(std)
    return to_format(v, dt)


def uniform(shape, lo: float, hi: float, dt: str, k: int) -> torch.Tensor:
    r = rng(k)
    v = r.random(shape, dtype=np.float32) * np.float32(hi - lo) + np.float32(lo)
    return to_format(v, dt)


def uniform_with_outliers(n: int, lo: float, hi: float, p: float, mag: float, dt: str,
                          k: int) -> torch.Tensor:
    r = rng(k)
    v = r.random(n, dtype=np.float32) * np.float32(hi - lo) + np.float32(lo)
    hit = r.random(n, dtype=np.float32) < np.float32(p)
    sign = np.where(r.random(n, dtype=np.float32) < 0.5, np.float32(-mag), np.float32(mag))
    v[hit] = sign[hit]
    return to_format(v, dt)


def causal_scores(batch_heads: int, seq: int, dt: str, k: int, rows: int | None = None) -> torch.Tensor:
    """N(0,1) scores of shape [batch_heads*seq, seq], -inf where column > row."""
    total = batch_heads * seq
    rows = total if rows is None else rows
    v = rng(k).standard_normal((rows, seq), dtype=np.float32)
    i = (np.arange(rows) % seq)[:, None]
    j = np.arange(seq)[None, :]
    v[j > i] = -np.inf
    return to_format(v, dt)


def spiked_logits(rows: int, cols: int, std: float, spikes: int, spike_val: float, dt: str,
                  k: int) -> torch.Tensor:
    r = rng(k)
    v = r.standard_normal((rows, cols), dtype=np.float32) * np.float32(std)
    for i in range(rows):
        cj = r.choice(cols, size=spikes, replace=False)
        v[i, cj] = np.float32(spike_val)
    return to_format(v, dt)


def attention_inputs(heads: int, seq: int, k: int, dim: int = 64, ldv: int | None = None,
                     pad: float = 0.0, heads_total: int | None = None, dt: str = "bf16"):
    """q, k [heads, seq, dim] and v transposed, vt [heads, dim, ldv], all in
    16-bit format dt with N(0,1) entries (so with t = 1/sqrt(dim) the scaled
    scores are about N(0,1)); vt's columns seq .. ldv-1 are set to `pad`.
    `heads` may be a prefix of `heads_total` heads drawn by the same generator."""
    ldv = seq if ldv is None else ldv
    total = heads if heads_total is None else heads_total
    r = rng(k)
    q = r.standard_normal((total, seq, dim), dtype=np.float32)[:heads]
    kk = r.standard_normal((total, seq, dim), dtype=np.float32)[:heads]
    v = r.standard_normal((total, dim, seq), dtype=np.float32)[:heads]
    vt = np.full((heads, dim, ldv), np.float32(pad), np.float32)
    vt[:, :, :seq] = v
    return to_format(q, dt), to_format(kk, dt), to_format(vt, dt)


# --------------------------------------------------------------------------
# The five workloads
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class Workload:
    name: str
    op: str              # "softmax" | "gelu" | "sigmoid" | "silu"
    dt: str              # "f32" | "f16" | "bf16"
    shape: tuple         # full logical shape
    rows: int            # softmax rows (0 for elementwise)
    cols: int            # softmax row length (0 for elementwise)
    t: float = 1.0       # softmax temperature
    seed: int = 0

    @property
    def numel(self) -> int:
        n = 1
        for s in self.shape:
            n *= s
        return n

    @property
    def algo_bytes(self) -> int:
        """Each input element read once and each output element written once."""
        return 2 * ELEM_BYTES[self.dt] * self.numel

    def make(self, rows: int | None = None, n: int | None = None) -> torch.Tensor:
        """CPU tensor of inputs; softmax workloads are 2-D [rows, cols]."""
        if self.name == "softmax_f32_64x128":
            r = self.rows if rows is None else rows
            return normal((r, self.cols), 4.0, self.dt, self.seed)
        if self.name == "gelu_bf16_4096x3072":
            m = self.numel if n is None else n
            return normal((m,), 1.5, self.dt, self.seed)
        if self.name == "attn_softmax_bf16_causal":
            return causal_scores(self.shape[0] * self.shape[1], self.cols, self.dt, self.seed,
                                 rows=rows)
        if self.name in ("sigmoid_f16_2p28", "silu_f16_2p28", "exp_f16_2p28"):
            m = self.numel if n is None else n
            return uniform_with_outliers(m, -12.0, 12.0, 0.01, 80.0, self.dt, self.seed)
        if self.name == "lmhead_softmax_f32_64x128256":
            r = self.rows if rows is None else rows
            return spiked_logits(r, self.cols, 3.0, 16, 20.0, self.dt, self.seed)
        if self.name == "softmax_f32_16384x16384":
            r = self.rows if rows is None else rows
            return normal((r, self.cols), 4.0, self.dt, self.seed)
        if self.name == "gelu_f32_260k":
            m = self.numel if n is None else n
            return normal((m,), 1.5, self.dt, self.seed)
        raise KeyError(self.name)


# The op-level shapes of the paper's fusion study (Sec. V-A, Table IV): a
# row softmax of a 16384 x 16384 matrix and GELU of a 260k-element vector, both
# binary32 (values 4*N(0,1) and N(0, 1.5^2)).
TABLE4_WORKLOADS = {
    w.name: w for w in [
        Workload("softmax_f32_16384x16384", "softmax", "f32", (16384, 16384), 16384, 16384, 1.0, 6),
        Workload("gelu_f32_260k", "gelu", "f32", (260000,), 0, 0, 1.0, 7),
    ]
}

# The exponential alone on the Logistic input (e^x in the binary32 path against
# the construction in binary16's own layout, quake_exp16).
EXTRA_WORKLOADS = {
    w.name: w for w in [
        Workload("exp_f16_2p28", "exp", "f16", (1 << 28,), 0, 0, 1.0, 4),
    ]
}

WORKLOADS = {
    w.name: w for w in [
        Workload("softmax_f32_64x128", "softmax", "f32", (64, 128), 64, 128, 1.0, 1),
        Workload("gelu_bf16_4096x3072", "gelu", "bf16", (4096, 3072), 0, 0, 1.0, 2),
        Workload("attn_softmax_bf16_causal", "softmax", "bf16", (8, 12, 512, 512),
                 8 * 12 * 512, 512, 0.125, 3),
        Workload("sigmoid_f16_2p28", "sigmoid", "f16", (1 << 28,), 0, 0, 1.0, 4),
        Workload("silu_f16_2p28", "silu", "f16", (1 << 28,), 0, 0, 1.0, 4),
        Workload("lmhead_softmax_f32_64x128256", "softmax", "f32", (64, 128256), 64, 128256,
                 1.0, 5),
    ]
}
