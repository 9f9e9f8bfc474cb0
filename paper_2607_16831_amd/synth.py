"""Seeded synthetic inputs for the Gated DeltaNet prefill and decode paths.

This module is shared by the tests, the benchmark and the smoke check, and it
feeds both the HIP library and the CPU oracle. It holds only input
distributions -- no step of the recurrence itself.

Distributions (the paper publishes no workloads, so these stand in for the
contest's 54 decode and 100 prefill workloads):

* q, k ~ N(0, 1), L2-normalised per (token, head); q is further scaled by
  1/sqrt(d_k) (the recurrence itself has no scale).
* v ~ N(0, 1).
* g = -softplus(N(mu, 1)) is the log of the per-token decay, alpha = exp(g);
  mu = 0 gives a mean alpha of 0.50, mu = 1 (strong decay) 0.30, mu = -4 a weak
  decay (alpha ~ 0.98) that keeps the state carry visible in the outputs.
* beta = sigmoid(N(0, 1)).
* initial states ~ N(0, 0.1^2) where present.
* raw gate inputs (workloads with raw_gate): a, b ~ N(0, 1) per (token, head),
  A_log = log(A) with A ~ U(1, 16) per head, and dt_bias the inverse softplus
  of dt = exp(U(log 0.001, log 0.1)) per head -- the usual initialisation of
  these parameters in gated linear-attention layers. Such a workload carries
  no g and beta: the gate activation is part of the method, so only its
  implementations form them (the kernels, and the oracle's gate for the
  tests).
* q, k, v are produced in fp32 and rounded to bf16 (round to nearest even)
  when the workload is bf16; g, beta and states stay fp32.

One seeded torch CPU generator per workload (deterministic for a given seed
and torch build); draw order: sequence lengths, q, k, v, g noise, beta noise,
initial state, then (raw_gate only) a, b, A, dt. Arithmetic on the draws is
fp32.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    kind: str                       # "prefill" or "decode"
    n_seqs: int                     # sequences (prefill) or batch (decode)
    hqk: int
    hv: int
    d: int                          # d_k = d_v
    chunk: int = 64
    dtype: str = "bf16"             # element type of q, k, v, o
    seq_len: Optional[int] = None   # fixed length per sequence
    len_range: Optional[Tuple[int, int]] = None  # inclusive range, drawn
    lengths: Optional[Tuple[int, ...]] = None    # explicit lengths
    g_mu: float = 0.0
    g_zero: bool = False            # alpha = 1 exactly
    g_scale: float = 1.0            # multiplies g (stress: very strong decay)
    state_std: float = 0.0          # 0 -> no initial state
    raw_gate: bool = False          # also draw a, b, A_log, dt_bias
    seed: int = 1000

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads of the study, by what they are.
PREFILL_TINY = Workload("prefill_tiny_T64_d32_f32", "prefill", n_seqs=1, hqk=1,
                        hv=1, d=32, chunk=16, dtype="f32", seq_len=64,
                        seed=1000)
DECODE_B64 = Workload("decode_B64_hqk16_hv32_d128", "decode", n_seqs=64,
                      hqk=16, hv=32, d=128, state_std=0.1, seed=1001)
PREFILL_4K = Workload("prefill_T4096_hqk16_hv32_d128_C64", "prefill", n_seqs=1,
                      hqk=16, hv=32, d=128, chunk=64, seq_len=4096, seed=1002)
PREFILL_VARLEN = Workload("prefill_varlen16_U64-8192_hqk16_hv32_d128_C64",
                          "prefill", n_seqs=16, hqk=16, hv=32, d=128, chunk=64,
                          len_range=(64, 8192), state_std=0.1, seed=1003)
PREFILL_LONG = Workload("prefill_2x32768_strongdecay_hqk16_hv32_d128_C64",
                        "prefill", n_seqs=2, hqk=16, hv=32, d=128, chunk=64,
                        seq_len=32768, g_mu=1.0, seed=1004)

WORKLOADS = {w.name: w for w in
             (PREFILL_TINY, DECODE_B64, PREFILL_4K, PREFILL_VARLEN,
              PREFILL_LONG)}


def _unit_rows(x: torch.Tensor) -> torch.Tensor:
    return x / torch.linalg.vector_norm(x, dim=-1, keepdim=True).clamp_min(1e-30)


def _cast(x: torch.Tensor, dtype: str) -> torch.Tensor:
    x = x.contiguous()
    return x.to(torch.bfloat16) if dtype == "bf16" else x


def seq_lengths(w: Workload, gen: Optional[torch.Generator] = None):
    if w.lengths is not None:
        return np.asarray(w.lengths, dtype=np.int64)
    if w.seq_len is not None:
        return np.full(w.n_seqs, w.seq_len, dtype=np.int64)
    if w.len_range is not None:
        assert gen is not None
        lo, hi = w.len_range
        return torch.randint(lo, hi + 1, (w.n_seqs,), generator=gen).numpy().astype(np.int64)
    if w.kind == "decode":
        return np.ones(w.n_seqs, dtype=np.int64)
    raise ValueError("workload %s has no length rule" % w.name)


def make(w: Workload, seed: Optional[int] = None) -> dict:
    """Draw one input set for workload ``w`` as CPU torch tensors.

    Returns a dict with q, k, v (bf16 or f32), g, beta (f32), cu_seqlens
    (int32), initial_state (f32 or None; for decode the state that is
    advanced in place) and the workload itself under "w". With w.raw_gate it
    holds a, b [T, HV] and A_log, dt_bias [HV] (f32) instead, and g, beta
    are None.
    """
    gen = torch.Generator().manual_seed(w.seed if seed is None else seed)
    lens = seq_lengths(w, gen)
    T = int(lens.sum())
    d = w.d
    q = _unit_rows(torch.randn((T, w.hqk, d), generator=gen)) / float(np.sqrt(d))
    k = _unit_rows(torch.randn((T, w.hqk, d), generator=gen))
    v = torch.randn((T, w.hv, d), generator=gen)
    gz = torch.randn((T, w.hv), generator=gen)
    bz = torch.randn((T, w.hv), generator=gen)
    if w.g_zero:
        g = torch.zeros((T, w.hv))
    else:
        g = -w.g_scale * torch.nn.functional.softplus(gz + w.g_mu)
    beta = torch.sigmoid(bz)
    s0 = None
    if w.state_std > 0:
        s0 = w.state_std * torch.randn((w.n_seqs, w.hv, d, d), generator=gen)
    elif w.kind == "decode":
        s0 = torch.zeros((w.n_seqs, w.hv, d, d))
    cu = np.zeros(w.n_seqs + 1, dtype=np.int32)
    cu[1:] = np.cumsum(lens)
    out = dict(w=w, q=_cast(q, w.dtype), k=_cast(k, w.dtype), v=_cast(v, w.dtype),
               initial_state=s0, cu_seqlens=torch.from_numpy(cu))
    if w.raw_gate:
        a = torch.randn((T, w.hv), generator=gen)
        b = torch.randn((T, w.hv), generator=gen)
        A = 1.0 + 15.0 * torch.rand((w.hv,), generator=gen)
        dt = torch.exp(np.log(1e-3) + (np.log(1e-1) - np.log(1e-3)) *
                       torch.rand((w.hv,), generator=gen))
        dt_bias = dt + torch.log(-torch.expm1(-dt))  # softplus(dt_bias) = dt
        out.update(a=a.contiguous(), b=b.contiguous(), A_log=torch.log(A).contiguous(),
                   dt_bias=dt_bias.contiguous(), g=None, beta=None)
        return out
    out.update(g=g.float().contiguous(), beta=beta.float().contiguous())
    return out
