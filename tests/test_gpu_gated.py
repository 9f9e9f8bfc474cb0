"""Gated entry points on the GPU: gate activation inside the kernels.

gdn_prefill_gated / gdn_decode_gated form g = -exp(A_log) softplus(a +
dt_bias) and beta = sigmoid(b) in fp32 inside the kernels (paper, Section
3.2). They are compared with the fp64 oracle run on the same raw inputs (bars
as for the plain entry points), and with the plain entry points fed g and beta
from the oracle's gate rounded to fp32 (agreement to fp32 rounding of the
gates).
"""
import numpy as np
import pytest
import torch

import oracle
from _helpers import O_BAR, chunked_bars, gates_from_raw, rel_l2, require_gpu, to_dev
from paper_2607_16831_amd import gdn, synth

pytestmark = pytest.mark.gpu


def _log(name, **errs):
    print("[parity] %s %s" % (name, " ".join("%s=%.3e" % kv for kv in errs.items())),
          flush=True)


def _prefill_case(dtype, d, chunk, lengths, seed):
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=lengths, n_seqs=len(lengths), hqk=2,
                                 hv=4, d=d, chunk=chunk, dtype=dtype, state_std=0.1,
                                 raw_gate=True, seed=seed)
    return synth.make(w)


@pytest.mark.parametrize("dtype,d,chunk", [("bf16", 128, 64), ("bf16", 64, 32), ("f32", 32, 16)])
def test_prefill_gated_vs_oracle(dtype, d, chunk):
    dev = require_gpu()
    x = _prefill_case(dtype, d, chunk, (150, 0, 64, 33, 257), 31)
    dd = to_dev(x, dev)
    o, sT = gdn.prefill_gated(dd["q"], dd["k"], dd["v"], dd["a"], dd["b"], dd["A_log"],
                              dd["dt_bias"], dd["cu_seqlens"],
                              initial_state=dd["initial_state"], chunk=chunk)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.prefill_gated(x["q"], x["k"], x["v"], x["a"], x["b"], x["A_log"],
                                        x["dt_bias"], x["cu_seqlens"], x["initial_state"])
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(sT.cpu(), s_ref)
    _log("prefill_gated_%s_d%d_C%d" % (dtype, d, chunk), o=eo, state=es)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    ob, sb = chunked_bars(dtype)
    assert eo <= ob and es <= sb


def test_prefill_gated_matches_plain():
    dev = require_gpu()
    x = _prefill_case("bf16", 128, 64, (300, 77), 32)
    dd = to_dev(x, dev)
    o1, s1 = gdn.prefill_gated(dd["q"], dd["k"], dd["v"], dd["a"], dd["b"], dd["A_log"],
                               dd["dt_bias"], dd["cu_seqlens"],
                               initial_state=dd["initial_state"], chunk=64)
    g, beta = (t.to(dev) for t in gates_from_raw(x))
    o2, s2 = gdn.prefill(dd["q"], dd["k"], dd["v"], g, beta, dd["cu_seqlens"],
                         initial_state=dd["initial_state"], chunk=64)
    torch.cuda.synchronize()
    eo, es = rel_l2(o1, o2), rel_l2(s1, s2)
    _log("prefill_gated_vs_plain", o=eo, state=es)
    # the two differ only by fp32 rounding of the gates (and its propagation
    # through the bf16 products)
    assert eo <= 2e-3 and es <= 2e-4


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_decode_gated_vs_oracle(dtype):
    dev = require_gpu()
    w = synth.DECODE_B64.replace(n_seqs=8, dtype=dtype, raw_gate=True, seed=33)
    x = synth.make(w)
    dd = to_dev(x, dev)
    state = dd["initial_state"].clone()
    o = gdn.decode_gated(dd["q"], dd["k"], dd["v"], dd["a"], dd["b"], dd["A_log"],
                         dd["dt_bias"], state)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.decode_gated(x["q"], x["k"], x["v"], x["a"], x["b"], x["A_log"],
                                       x["dt_bias"], x["initial_state"])
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(state.cpu(), s_ref)
    _log("decode_gated_%s" % dtype, o=eo, state=es)
    assert eo <= (O_BAR if dtype == "bf16" else 1e-5) and es <= 1e-5
    # and equal to the plain step on host-formed gates, to fp32 rounding
    state2 = dd["initial_state"].clone()
    g, beta = (t.to(dev) for t in gates_from_raw(x))
    o2 = gdn.decode(dd["q"], dd["k"], dd["v"], g, beta, state2)
    torch.cuda.synchronize()
    assert rel_l2(state, state2) <= 1e-6
    assert rel_l2(o.float(), o2.float()) <= (8e-3 if dtype == "bf16" else 1e-6)
