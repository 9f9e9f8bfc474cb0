"""Seeded generator: determinism, shapes and the stated distributions."""
import numpy as np
import torch

from paper_2607_16831_amd import synth


def test_deterministic_and_shapes():
    w = synth.PREFILL_TINY
    a, b = synth.make(w), synth.make(w)
    for key in ("q", "k", "v", "g", "beta", "cu_seqlens"):
        assert torch.equal(a[key], b[key])
    assert a["q"].shape == (64, 1, 32) and a["q"].dtype == torch.float32
    assert a["initial_state"] is None
    c = synth.make(w, seed=5)
    assert not torch.equal(a["q"], c["q"])


def test_distributions():
    w = synth.PREFILL_TINY.replace(seq_len=4096, d=64, hv=2)
    x = synth.make(w)
    kn = x["k"].double().norm(dim=-1)
    qn = x["q"].double().norm(dim=-1)
    assert torch.allclose(kn, torch.ones_like(kn), atol=1e-6)
    assert torch.allclose(qn, torch.full_like(qn, 1 / 8), atol=1e-6)
    g, beta = x["g"].double(), x["beta"].double()
    assert (g < 0).all() and (beta > 0).all() and (beta < 1).all()
    assert abs(g.exp().mean().item() - 0.50) < 0.02          # mean alpha at mu=0
    strong = synth.make(w.replace(g_mu=1.0))["g"].double()
    assert abs(strong.exp().mean().item() - 0.30) < 0.02
    assert abs(beta.mean().item() - 0.5) < 0.02


def test_bf16_and_varlen():
    w = synth.PREFILL_VARLEN.replace(hqk=1, hv=2, d=8)
    x = synth.make(w)
    cu = x["cu_seqlens"].numpy()
    lens = np.diff(cu)
    assert len(lens) == 16 and lens.min() >= 64 and lens.max() <= 8192
    assert x["q"].dtype == torch.bfloat16 and x["g"].dtype == torch.float32
    assert x["initial_state"].shape == (16, 2, 8, 8)
    assert abs(x["initial_state"].std().item() - 0.1) < 0.01


def test_decode_workload():
    w = synth.DECODE_B64.replace(hqk=2, hv=4, d=16)
    x = synth.make(w)
    assert x["q"].shape == (64, 2, 16) and x["v"].shape == (64, 4, 16)
    assert x["g"].shape == (64, 4)
    assert x["initial_state"].shape == (64, 4, 16, 16)


def test_raw_gate_draws_leave_other_inputs_alone():
    w = synth.PREFILL_VARLEN.replace(hqk=1, hv=3, d=8, n_seqs=3)
    x, y = synth.make(w), synth.make(w.replace(raw_gate=True))
    for key in ("q", "k", "v", "cu_seqlens", "initial_state"):
        assert torch.equal(x[key], y[key]), key
    T = y["q"].shape[0]
    assert y["a"].shape == (T, 3) and y["b"].shape == (T, 3)
    assert y["A_log"].shape == (3,) and y["dt_bias"].shape == (3,)
    A = y["A_log"].exp()
    assert (A >= 1).all() and (A <= 16).all()
    dt = torch.nn.functional.softplus(y["dt_bias"].double())
    assert (dt >= 0.999e-3).all() and (dt <= 0.1001).all()
    # the gate activation is left to its implementations
    assert y["g"] is None and y["beta"] is None
