"""Prefill shape dispatch on the GPU: the token-serial path, chunk = 0 and the
Neumann-product chunk solve.

chunk = 1 runs the token-serial kernel (the recurrence token by token in fp32,
state in registers). Its arithmetic is the definition itself in fp32, so it is
held to fp32-level bars against the fp64 oracle: state rel-L2 <= 2e-5, o <=
1e-5 for fp32 outputs and <= 4e-3 for bf16 outputs (the bf16 rounding of o is
at most 2^-8 relative per element). chunk = 0 must run exactly what
gdn_prefill_auto_chunk reports (bitwise equal results: every path is
deterministic) and meet the oracle bars of that path. chunk | CHUNK_NEUMANN
meets the chunked path's bars (o 2e-2, state 5e-3).
"""
import numpy as np
import pytest
import torch

import oracle
from _helpers import O_BAR, STATE_BAR, chain_slice, chunked_bars, rel_l2, require_gpu, to_dev
from paper_2607_16831_amd import gdn, synth

pytestmark = pytest.mark.gpu

SERIAL_STATE_BAR = 2e-5


def _log(name, **errs):
    print("[parity] %s %s" % (name, " ".join("%s=%.3e" % kv for kv in errs.items())),
          flush=True)


def _o_bar(dtype):
    return 4e-3 if dtype == "bf16" else 1e-5


def _case(lengths, hqk=2, hv=4, d=128, dtype="bf16", state_std=0.1, g_mu=0.0,
          raw_gate=False, seed=70):
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=tuple(lengths), n_seqs=len(lengths),
                                 hqk=hqk, hv=hv, d=d, dtype=dtype, state_std=state_std,
                                 g_mu=g_mu, raw_gate=raw_gate, seed=seed)
    return synth.make(w)


def _run(x, dev, chunk, alias=False):
    d = to_dev(x, dev)
    s0 = d["initial_state"]
    fs = s0.clone() if (alias and s0 is not None) else None
    o, sT = gdn.prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["cu_seqlens"],
                        initial_state=fs if alias else s0, chunk=chunk, final_state=fs)
    torch.cuda.synchronize()
    return o.cpu(), sT.cpu()


def _oracle(x):
    return oracle.prefill(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu_seqlens"],
                          x["initial_state"])


# ------------------------------------------------------------ token-serial
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_serial_shapes(d, dtype):
    """Ragged lengths across the 4-token prefetch blocks, an empty sequence,
    grouped heads and a nonzero initial state."""
    dev = require_gpu()
    x = _case((1, 2, 3, 4, 5, 0, 9, 17, 33), d=d, dtype=dtype, g_mu=-4.0, seed=71 + d)
    o, sT = _run(x, dev, gdn.CHUNK_SERIAL)
    o_ref, s_ref = _oracle(x)
    eo, es = rel_l2(o, o_ref), rel_l2(sT, s_ref)
    _log("serial_d%d_%s" % (d, dtype), o=eo, state=es)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    assert eo <= _o_bar(dtype) and es <= SERIAL_STATE_BAR


def test_serial_long_sequence():
    """A sequence of hundreds of tokens through the token loop (weak decay so
    early tokens still matter at the end)."""
    dev = require_gpu()
    x = _case((301, 64), g_mu=-4.0, seed=75)
    o, sT = _run(x, dev, gdn.CHUNK_SERIAL)
    o_ref, s_ref = _oracle(x)
    eo, es = rel_l2(o, o_ref), rel_l2(sT, s_ref)
    _log("serial_long", o=eo, state=es)
    assert eo <= _o_bar("bf16") and es <= SERIAL_STATE_BAR


@pytest.mark.parametrize("n_seqs", [2, 64])
def test_serial_launch_shapes(n_seqs):
    """The benchmark's heads and head size with few sequences (two passes per
    wavefront) and many (four passes), no initial state."""
    dev = require_gpu()
    rng = np.random.default_rng(n_seqs)
    lengths = tuple(int(v) for v in rng.integers(1, 9, n_seqs))
    x = _case(lengths, hqk=16, hv=32, d=128, state_std=0.0, seed=76)
    o, sT = _run(x, dev, gdn.CHUNK_SERIAL)
    o_ref, s_ref = _oracle(x)
    eo, es = rel_l2(o, o_ref), rel_l2(sT, s_ref)
    _log("serial_N%d_hqk16_hv32" % n_seqs, o=eo, state=es)
    assert eo <= _o_bar("bf16") and es <= SERIAL_STATE_BAR


@pytest.mark.parametrize("n_seqs", [3, 256])
def test_serial_one_token(n_seqs):
    """One token per sequence (one-token prefetch) with an initial state."""
    dev = require_gpu()
    x = _case((1,) * n_seqs, hqk=16, hv=32, d=128, seed=86)
    o, sT = _run(x, dev, gdn.CHUNK_SERIAL)
    o_ref, s_ref = _oracle(x)
    eo, es = rel_l2(o, o_ref), rel_l2(sT, s_ref)
    _log("serial_one_token_N%d" % n_seqs, o=eo, state=es)
    assert eo <= _o_bar("bf16") and es <= SERIAL_STATE_BAR


def _sampled_chains(name, x, o, sT, chains):
    cu = x["cu_seqlens"].numpy()
    worst_o = worst_s = 0.0
    for n, h in chains:
        o_ref, s_ref = oracle.prefill(**chain_slice(x, n, h))
        worst_o = max(worst_o, rel_l2(o[cu[n]:cu[n + 1], h], o_ref[:, 0]))
        worst_s = max(worst_s, rel_l2(sT[n, h], s_ref[0, 0]))
    _log(name, o_max=worst_o, state_max=worst_s, chains=len(chains))
    assert worst_o <= _o_bar("bf16") and worst_s <= SERIAL_STATE_BAR


def test_serial_many_one_token_sequences():
    """4096 one-token sequences at the benchmark's heads: one-token prefetch
    and eight passes per wavefront. From a zero state one token gives
    S = beta v k^T and o = beta v (k . q) exactly; that closed form is checked
    for every (sequence, head), the oracle on sampled chains."""
    dev = require_gpu()
    n_seqs = 4096
    x = _case((1,) * n_seqs, hqk=16, hv=32, d=128, state_std=0.0, seed=87)
    o, sT = _run(x, dev, gdn.CHUNK_SERIAL)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    grp = 2
    k = x["k"].double().numpy()[:, np.repeat(np.arange(16), grp)]      # [N, 32, d]
    q = x["q"].double().numpy()[:, np.repeat(np.arange(16), grp)]
    v = x["v"].double().numpy()
    b = x["beta"].double().numpy()
    worst_s = worst_o = 0.0
    for n0 in range(0, n_seqs, 256):
        sl = slice(n0, n0 + 256)
        s_ref = b[sl, :, None, None] * v[sl, :, :, None] * k[sl, :, None, :]
        o_ref = b[sl, :, None] * v[sl] * np.sum(k[sl] * q[sl], axis=-1)[..., None]
        worst_s = max(worst_s, rel_l2(sT[sl], s_ref))
        worst_o = max(worst_o, rel_l2(o[sl], o_ref))
    _log("serial_4096x1_closed_form", o_max=worst_o, state_max=worst_s)
    assert worst_o <= _o_bar("bf16") and worst_s <= SERIAL_STATE_BAR
    _sampled_chains("serial_4096x1", x, o, sT, [(n, h) for n in (0, 1777, 4095) for h in (0, 31)])


def test_serial_many_short_sequences_with_state():
    """2048 sequences of 1-3 tokens with initial states: four-token prefetch
    and eight passes per wavefront, oracle on sampled chains."""
    dev = require_gpu()
    rng = np.random.default_rng(88)
    lengths = tuple(int(v) for v in rng.integers(1, 4, 2048))
    x = _case(lengths, hqk=16, hv=32, d=128, seed=88)
    o, sT = _run(x, dev, gdn.CHUNK_SERIAL)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    _sampled_chains("serial_2048x1-3", x, o, sT,
                    [(n, h) for n in (0, 1000, 2047) for h in (0, 7, 31)])


def test_serial_alias_in_place():
    dev = require_gpu()
    x = _case((7, 12, 1), seed=77)
    o1, s1 = _run(x, dev, gdn.CHUNK_SERIAL, alias=False)
    o2, s2 = _run(x, dev, gdn.CHUNK_SERIAL, alias=True)
    assert torch.equal(o1, o2) and torch.equal(s1, s2)


def test_serial_all_empty():
    dev = require_gpu()
    x = _case((0, 0, 0), seed=78)
    o, sT = _run(x, dev, gdn.CHUNK_SERIAL)
    assert o.numel() == 0
    assert torch.equal(sT, x["initial_state"])
    x0 = _case((0, 0), state_std=0.0, seed=79)
    o, sT = _run(x0, dev, gdn.CHUNK_SERIAL)
    assert torch.count_nonzero(sT) == 0


def test_serial_equals_decode_steps():
    """One token per sequence: the token-serial prefill is the decode step."""
    dev = require_gpu()
    x = _case((1,) * 6, hqk=4, hv=8, seed=80)
    o, sT = _run(x, dev, gdn.CHUNK_SERIAL)
    d = to_dev(x, dev)
    state = d["initial_state"].clone()
    od = gdn.decode(d["q"], d["k"], d["v"], d["g"], d["beta"], state)
    torch.cuda.synchronize()
    eo, es = rel_l2(o, od.cpu()), rel_l2(sT, state.cpu())
    _log("serial_vs_decode", o=eo, state=es)
    assert eo <= 4e-3 and es <= 1e-6


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_serial_gated(dtype):
    dev = require_gpu()
    x = _case((5, 0, 13, 2), d=64, dtype=dtype, raw_gate=True, seed=81)
    dd = to_dev(x, dev)
    o, sT = gdn.prefill_gated(dd["q"], dd["k"], dd["v"], dd["a"], dd["b"], dd["A_log"],
                              dd["dt_bias"], dd["cu_seqlens"],
                              initial_state=dd["initial_state"], chunk=gdn.CHUNK_SERIAL)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.prefill_gated(x["q"], x["k"], x["v"], x["a"], x["b"], x["A_log"],
                                        x["dt_bias"], x["cu_seqlens"], x["initial_state"])
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(sT.cpu(), s_ref)
    _log("serial_gated_%s" % dtype, o=eo, state=es)
    assert eo <= _o_bar(dtype) and es <= 1e-4


def _gated_chain(x, n, h):
    """Inputs of one (sequence, value head) chain of a raw-gate problem."""
    c = chain_slice(x, n, h)
    cu = x["cu_seqlens"].numpy()
    t0, t1 = int(cu[n]), int(cu[n + 1])
    return dict(q=c["q"], k=c["k"], v=c["v"], a=x["a"][t0:t1, h:h + 1],
                b=x["b"][t0:t1, h:h + 1], a_log=x["A_log"][h:h + 1],
                dt_bias=x["dt_bias"][h:h + 1], cu_seqlens=c["cu_seqlens"],
                initial_state=c["initial_state"])


@pytest.mark.parametrize("n_seqs,lengths", [(5, "ones"), (4096, "ones"), (2048, "1-3")])
def test_serial_gated_launch_paths(n_seqs, lengths):
    """Raw gates on the one-token prefetch path (5 and 4096 sequences of one
    token) and on eight passes per wavefront (4096 x 1, 2048 x 1-3)."""
    dev = require_gpu()
    if lengths == "ones":
        lens = (1,) * n_seqs
    else:
        lens = tuple(int(v) for v in np.random.default_rng(89).integers(1, 4, n_seqs))
    x = _case(lens, hqk=16, hv=32, d=128, raw_gate=True, state_std=0.1 if n_seqs < 100 else 0.0,
              seed=89 + n_seqs)
    dd = to_dev(x, dev)
    o, sT = gdn.prefill_gated(dd["q"], dd["k"], dd["v"], dd["a"], dd["b"], dd["A_log"],
                              dd["dt_bias"], dd["cu_seqlens"],
                              initial_state=dd["initial_state"], chunk=gdn.CHUNK_SERIAL)
    torch.cuda.synchronize()
    o, sT = o.cpu(), sT.cpu()
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    cu = x["cu_seqlens"].numpy()
    seqs = sorted({0, n_seqs // 2, n_seqs - 1})
    worst_o = worst_s = 0.0
    for n in seqs:
        for h in (0, 5, 31):
            o_ref, s_ref = oracle.prefill_gated(**_gated_chain(x, n, h))
            worst_o = max(worst_o, rel_l2(o[cu[n]:cu[n + 1], h], o_ref[:, 0]))
            worst_s = max(worst_s, rel_l2(sT[n, h], s_ref[0, 0]))
    _log("serial_gated_N%d_%s" % (n_seqs, lengths), o_max=worst_o, state_max=worst_s)
    assert worst_o <= _o_bar("bf16") and worst_s <= 1e-4


# ------------------------------------------------------------ chunk = 0
@pytest.mark.parametrize("n_seqs,length", [(256, 1), (256, 3), (64, 12), (48, 40), (8, 200), (2, 400),
                                           (16, 512)])
def test_auto_runs_the_reported_path(n_seqs, length):
    """chunk = 0 at the benchmark's heads: bitwise the path the library
    reports, and within that path's oracle bars."""
    dev = require_gpu()
    x = _case((length,) * n_seqs, hqk=16, hv=32, d=128, seed=82 + length)
    picked = gdn.prefill_auto_chunk(n_seqs, n_seqs * length, 16, 32, 128, 128)
    assert picked in (1, 16, 32, 64)
    o0, s0 = _run(x, dev, gdn.CHUNK_AUTO)
    o1, s1 = _run(x, dev, picked)
    assert torch.equal(o0, o1) and torch.equal(s0, s1)
    # oracle on sampled chains (sequence, value head)
    rng = np.random.default_rng(length)
    for n in rng.choice(n_seqs, size=min(n_seqs, 6), replace=False):
        h = int(rng.integers(0, 32))
        c = chain_slice(x, int(n), h)
        o_ref, s_ref = oracle.prefill(c["q"], c["k"], c["v"], c["g"], c["beta"],
                                      c["cu_seqlens"], c["initial_state"])
        cu = x["cu_seqlens"].numpy()
        t0, t1 = int(cu[n]), int(cu[n + 1])
        eo = rel_l2(o0[t0:t1, h:h + 1], o_ref)
        es = rel_l2(s0[n:n + 1, h:h + 1], s_ref)
        ob, sb = (_o_bar("bf16"), SERIAL_STATE_BAR) if picked == 1 else (O_BAR, STATE_BAR)
        assert eo <= ob and es <= sb, (n, h, eo, es)
    _log("auto_N%d_L%d_C%d" % (n_seqs, length, picked), o=eo, state=es)


# ------------------------------------------------------------ Neumann inverse
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("chunk", [16, 32, 64])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_neumann_shapes(d, chunk, dtype):
    """Diagonal blocks of the WY factor by the Neumann product: oracle bars of
    the chunked path, and close to the forward-substitution run (the two
    differ only in the fp32 rounding of the inverse before its bf16 rounding)."""
    dev = require_gpu()
    x = _case((1, 63, 64, 65, 200, 0, 130, 17), d=d, dtype=dtype, g_mu=-4.0,
              seed=90 + d + chunk)
    o, sT = _run(x, dev, chunk | gdn.CHUNK_NEUMANN)
    o_ref, s_ref = _oracle(x)
    eo, es = rel_l2(o, o_ref), rel_l2(sT, s_ref)
    o2, s2 = _run(x, dev, chunk)
    do, ds = rel_l2(o, o2), rel_l2(sT, s2)
    _log("neumann_d%d_C%d_%s" % (d, chunk, dtype), o=eo, state=es, o_vs_fs=do, state_vs_fs=ds)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    ob, sb = chunked_bars(dtype)
    assert eo <= ob and es <= sb
    assert do <= 5e-3 and ds <= 2e-3


def test_neumann_prefill_4k_full():
    """The benchmark workload (4096 tokens, 16/32 heads, d = 128, C = 64)."""
    dev = require_gpu()
    x = synth.make(synth.PREFILL_4K)
    o, sT = _run(x, dev, 64 | gdn.CHUNK_NEUMANN)
    o_ref, s_ref = _oracle(x)
    eo, es = rel_l2(o, o_ref), rel_l2(sT, s_ref)
    _log("neumann_prefill_4k", o=eo, state=es)
    assert eo <= O_BAR and es <= STATE_BAR


def test_neumann_gated():
    dev = require_gpu()
    x = _case((150, 0, 64, 33), d=128, raw_gate=True, seed=95)
    dd = to_dev(x, dev)
    o, sT = gdn.prefill_gated(dd["q"], dd["k"], dd["v"], dd["a"], dd["b"], dd["A_log"],
                              dd["dt_bias"], dd["cu_seqlens"],
                              initial_state=dd["initial_state"], chunk=64 | gdn.CHUNK_NEUMANN)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.prefill_gated(x["q"], x["k"], x["v"], x["a"], x["b"], x["A_log"],
                                        x["dt_bias"], x["cu_seqlens"], x["initial_state"])
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(sT.cpu(), s_ref)
    _log("neumann_gated", o=eo, state=es)
    assert eo <= O_BAR and es <= STATE_BAR


# ------------------------------------------------------------ single-wave carry
def _short_lengths(C):
    """Ragged lengths whose average fits in one chunk (the single-wave carry
    runs), with an empty sequence and sequences of one, several and C tokens
    and one of more than two chunks."""
    return (1, 5, C, 2 * C + 3, 0, 7, 9, 11, 13, 2, C - 1, 3)


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("chunk", [16, 32, 64])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_wave_carry_shapes(d, chunk, dtype):
    dev = require_gpu()
    lengths = _short_lengths(chunk)
    assert sum(lengths) <= len(lengths) * chunk
    x = _case(lengths, d=d, dtype=dtype, g_mu=-4.0, seed=100 + d + chunk)
    o, sT = _run(x, dev, chunk)
    o_ref, s_ref = _oracle(x)
    eo, es = rel_l2(o, o_ref), rel_l2(sT, s_ref)
    _log("wave_carry_d%d_C%d_%s" % (d, chunk, dtype), o=eo, state=es)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    ob, sb = chunked_bars(dtype)  # (float32 inputs take the float32 form)
    assert eo <= ob and es <= sb


def test_wave_carry_benchmark_heads_no_state():
    """The benchmark's heads, 128 sequences of 16 tokens, zero initial state
    (the shape of the bench's short-sequence batch)."""
    dev = require_gpu()
    x = _case((16,) * 128, hqk=16, hv=32, d=128, state_std=0.0, seed=110)
    o, sT = _run(x, dev, 16)
    rng = np.random.default_rng(7)
    for n in rng.choice(128, size=6, replace=False):
        h = int(rng.integers(0, 32))
        c = chain_slice(x, int(n), h)
        o_ref, s_ref = oracle.prefill(c["q"], c["k"], c["v"], c["g"], c["beta"],
                                      c["cu_seqlens"], c["initial_state"])
        cu = x["cu_seqlens"].numpy()
        eo = rel_l2(o[int(cu[n]):int(cu[n + 1]), h:h + 1], o_ref)
        es = rel_l2(sT[n:n + 1, h:h + 1], s_ref)
        assert eo <= O_BAR and es <= STATE_BAR, (n, h, eo, es)
    _log("wave_carry_N128_L16", o=eo, state=es)


def test_wave_carry_alias_and_gated():
    dev = require_gpu()
    x = _case(_short_lengths(32), d=64, raw_gate=True, seed=111)
    dd = to_dev(x, dev)
    fs = dd["initial_state"].clone()
    o, sT = gdn.prefill_gated(dd["q"], dd["k"], dd["v"], dd["a"], dd["b"], dd["A_log"],
                              dd["dt_bias"], dd["cu_seqlens"], initial_state=fs, chunk=32,
                              final_state=fs)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.prefill_gated(x["q"], x["k"], x["v"], x["a"], x["b"], x["A_log"],
                                        x["dt_bias"], x["cu_seqlens"], x["initial_state"])
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(sT.cpu(), s_ref)
    _log("wave_carry_gated_in_place", o=eo, state=es)
    assert eo <= O_BAR and es <= STATE_BAR
