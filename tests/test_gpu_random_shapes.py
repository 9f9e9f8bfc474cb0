"""Seeded random configurations of the prefill and decode against the fp64 oracle.

Each case draws a head size, a GQA grouping, a ragged batch (empty
sequences included), a chunk setting (automatic, token-serial, 16/32/64,
the Neumann solve), the input dtype, whether an initial state is given and
the decay strength, so that combinations the fixed tests do not name are
exercised. Bars are those of the path that runs: the token-serial path is
fp32 arithmetic (state 2e-5; o 1e-5 in fp32, 4e-3 in bf16), the chunked
paths bf16 operands with fp32 accumulation (o 2e-2, state 5e-3)."""
import numpy as np
import pytest
import torch

import oracle
from _helpers import chain_errors, chunked_bars, rel_l2, require_gpu, to_dev
from paper_2607_16831_amd import gdn, synth

pytestmark = pytest.mark.gpu

HEADS = [(1, 1), (2, 4), (4, 4), (1, 4), (2, 2)]
CHUNKS = [gdn.CHUNK_AUTO, gdn.CHUNK_SERIAL, 16, 32, 64, 16 | gdn.CHUNK_NEUMANN,
          64 | gdn.CHUNK_NEUMANN]


def _draw(seed):
    rng = np.random.default_rng(1000 + seed)
    d = int(rng.choice([32, 64, 128]))
    hqk, hv = HEADS[int(rng.integers(len(HEADS)))]
    n = int(rng.integers(1, 7))
    lengths = [int(x) for x in rng.integers(0, 180, n)]
    if rng.random() < 0.3:
        lengths[int(rng.integers(n))] = 0
    chunk = int(CHUNKS[int(rng.integers(len(CHUNKS)))])
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    state_std = 0.1 if rng.random() < 0.6 else 0.0
    g_mu = float(rng.uniform(-4.0, 1.0))
    return d, hqk, hv, tuple(lengths), chunk, dtype, state_std, g_mu


@pytest.mark.parametrize("seed", range(16))
def test_random_configuration(seed):
    dev = require_gpu()
    d, hqk, hv, lengths, chunk, dtype, state_std, g_mu = _draw(seed)
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=lengths, n_seqs=len(lengths), hqk=hqk,
                                 hv=hv, d=d, dtype=dtype, state_std=state_std, g_mu=g_mu,
                                 seed=2000 + seed)
    x = synth.make(w)
    dd = to_dev(x, dev)
    o, sT = gdn.prefill(dd["q"], dd["k"], dd["v"], dd["g"], dd["beta"], dd["cu_seqlens"],
                        initial_state=dd["initial_state"], chunk=chunk)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.prefill(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu_seqlens"],
                                  x["initial_state"])
    o, sT = o.cpu(), sT.cpu()
    serial = chunk == gdn.CHUNK_SERIAL or (
        chunk == gdn.CHUNK_AUTO and
        gdn.prefill_auto_chunk(len(lengths), sum(lengths), hqk, hv, d, d) == gdn.CHUNK_SERIAL)
    e = chain_errors(o, sT, o_ref, s_ref, x["cu_seqlens"])
    eo = e["o"] if o.numel() else 0.0
    es = e["state"]
    print("[parity] random%d d=%d heads=%d/%d lengths=%s chunk=%#x %s S0=%s g_mu=%.2f "
          "o=%.3e state=%.3e o_chain_max=%.3e state_chain_max=%.3e worst=%s"
          % (seed, d, hqk, hv, lengths, chunk, dtype, state_std > 0, g_mu, eo, es,
             e["o_max"], e["state_max"], e["worst"]), flush=True)
    # whole tensor and every (sequence, value head) chain on its own
    if serial:
        ob, sb = (4e-3 if dtype == "bf16" else 1e-5), 2e-5
    else:
        ob, sb = chunked_bars(dtype)
    assert eo <= ob and es <= sb
    assert e["o_max"] <= ob and e["state_max"] <= sb


@pytest.mark.parametrize("seed", range(8))
def test_random_decode(seed):
    """One decode step at a random batch, head size, grouping and dtype, from
    g and beta or from the raw gate inputs (state updated in place)."""
    dev = require_gpu()
    rng = np.random.default_rng(3000 + seed)
    d = int(rng.choice([32, 64, 128]))
    hqk, hv = HEADS[int(rng.integers(len(HEADS)))]
    B = int(rng.integers(1, 97))
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    raw = bool(rng.random() < 0.5)
    w = synth.DECODE_B64.replace(n_seqs=B, hqk=hqk, hv=hv, d=d, dtype=dtype, raw_gate=raw,
                                 seed=4000 + seed)
    x = synth.make(w)
    dd = to_dev(x, dev)
    state = dd["initial_state"].clone()
    if raw:
        o = gdn.decode_gated(dd["q"], dd["k"], dd["v"], dd["a"], dd["b"], dd["A_log"],
                             dd["dt_bias"], state)
        o_ref, s_ref = oracle.decode_gated(x["q"], x["k"], x["v"], x["a"], x["b"], x["A_log"],
                                           x["dt_bias"], x["initial_state"])
    else:
        o = gdn.decode(dd["q"], dd["k"], dd["v"], dd["g"], dd["beta"], state)
        o_ref, s_ref = oracle.decode(x["q"], x["k"], x["v"], x["g"], x["beta"],
                                     x["initial_state"])
    torch.cuda.synchronize()
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(state.cpu(), s_ref)
    print("[parity] random_decode%d B=%d d=%d heads=%d/%d %s raw_gates=%s o=%.3e state=%.3e"
          % (seed, B, d, hqk, hv, dtype, raw, eo, es), flush=True)
    assert eo <= (4e-3 if dtype == "bf16" else 1e-5) and es <= 1e-5
