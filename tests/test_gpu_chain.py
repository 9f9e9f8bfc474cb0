"""The whole-chain carry over segments, against the fp64 oracle (needs a GPU).

A sequence longer than one segment (L chunks) runs in three launches: every
segment at once (segment 0 from the true initial state, the others from zero
for their B and from the identity for their map M), the composition
S_in(s + 1) = S_in(s) M_s + B_s, and the segments after the first from their
composed states. GDN_CHUNK_SEGMENT(L) forces small segments so that short
batches exercise every role: sequences of one, two and many segments, empty
sequences, partial last chunks and segments. Decay settings range from none
(g = 0, where the maps carry everything) to 40 times the long-context draw.
Every case asserts the whole-tensor and the per-chain bars.
"""
import numpy as np
import pytest
import torch

import oracle
from _helpers import O_BAR, STATE_BAR, chain_errors, require_gpu, to_dev
from paper_2607_16831_amd import gdn, synth

pytestmark = pytest.mark.gpu

LENS = (1000, 0, 65, 300, 777, 64, 1, 129)


def _run(x, dev, chunk, alias=False):
    d = to_dev(x, dev)
    s0 = d["initial_state"]
    fs = s0.clone() if (alias and s0 is not None) else None
    o, sT = gdn.prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["cu_seqlens"],
                        initial_state=fs if alias else s0, chunk=chunk, final_state=fs)
    torch.cuda.synchronize()
    return o.cpu(), sT.cpu()


def _check(name, x, dev, chunk, alias=False):
    o, sT = _run(x, dev, chunk, alias)
    o_ref, s_ref = oracle.prefill(x["q"], x["k"], x["v"], x["g"], x["beta"],
                                  x["cu_seqlens"], x["initial_state"])
    e = chain_errors(o, sT, o_ref, s_ref, x["cu_seqlens"].numpy())
    print("[chain] %s o=%.3e state=%.3e o_chain_max=%.3e state_chain_max=%.3e worst=%s"
          % (name, e["o"], e["state"], e["o_max"], e["state_max"], e["worst"]), flush=True)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    assert e["o"] <= O_BAR and e["state"] <= STATE_BAR
    assert e["o_max"] <= O_BAR and e["state_max"] <= STATE_BAR
    return o, sT


@pytest.mark.parametrize("chunk", [16, 32, 64])
@pytest.mark.parametrize("seg", [1, 2, 3])
@pytest.mark.parametrize("g_mu", [-4.0, 0.0])
def test_segments_ragged(chunk, seg, g_mu):
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=LENS, n_seqs=len(LENS), hqk=2, hv=4,
                                 g_mu=g_mu, state_std=0.1, seed=301)
    _check("ragged_C%d_L%d_mu%g" % (chunk, seg, g_mu), synth.make(w), dev,
           chunk | gdn.CHUNK_SEGMENT(seg))


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("chunk", [16, 32, 64])
def test_segments_head_sizes(d, chunk):
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=LENS, n_seqs=len(LENS), hqk=2, hv=4, d=d,
                                 g_mu=-4.0, state_std=0.1, seed=303)
    _check("heads_d%d_C%d" % (d, chunk), synth.make(w), dev, chunk | gdn.CHUNK_SEGMENT(2))


def test_segments_no_decay_many_maps():
    """g = 0: nothing decays, so every segment's map M carries the whole
    incoming state; 1000 tokens in one-chunk segments compose 14 maps."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=(1000, 130), n_seqs=2, hqk=1, hv=2,
                                 g_zero=True, state_std=0.1, seed=305)
    _check("no_decay_L1", synth.make(w), dev, 64 | gdn.CHUNK_SEGMENT(1))


def test_segments_strong_decay_stays_finite():
    dev = require_gpu()
    w = synth.PREFILL_LONG.replace(seq_len=None, lengths=(900, 77, 400), n_seqs=3, hqk=2, hv=4,
                                   g_scale=40.0, seed=307)
    _check("strong_decay_x40_L2", synth.make(w), dev, 64 | gdn.CHUNK_SEGMENT(2))


@pytest.mark.parametrize("seg", [1, 3])
def test_segments_in_place(seg):
    """final_state aliasing initial_state: the state is read by the first
    launch and written by the last."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=LENS, n_seqs=len(LENS), hqk=2, hv=4,
                                 g_mu=-3.0, state_std=0.1, seed=309)
    _check("in_place_L%d" % seg, synth.make(w), dev, 32 | gdn.CHUNK_SEGMENT(seg), alias=True)


@pytest.mark.parametrize("seg", [2, 4, 16, 64])
def test_segments_4k(seg):
    """The 4096-token workload (16/32 heads) with 32, 16, 4 and 1 segments."""
    dev = require_gpu()
    _check("4k_L%d" % seg, synth.make(synth.PREFILL_4K), dev, 64 | gdn.CHUNK_SEGMENT(seg))


def test_segments_gated():
    """Raw gate inputs (gates formed in the chunk-local kernel) with segments."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=(700, 5, 260), n_seqs=3, hqk=2, hv=4,
                                 state_std=0.1, raw_gate=True, seed=311)
    x = synth.make(w)
    d = to_dev(x, dev)
    o, sT = gdn.prefill_gated(d["q"], d["k"], d["v"], d["a"], d["b"], d["A_log"], d["dt_bias"],
                              d["cu_seqlens"], initial_state=d["initial_state"],
                              chunk=64 | gdn.CHUNK_SEGMENT(2))
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.prefill_gated(x["q"], x["k"], x["v"], x["a"], x["b"], x["A_log"],
                                        x["dt_bias"], x["cu_seqlens"], x["initial_state"])
    e = chain_errors(o.cpu(), sT.cpu(), o_ref, s_ref, x["cu_seqlens"].numpy())
    print("[chain] gated_L2 o=%.3e state=%.3e o_chain_max=%.3e state_chain_max=%.3e"
          % (e["o"], e["state"], e["o_max"], e["state_max"]), flush=True)
    assert e["o_max"] <= O_BAR and e["state_max"] <= STATE_BAR


def _check_prefilled(name, x, dev, chunk):
    """Outputs and final states start as NaN, so a segment that no work-group
    carries (a hole in the longest-first order) cannot pass on stale memory."""
    d = to_dev(x, dev)
    T, hv, dv = d["v"].shape
    n = len(x["cu_seqlens"]) - 1
    o = torch.full((T, hv, dv), float("nan"), dtype=d["v"].dtype, device=dev)
    fs = torch.full((n, hv, dv, d["k"].shape[2]), float("nan"), device=dev)
    gdn.prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["cu_seqlens"],
                initial_state=d["initial_state"], chunk=chunk, o=o, final_state=fs)
    torch.cuda.synchronize()
    o, sT = o.cpu(), fs.cpu()
    o_ref, s_ref = oracle.prefill(x["q"], x["k"], x["v"], x["g"], x["beta"],
                                  x["cu_seqlens"], x["initial_state"])
    e = chain_errors(o, sT, o_ref, s_ref, x["cu_seqlens"].numpy())
    print("[chain] %s o=%.3e state=%.3e o_chain_max=%.3e state_chain_max=%.3e worst=%s"
          % (name, e["o"], e["state"], e["o_max"], e["state_max"], e["worst"]), flush=True)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    assert e["o_max"] <= O_BAR and e["state_max"] <= STATE_BAR


@pytest.mark.parametrize("seg", [64, 2])
def test_longest_first_order_ragged(seg):
    """More than one sequence: the output launch takes its segments longest
    first from a list the library builds on the device. Lengths rising
    through the batch (the order is reversed), an empty sequence; seg = 64
    keeps every sequence in one segment, seg = 2 mixes two-chunk segments
    with shorter last ones."""
    dev = require_gpu()
    lens = (0, 1, 70, 130, 300, 511, 777, 1000, 1500)
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=lens, n_seqs=len(lens), hqk=2, hv=4,
                                 g_mu=-4.0, state_std=0.1, seed=313)
    _check_prefilled("order_L%d" % seg, synth.make(w), dev, 64 | gdn.CHUNK_SEGMENT(seg))


def test_longest_first_order_many_sequences():
    """1100 sequences (more than the ordering work-group's 1024 threads), one
    value head each: the whole-chain carry, every chain in the list once."""
    dev = require_gpu()
    rng = np.random.default_rng(317)
    lens = tuple(int(v) for v in rng.integers(65, 200, size=1100))
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=lens, n_seqs=len(lens), hqk=1, hv=1, d=32,
                                 g_mu=-4.0, state_std=0.1, seed=319)
    _check_prefilled("order_many", synth.make(w), dev, 64)


def test_longest_first_order_long_segments():
    """Segments of more than 960 chunks (C = 16), which the order ranks by
    power-of-two buckets, beside short ones."""
    dev = require_gpu()
    lens = (300, 15500, 40, 16000, 9000)
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=lens, n_seqs=len(lens), hqk=1, hv=1, d=32,
                                 g_mu=-4.0, state_std=0.1, seed=321)
    _check_prefilled("order_long_C16", synth.make(w), dev, 16 | gdn.CHUNK_SEGMENT(4095))
