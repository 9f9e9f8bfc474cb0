"""Parity of the HIP library against the fp64 CPU oracle (needs a gfx950 GPU).

Bars (rel-L2 over the compared tensor, oracle as reference): o <= 2e-2 for the
bf16 outputs, final state <= 5e-3. Decode does all arithmetic in fp32, so its
state is additionally held to 1e-5 (a few fp32 ulps accumulated over d = 128
terms). Every case prints its measured errors.

Every prefill comparison asserts the whole-tensor rel-L2 AND the largest
rel-L2 over the (sequence, value head) chains, so that one wrong chain (or a
wrong partial chunk of one sequence) cannot hide in the average.

Full-size workloads: the 4096-token prefill, the batch-64 decode, the ~66K-token
varlen batch and the 2 x 32768 long-context batch are all compared whole; the
last two run whole on the GPU in the launch configuration the benchmark uses,
and the oracle runs them sequence by sequence (every chain is compared).
"""
import numpy as np
import pytest
import torch

import oracle
from _helpers import O_BAR, STATE_BAR, F32_BAR, chain_errors, chunked_bars, rel_l2, require_gpu, to_dev
from paper_2607_16831_amd import gdn, synth

pytestmark = pytest.mark.gpu


def _log(name, **errs):
    print("[parity] %s %s" % (name, " ".join("%s=%.3e" % kv for kv in errs.items())),
          flush=True)


def run_prefill(x, dev, chunk=None, alias=False):
    d = to_dev(x, dev)
    w = x["w"]
    chunk = chunk or w.chunk
    s0 = d["initial_state"]
    fs = s0.clone() if (alias and s0 is not None) else None
    o, sT = gdn.prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["cu_seqlens"],
                        initial_state=fs if alias else s0, chunk=chunk,
                        final_state=fs)
    torch.cuda.synchronize()
    return o.cpu(), sT.cpu()


def oracle_prefill(x):
    return oracle.prefill(x["q"], x["k"], x["v"], x["g"], x["beta"],
                          x["cu_seqlens"], x["initial_state"])


def check_result(name, o, sT, o_ref, s_ref, cu, o_bar=O_BAR, s_bar=STATE_BAR):
    """Whole-tensor and per-chain bars; prints both."""
    e = chain_errors(o, sT, o_ref, s_ref, cu)
    print("[parity] %s o=%.3e state=%.3e o_chain_max=%.3e state_chain_max=%.3e worst=%s"
          % (name, e["o"], e["state"], e["o_max"], e["state_max"], e["worst"]), flush=True)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    assert e["o"] <= o_bar and e["state"] <= s_bar
    assert e["o_max"] <= o_bar and e["state_max"] <= s_bar
    return e


def check_full(name, x, dev, chunk=None, alias=False, o_bar=O_BAR, s_bar=STATE_BAR):
    o, sT = run_prefill(x, dev, chunk, alias)
    o_ref, s_ref = oracle_prefill(x)
    check_result(name, o, sT, o_ref, s_ref, x["cu_seqlens"].numpy(), o_bar, s_bar)
    return o, sT


# ------------------------------------------------------------------ decode
def test_decode_batch64_full():
    dev = require_gpu()
    x = synth.make(synth.DECODE_B64)
    d = to_dev(x, dev)
    state = d["initial_state"].clone()
    o = gdn.decode(d["q"], d["k"], d["v"], d["g"], d["beta"], state)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.decode(x["q"], x["k"], x["v"], x["g"], x["beta"],
                                 x["initial_state"])
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(state.cpu(), s_ref)
    _log("decode_B64", o=eo, state=es)
    assert eo <= O_BAR and es <= 1e-5


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("hqk,hv", [(1, 1), (2, 4), (1, 4)])
def test_decode_shapes(d, dtype, hqk, hv):
    dev = require_gpu()
    w = synth.DECODE_B64.replace(n_seqs=5, hqk=hqk, hv=hv, d=d, dtype=dtype, seed=11)
    x = synth.make(w)
    dd = to_dev(x, dev)
    state = dd["initial_state"].clone()
    o = gdn.decode(dd["q"], dd["k"], dd["v"], dd["g"], dd["beta"], state)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.decode(x["q"], x["k"], x["v"], x["g"], x["beta"],
                                 x["initial_state"])
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(state.cpu(), s_ref)
    _log("decode_d%d_%s_%dx%d" % (d, dtype, hqk, hv), o=eo, state=es)
    assert eo <= (O_BAR if dtype == "bf16" else 1e-5) and es <= 1e-5


@pytest.mark.parametrize("B", [1, 2, 8, 16, 48])
def test_decode_small_batches(B):
    """Both launch shapes of the decode kernel (2 passes below two work-groups
    per CU, 4 above) at the benchmark's heads and head size."""
    dev = require_gpu()
    x = synth.make(synth.DECODE_B64.replace(n_seqs=B, seed=40 + B))
    d = to_dev(x, dev)
    state = d["initial_state"].clone()
    o = gdn.decode(d["q"], d["k"], d["v"], d["g"], d["beta"], state)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle.decode(x["q"], x["k"], x["v"], x["g"], x["beta"],
                                 x["initial_state"])
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(state.cpu(), s_ref)
    _log("decode_B%d" % B, o=eo, state=es)
    assert eo <= O_BAR and es <= 1e-5


def test_decode_repeated_steps_match_prefill():
    """Eight decode steps on the GPU == one 8-token prefill (oracle-checked)."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=8, n_seqs=3, hqk=2, hv=4, state_std=0.1,
                                 g_mu=-4.0, seed=21)
    x = synth.make(w)
    d = to_dev(x, dev)
    T = 8
    state = d["initial_state"].clone()
    outs = []
    for t in range(T):
        idx = torch.arange(3, device=dev) * T + t
        outs.append(gdn.decode(d["q"][idx].contiguous(), d["k"][idx].contiguous(),
                               d["v"][idx].contiguous(), d["g"][idx].contiguous(),
                               d["beta"][idx].contiguous(), state))
    torch.cuda.synchronize()
    o_dec = torch.stack(outs, 1).reshape(3 * T, 4, 128).cpu()
    o_ref, s_ref = oracle_prefill(x)
    eo, es = rel_l2(o_dec, o_ref), rel_l2(state.cpu(), s_ref)
    _log("decode_x8_vs_prefill", o=eo, state=es)
    assert eo <= O_BAR and es <= 1e-5


# ------------------------------------------------------------------ prefill
def test_prefill_tiny_f32():
    dev = require_gpu()
    # float32 throughout: the canary bar on o and the state
    check_full("prefill_tiny", synth.make(synth.PREFILL_TINY), dev, o_bar=F32_BAR,
               s_bar=F32_BAR)


def test_prefill_4k_full():
    dev = require_gpu()
    check_full("prefill_4k", synth.make(synth.PREFILL_4K), dev)


def _whole_by_sequence(name, x, dev):
    """Run the whole batch on the GPU, then the oracle one sequence at a time
    (all heads), comparing every chain; the whole-tensor figures are summed
    over the sequences."""
    o, sT = run_prefill(x, dev)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    cu = x["cu_seqlens"].numpy().astype(np.int64)
    s0 = x["initial_state"]
    num_o = den_o = num_s = den_s = 0.0
    o_max = s_max = 0.0
    for n in range(len(cu) - 1):
        t0, t1 = int(cu[n]), int(cu[n + 1])
        o_ref, s_ref = oracle.prefill(
            x["q"][t0:t1], x["k"][t0:t1], x["v"][t0:t1], x["g"][t0:t1], x["beta"][t0:t1],
            np.array([0, t1 - t0], np.int32), None if s0 is None else s0[n:n + 1])
        e = chain_errors(o[t0:t1], sT[n:n + 1], o_ref, s_ref, np.array([0, t1 - t0]))
        o_max, s_max = max(o_max, e["o_max"]), max(s_max, e["state_max"])
        do = o[t0:t1].double().numpy() - o_ref
        ds = sT[n:n + 1].double().numpy() - s_ref
        num_o += float((do * do).sum())
        den_o += float((o_ref * o_ref).sum())
        num_s += float((ds * ds).sum())
        den_s += float((s_ref * s_ref).sum())
        del o_ref, s_ref, do, ds
    eo, es = (num_o / den_o) ** 0.5, (num_s / den_s) ** 0.5
    print("[parity] %s o=%.3e state=%.3e o_chain_max=%.3e state_chain_max=%.3e chains=%d"
          % (name, eo, es, o_max, s_max, (len(cu) - 1) * x["w"].hv), flush=True)
    assert eo <= O_BAR and es <= STATE_BAR
    assert o_max <= O_BAR and s_max <= STATE_BAR


def test_prefill_varlen_full():
    dev = require_gpu()
    _whole_by_sequence("prefill_varlen", synth.make(synth.PREFILL_VARLEN), dev)


def test_prefill_long_full():
    dev = require_gpu()
    _whole_by_sequence("prefill_long", synth.make(synth.PREFILL_LONG), dev)


# ------------------------------------------------------ carry-sensitive cases
RAGGED = (1, 63, 64, 65, 200, 0, 130, 17)


@pytest.mark.parametrize("g_mu,g_zero", [(-4.0, False), (0.0, True)])
def test_prefill_carry_weak_decay(g_mu, g_zero):
    """Weak or no decay with a nonzero initial state: dropping the chunk carry
    or the initial state is visible far above the bars here."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=RAGGED, n_seqs=len(RAGGED),
                                 g_mu=g_mu, g_zero=g_zero, state_std=0.1, seed=31)
    check_full("carry_weak_mu%g_zero%d" % (g_mu, g_zero), synth.make(w), dev)


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("chunk", [16, 32, 64])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_prefill_shapes(d, chunk, dtype):
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=(37, 0, 100, 16, 64),
                                 n_seqs=5, hqk=2, hv=4, d=d, dtype=dtype,
                                 g_mu=-2.0, state_std=0.1, seed=41)
    ob, sb = chunked_bars(dtype)
    check_full("shape_d%d_C%d_%s" % (d, chunk, dtype), synth.make(w), dev, chunk=chunk,
               o_bar=ob, s_bar=sb)


@pytest.mark.parametrize("chunk", [16, 32, 64])
def test_tile_carry_chunk_counts(chunk):
    """The per-tile carry on one sequence of each length from 1 to 9 chunks
    of 64 tokens, each with a ragged tail: the loaders' look-ahead of three
    chunks, issued in parts over the phases, starts, runs and drains at
    every count."""
    dev = require_gpu()
    lengths = tuple(64 * n - 5 for n in range(1, 10))
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=lengths, n_seqs=len(lengths), hqk=1,
                                 hv=2, g_mu=-3.0, state_std=0.1, seed=43)
    check_full("tile_counts_C%d" % chunk, synth.make(w), dev,
               chunk=chunk | gdn.CHUNK_TILE_CARRY)


def test_prefill_alias_in_place():
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=(90, 7), n_seqs=2,
                                 g_mu=-3.0, state_std=0.1, seed=51)
    check_full("alias", synth.make(w), dev, alias=True)


@pytest.mark.parametrize("alias", [False, True])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_prefill_ragged_c16(alias, dtype):
    """Ragged batch at C = 16 (30 chunk slots): long and short sequences, an
    empty one, a nonzero initial state, also updated in place."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=(150, 0, 33, 200, 5), n_seqs=5,
                                 hqk=2, hv=4, d=64, dtype=dtype, g_mu=-4.0,
                                 state_std=0.1, seed=53)
    ob, sb = chunked_bars(dtype)
    check_full("ragged_c16_alias%d_%s" % (alias, dtype), synth.make(w), dev, chunk=16,
               alias=alias, o_bar=ob, s_bar=sb)


def test_prefill_group4_and_group1():
    dev = require_gpu()
    for hqk, hv in ((2, 8), (4, 4)):
        w = synth.PREFILL_4K.replace(seq_len=150, n_seqs=2, hqk=hqk, hv=hv,
                                     g_mu=-3.0, state_std=0.1, seed=61)
        check_full("group_%dx%d" % (hqk, hv), synth.make(w), dev)


def test_prefill_split_composition():
    """prefill(A || B) == prefill(B, initial = final of prefill(A)) on the GPU."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=300, n_seqs=1, hqk=2, hv=4, g_mu=-4.0,
                                 state_std=0.1, seed=71)
    x = to_dev(synth.make(w), dev)
    m = 170
    o, sT = gdn.prefill(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu_seqlens"],
                        initial_state=x["initial_state"])
    cuA = torch.tensor([0, m], dtype=torch.int32, device=dev)
    cuB = torch.tensor([0, 300 - m], dtype=torch.int32, device=dev)
    sl = lambda t, a, b: t[a:b].contiguous()
    oA, sA = gdn.prefill(sl(x["q"], 0, m), sl(x["k"], 0, m), sl(x["v"], 0, m),
                         sl(x["g"], 0, m), sl(x["beta"], 0, m), cuA,
                         initial_state=x["initial_state"])
    oB, sB = gdn.prefill(sl(x["q"], m, 300), sl(x["k"], m, 300), sl(x["v"], m, 300),
                         sl(x["g"], m, 300), sl(x["beta"], m, 300), cuB, initial_state=sA)
    torch.cuda.synchronize()
    eo = rel_l2(torch.cat([oA, oB]).cpu(), o.cpu())
    es = rel_l2(sB.cpu(), sT.cpu())
    _log("split_composition", o=eo, state=es)
    assert eo <= O_BAR and es <= STATE_BAR


@pytest.mark.parametrize("chunk", [16, 64])
def test_prefill_poisoned_workspace(chunk):
    """Every workspace byte set to 0xFF (NaN in bf16 and fp32) before the
    call: a table entry read without having been written this call (such as
    a fragment above the diagonal) would turn the output into NaN."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=None, lengths=(200, 1, 64, 130), n_seqs=4,
                                 hqk=2, hv=4, g_mu=-3.0, state_std=0.1, seed=57)
    x = synth.make(w)
    d = to_dev(x, dev)
    T = int(x["cu_seqlens"][-1])
    ws = gdn.alloc_workspace(w.n_seqs, T, w.hqk, w.hv, w.d, chunk, dev)
    ws.fill_(0xFF)
    o, sT = gdn.prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["cu_seqlens"],
                        initial_state=d["initial_state"], chunk=chunk, workspace=ws)
    torch.cuda.synchronize()
    o_ref, s_ref = oracle_prefill(x)
    eo, es = rel_l2(o.cpu(), o_ref), rel_l2(sT.cpu(), s_ref)
    _log("poisoned_ws_C%d" % chunk, o=eo, state=es)
    assert torch.isfinite(o.float()).all() and torch.isfinite(sT).all()
    assert eo <= O_BAR and es <= STATE_BAR


def test_prefill_all_empty():
    dev = require_gpu()
    s0 = torch.randn(3, 4, 128, 128, device=dev)
    cu = torch.zeros(4, dtype=torch.int32, device=dev)
    e = torch.empty(0, 2, 128, dtype=torch.bfloat16, device=dev)
    ev = torch.empty(0, 4, 128, dtype=torch.bfloat16, device=dev)
    gb = torch.empty(0, 4, device=dev)
    o, sT = gdn.prefill(e, e, ev, gb, gb, cu, initial_state=s0)
    torch.cuda.synchronize()
    assert o.shape == (0, 4, 128) and torch.equal(sT, s0)
    o, sT = gdn.prefill(e, e, ev, gb, gb, cu, initial_state=None)
    torch.cuda.synchronize()
    assert not sT.any()


def test_prefill_strong_decay_stays_finite():
    """Gates 40x the long-context draw: in-chunk log-decay reaches hundreds;
    every exponent must stay a masked non-positive difference."""
    dev = require_gpu()
    w = synth.PREFILL_LONG.replace(seq_len=None, lengths=(500, 77), n_seqs=2,
                                   g_scale=40.0, seed=81)
    check_full("strong_decay_x40", synth.make(w), dev)


def test_identity_padding_tokens():
    """Tokens with g = 0 and beta = 0 leave the state unchanged."""
    dev = require_gpu()
    w = synth.PREFILL_4K.replace(seq_len=70, n_seqs=1, hqk=1, hv=2, g_mu=-3.0,
                                 state_std=0.1, seed=91)
    x = synth.make(w)
    y = dict(x)
    pad = 45
    for key in ("q", "k", "v"):
        y[key] = torch.cat([x[key], torch.randn((pad,) + x[key].shape[1:]).to(x[key].dtype)])
    y["g"] = torch.cat([x["g"], torch.zeros(pad, 2)])
    y["beta"] = torch.cat([x["beta"], torch.zeros(pad, 2)])
    y["cu_seqlens"] = torch.tensor([0, 70 + pad], dtype=torch.int32)
    _, s1 = run_prefill(x, dev)
    _, s2 = run_prefill(y, dev)
    e = rel_l2(s2, s1)
    _log("identity_padding", state=e)
    assert e <= 1e-5
