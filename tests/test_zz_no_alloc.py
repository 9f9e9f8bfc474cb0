"""gdn_prefill_scratch (the entry point that allocates nothing) against
gdn_prefill on the GPU.

Both run the same kernels, so the outputs must agree bit for bit. Two calls
in a row: the 4096-token workload (16/32 heads, d = 128, chunk 64: a 50 MiB
workspace), then a smaller ragged batch with initial states and another
chunk size, which runs over whatever the first call left in the library's
array. Both are also held to the oracle's bars.
"""
import pytest
import torch

import oracle
from _helpers import O_BAR, STATE_BAR, chain_errors, require_gpu, to_dev
from paper_2607_16831_amd import gdn, synth

pytestmark = pytest.mark.gpu


def _pair(x, dev, chunk):
    d = to_dev(x, dev)
    T = d["q"].shape[0]
    N = d["cu_seqlens"].shape[0] - 1
    w = x["w"]
    o1 = torch.full((T, w.hv, w.d), float("nan"), dtype=d["q"].dtype, device=dev)
    s1 = torch.full((N, w.hv, w.d, w.d), float("nan"), device=dev)
    print("[no_alloc] %s T=%d N=%d chunk=%d" % (w.name, T, N, chunk), flush=True)
    gdn.prefill_scratch(d["q"], d["k"], d["v"], d["g"], d["beta"], d["cu_seqlens"],
                        initial_state=d["initial_state"], chunk=chunk, o=o1, final_state=s1)
    o2, s2 = gdn.prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["cu_seqlens"],
                         initial_state=d["initial_state"], chunk=chunk)
    torch.cuda.synchronize()
    return o1.cpu(), s1.cpu(), o2.cpu(), s2.cpu()


def test_scratch_entry_matches_workspace_entry_twice():
    dev = require_gpu()
    big = synth.make(synth.PREFILL_4K)
    small = synth.make(synth.PREFILL_4K.replace(seq_len=None, lengths=(300, 0, 77, 129),
                                                n_seqs=4, hqk=2, hv=4, chunk=32,
                                                state_std=0.1, g_mu=-2.0, seed=77))
    for x, chunk in ((big, 64), (small, 32)):
        o1, s1, o2, s2 = _pair(x, dev, chunk)
        assert torch.equal(o1, o2) and torch.equal(s1, s2)
        o_ref, s_ref = oracle.prefill(x["q"], x["k"], x["v"], x["g"], x["beta"],
                                      x["cu_seqlens"], x["initial_state"])
        e = chain_errors(o1, s1, o_ref, s_ref, x["cu_seqlens"])
        print("[no_alloc] o=%.3e state=%.3e o_chain_max=%.3e state_chain_max=%.3e"
              % (e["o"], e["state"], e["o_max"], e["state_max"]), flush=True)
        assert e["o"] <= O_BAR and e["state"] <= STATE_BAR
        assert e["o_max"] <= O_BAR and e["state_max"] <= STATE_BAR


def test_scratch_entry_refuses_oversized_workspace():
    dev = require_gpu()
    x = to_dev(synth.make(synth.PREFILL_4K.replace(seq_len=16384, hqk=16, hv=32)), dev)
    assert gdn.prefill_workspace_size(1, 16384, 16, 32, 128, 128, 64) > \
        gdn.PREFILL_SCRATCH_MAX_BYTES
    with pytest.raises(gdn.GdnError) as err:
        gdn.prefill_scratch(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu_seqlens"],
                            chunk=64)
    assert err.value.status == gdn.GDN_ERR_WORKSPACE
