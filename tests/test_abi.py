"""The C ABI without a GPU: exports, version, workspace sizing, validation.

Every rejected call below returns before the library makes any HIP call, so
no device is needed; pointers that would never be dereferenced are passed as
small fake integers where validation must look past them.
"""
import os
import re

import pytest

from paper_2607_16831_amd import gdn

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "gdn.h")
FAKE = 256  # never dereferenced: validation fails first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gdn_\w+)\s*\(", text)))


def test_header_declares_what_binding_expects():
    assert declared_functions() == sorted(gdn.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = gdn.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version_and_status_strings():
    assert gdn.version() >= 10000
    for st in range(5):
        assert gdn.status_string(st)
    assert gdn.status_string(99) == "unknown status"


def test_workspace_size():
    ws = gdn.prefill_workspace_size
    a = ws(1, 4096, 16, 32, 128, 128, 64)
    assert a > 0 and a % 256 == 0
    assert ws(2, 4096, 16, 32, 128, 128, 64) >= a          # more sequences
    assert ws(1, 8192, 16, 32, 128, 128, 64) > a           # more tokens
    assert ws(1, 0, 16, 32, 128, 128, 64) > 0              # one (empty) chunk slot
    assert ws(1, 4096, 16, 32, 128, 128, 48) == 0          # chunk not built
    assert ws(1, 4096, 16, 32, 96, 96, 64) == 0            # head size not built
    assert ws(1, 4096, 16, 24, 128, 128, 64) == 0          # HV % HQK != 0
    assert ws(-1, 4096, 16, 32, 128, 128, 64) == 0
    # the T/P tables dominate: 2 * 2 bytes * C^2 per (chunk bound, value head)
    assert a >= (4096 // 64 + 1) * 32 * 64 * 64 * 4


def test_workspace_size_serial_and_auto():
    ws = gdn.prefill_workspace_size
    # the token-serial path needs none and reports the 256-byte minimum
    assert ws(64, 256, 16, 32, 128, 128, gdn.CHUNK_SERIAL) == 256
    assert ws(0, 0, 16, 32, 128, 128, gdn.CHUNK_SERIAL) == 256
    # automatic: the largest size over every choice, for any batch shape
    for n, t in ((1, 4096), (64, 64), (4096, 4096), (16, 66000), (3, 7)):
        auto = ws(n, t, 16, 32, 128, 128, gdn.CHUNK_AUTO)
        for c in (1, 16, 32, 64):
            assert auto >= ws(n, t, 16, 32, 128, 128, c)
        assert auto in [ws(n, t, 16, 32, 128, 128, c) for c in (1, 16, 32, 64)]
    assert ws(1, 4096, 16, 32, 96, 96, gdn.CHUNK_AUTO) == 0
    assert ws(1, 4096, 16, 32, 128, 128, 2) == 0


def test_neumann_flag_sizes_and_validation():
    ws = gdn.prefill_workspace_size
    N = gdn.CHUNK_NEUMANN
    for c in (16, 32, 64):
        assert ws(3, 1000, 2, 4, 64, 64, c | N) == ws(3, 1000, 2, 4, 64, 64, c)
    assert ws(3, 1000, 2, 4, 64, 64, 1 | N) == 0
    assert ws(3, 1000, 2, 4, 64, 64, 0 | N) == 0
    assert ws(3, 1000, 2, 4, 64, 64, 48 | N) == 0
    E = gdn
    assert _prefill(chunk=1 | N) == E.GDN_ERR_UNSUPPORTED
    assert _prefill(chunk=0 | N) == E.GDN_ERR_UNSUPPORTED
    assert _prefill(chunk=48 | N) == E.GDN_ERR_UNSUPPORTED
    assert _prefill(chunk=16 | N, workspace_bytes=0) == E.GDN_ERR_WORKSPACE
    assert _prefill(chunk=16 | N, q=None) == E.GDN_ERR_INVALID_ARG


def test_auto_chunk_rule():
    ac = gdn.prefill_auto_chunk
    picks = [ac(n, t, 16, 32, 128, 128) for n, t in
             ((4096, 4096), (512, 2048), (128, 128 * 12), (64, 64 * 40), (1, 4096),
              (1, 8192), (3, 12288), (16, 66000), (2, 65536), (4, 16384), (1, 16384))]
    # measured choices at d = 128: token-serial for single tokens, then 16, 32,
    # 64 while 32 would take the per-tile carry (few, short chains: one
    # sequence of 4096 or 8192 tokens), 32 where 32 takes the whole-chain
    # carry (many chains, or long ones: 3 x 4096 tokens and up)
    assert picks == [1, 16, 16, 32, 64, 64, 32, 32, 32, 32, 32]
    # at d = 32 only where 64 takes the whole-chain carry too
    assert ac(4, 16384, 16, 32, 32, 32) == 64 and ac(4, 16384, 16, 32, 64, 64) == 32
    assert ac(16, 66000, 16, 32, 32, 32) == 32
    # many sequences of a few tokens: token-serial at d = 128
    assert ac(2048, 8192, 16, 32, 128, 128) == 1 and ac(512, 2048, 16, 32, 128, 128) == 16
    order = {1: 0, 16: 1, 32: 2, 64: 3}
    for d in (32, 64, 128):
        # every length maps to a built size, monotone in the average length up
        # to where 64 sequences x 32 heads take the whole-chain carry at 32-
        # and 64-token chunks (L > 64), which runs 32-token chunks
        avg = [ac(64, 64 * L, 16, 32, d, d) for L in range(1, 1200)]
        assert set(avg) <= {1, 16, 32, 64} and avg[0] == 1 and avg[-1] == 32
        assert all(order[a] <= order[b] for a, b in zip(avg[:64], avg[1:64]))
        assert set(avg[64:]) == {32}
        # the average is rounded up: 64 sequences of 8 and one of 9 tokens
        # count as 9
        assert ac(65, 64 * 8 + 9, 16, 32, d, d) == ac(1, 9, 16, 32, d, d)
    # smaller heads keep the token-serial path longer (it costs 6 d^2 per token)
    serial_max = {d: max(L for L in range(1, 200) if ac(1, L, 1, 1, d, d) == 1)
                  for d in (32, 64, 128)}
    assert serial_max[32] >= serial_max[64] >= serial_max[128]
    assert ac(0, 0, 16, 32, 128, 128) in (1, 16, 32, 64)
    assert ac(-1, 0, 16, 32, 128, 128) == 0
    assert ac(1, 64, 16, 24, 128, 128) == 0
    assert ac(1, 64, 16, 32, 96, 96) == 0


def _prefill(**kw):
    args = dict(q=FAKE, k=FAKE, v=FAKE, g=FAKE, beta=FAKE, cu_seqlens=FAKE,
                initial_state=None, o=FAKE, final_state=FAKE, n_seqs=1,
                n_tokens=64, hqk=1, hv=1, dk=32, dv=32, chunk=16, dtype=gdn.GDN_F32,
                workspace=FAKE, workspace_bytes=0, stream=None)
    args.update(kw)
    return gdn.prefill_raw(**args)


def test_prefill_validation():
    E = gdn
    assert _prefill(n_seqs=-1) == E.GDN_ERR_INVALID_ARG
    assert _prefill(n_tokens=-5) == E.GDN_ERR_INVALID_ARG
    assert _prefill(hqk=2, hv=3) == E.GDN_ERR_INVALID_ARG
    assert _prefill(hqk=0) == E.GDN_ERR_INVALID_ARG
    assert _prefill(dk=128, dv=64) == E.GDN_ERR_UNSUPPORTED
    assert _prefill(dk=96, dv=96) == E.GDN_ERR_UNSUPPORTED
    assert _prefill(chunk=48) == E.GDN_ERR_UNSUPPORTED
    assert _prefill(chunk=2) == E.GDN_ERR_UNSUPPORTED
    assert _prefill(chunk=-1) == E.GDN_ERR_UNSUPPORTED
    # the token-serial path still takes a (256-byte) workspace argument
    assert _prefill(chunk=gdn.CHUNK_SERIAL, workspace=None) == E.GDN_ERR_WORKSPACE
    assert _prefill(chunk=gdn.CHUNK_SERIAL, workspace_bytes=255) == E.GDN_ERR_WORKSPACE
    assert _prefill(chunk=gdn.CHUNK_SERIAL, q=None, workspace_bytes=256) == \
        E.GDN_ERR_INVALID_ARG
    assert _prefill(chunk=gdn.CHUNK_AUTO, workspace_bytes=255) == E.GDN_ERR_WORKSPACE
    assert _prefill(dtype=7) == E.GDN_ERR_UNSUPPORTED
    assert _prefill(q=None) == E.GDN_ERR_INVALID_ARG
    assert _prefill(cu_seqlens=None) == E.GDN_ERR_INVALID_ARG
    assert _prefill(final_state=None) == E.GDN_ERR_INVALID_ARG
    assert _prefill(workspace=None) == E.GDN_ERR_WORKSPACE
    need = gdn.prefill_workspace_size(1, 64, 1, 1, 32, 32, 16)
    assert _prefill(workspace_bytes=need - 1) == E.GDN_ERR_WORKSPACE
    assert _prefill(workspace=FAKE + 16, workspace_bytes=need) == E.GDN_ERR_WORKSPACE
    # nothing to do: no sequences and no tokens
    assert _prefill(n_seqs=0, n_tokens=0, q=None, cu_seqlens=None) == E.GDN_OK
    assert _prefill(n_seqs=0, n_tokens=3) == E.GDN_ERR_INVALID_ARG


def _decode(**kw):
    args = dict(q=FAKE, k=FAKE, v=FAKE, g=FAKE, beta=FAKE, state=FAKE, o=FAKE,
                batch=4, hqk=2, hv=4, dk=64, dv=64, dtype=gdn.GDN_BF16, stream=None)
    args.update(kw)
    return gdn.decode_raw(**args)


def test_decode_validation():
    E = gdn
    assert _decode(batch=-1) == E.GDN_ERR_INVALID_ARG
    assert _decode(hqk=3) == E.GDN_ERR_INVALID_ARG
    assert _decode(dk=64, dv=32) == E.GDN_ERR_UNSUPPORTED
    assert _decode(dk=256, dv=256) == E.GDN_ERR_UNSUPPORTED
    assert _decode(dtype=5) == E.GDN_ERR_UNSUPPORTED
    assert _decode(state=None) == E.GDN_ERR_INVALID_ARG
    assert _decode(o=None) == E.GDN_ERR_INVALID_ARG
    assert _decode(batch=0, q=None, state=None) == E.GDN_OK


def _prefill_gated(**kw):
    args = dict(q=FAKE, k=FAKE, v=FAKE, a=FAKE, b=FAKE, a_log=FAKE, dt_bias=FAKE,
                cu_seqlens=FAKE, initial_state=None, o=FAKE, final_state=FAKE, n_seqs=1,
                n_tokens=64, hqk=1, hv=1, dk=32, dv=32, chunk=16, dtype=gdn.GDN_F32,
                workspace=FAKE, workspace_bytes=0, stream=None)
    args.update(kw)
    return gdn.prefill_gated_raw(**args)


def _decode_gated(**kw):
    args = dict(q=FAKE, k=FAKE, v=FAKE, a=FAKE, b=FAKE, a_log=FAKE, dt_bias=FAKE,
                state=FAKE, o=FAKE, batch=4, hqk=2, hv=4, dk=64, dv=64,
                dtype=gdn.GDN_BF16, stream=None)
    args.update(kw)
    return gdn.decode_gated_raw(**args)


def test_gated_validation():
    E = gdn
    for name in ("a", "b", "a_log", "dt_bias"):
        assert _prefill_gated(**{name: None}) == E.GDN_ERR_INVALID_ARG, name
        assert _decode_gated(**{name: None}) == E.GDN_ERR_INVALID_ARG, name
    assert _prefill_gated(dk=96, dv=96) == E.GDN_ERR_UNSUPPORTED
    assert _prefill_gated(hqk=2, hv=3) == E.GDN_ERR_INVALID_ARG
    # the gated call sizes its workspace like the plain one
    need = gdn.prefill_workspace_size(1, 64, 1, 1, 32, 32, 16)
    assert _prefill_gated(workspace_bytes=need - 1) == E.GDN_ERR_WORKSPACE
    assert _prefill_gated(n_seqs=0, n_tokens=0, q=None, a=None, b=None, a_log=None,
                          dt_bias=None, cu_seqlens=None) == E.GDN_OK
    assert _decode_gated(batch=0, q=None, a=None, state=None) == E.GDN_OK
    assert _decode_gated(dtype=5) == E.GDN_ERR_UNSUPPORTED
    # the plain entry points still need g and beta
    assert _prefill(g=None) == E.GDN_ERR_INVALID_ARG
    assert _decode(beta=None) == E.GDN_ERR_INVALID_ARG


def test_binding_refuses_host_tensors():
    import torch
    x = torch.zeros(4, 1, 32)
    with pytest.raises(ValueError):
        gdn.decode(x, x, x, torch.zeros(4, 1), torch.zeros(4, 1),
                   torch.zeros(4, 1, 32, 32), o=torch.zeros(4, 1, 32))


def test_carry_flags_sizes_and_validation():
    """The carry choice and GDN_CHUNK_SEGMENT(L). The 4096-token workload (one
    sequence, 16/32 heads, C = 64: 32 chains) takes the per-tile carry,
    whose workspace adds the Q fragment table and holds no segment maps; the
    66K-token batch of 16 sequences takes the whole-chain carry. With a forced
    segment length the workspace grows as segments shrink (more maps) and has
    no maps when one segment holds every sequence. Refused: a flag with
    chunk = 1, the tile flag together with a segment length, unknown bits."""
    ws = gdn.prefill_workspace_size
    S = gdn.CHUNK_SEGMENT
    TILE = gdn.CHUNK_TILE_CARRY
    auto = ws(1, 4096, 16, 32, 128, 128, 64)
    assert auto == ws(1, 4096, 16, 32, 128, 128, 64 | TILE)
    one = ws(1, 4096, 16, 32, 128, 128, 64 | S(64))
    # Q fragments: (64 + 1 chunk slots) x 16 key heads x 64 x 128 bf16
    assert auto - one == 65 * 16 * 64 * 128 * 2
    eight = ws(1, 4096, 16, 32, 128, 128, 64 | S(8))
    # 8 segments -> 7 maps, each B (fp32) + M^T hi/lo (bf16): 8 * 32 * 128 * 128 * 8 bytes
    assert eight - one == 8 * 32 * 128 * 128 * 8
    assert ws(1, 4096, 16, 32, 128, 128, 64 | S(4)) > eight
    assert one == ws(1, 4096, 16, 32, 128, 128, 64 | S(4095))
    # many chains: the whole-chain carry (no Q fragments), segments picked by size
    big = ws(16, 66000, 16, 32, 128, 128, 64)
    assert big < ws(16, 66000, 16, 32, 128, 128, 64 | TILE)
    # few but long chains (2 x 32768 tokens: 64 chains, automatic segments of
    # 1024 * 32 / 256 = 128 chunks): the whole-chain carry as with S(128)
    long = ws(2, 65536, 16, 32, 128, 128, 64)
    assert long == ws(2, 65536, 16, 32, 128, 128, 64 | S(128))
    assert long != ws(2, 65536, 16, 32, 128, 128, 64 | TILE)
    for bad in (1 | S(2), 1 | TILE, 64 | TILE | S(2), 64 | (1 << 30)):
        assert ws(1, 4096, 16, 32, 128, 128, bad) == 0
        assert _prefill(chunk=bad) == gdn.GDN_ERR_UNSUPPORTED
    assert ws(1, 4096, 16, 32, 128, 128, 0 | S(2)) >= ws(1, 4096, 16, 32, 128, 128, 64 | S(2))
    with pytest.raises(ValueError):
        S(0)
    with pytest.raises(ValueError):
        S(4096)
    assert _prefill(chunk=64 | S(2), workspace_bytes=0) == gdn.GDN_ERR_WORKSPACE


def test_binding_checks_every_shape_before_launch():
    """The binding compares every tensor with the sizes taken from q and v
    before it reaches the C ABI (which gets bare pointers): a short state,
    gate or output tensor raises ValueError naming the tensor, and no call is
    made. The tensors are host tensors, so a shape that passed would stop at
    the device check with a different message."""
    import torch
    T, N, hqk, hv, d = 12, 2, 1, 2, 32
    q = torch.zeros(T, hqk, d)
    v = torch.zeros(T, hv, d)
    g = torch.zeros(T, hv)
    cu = torch.tensor([0, 5, 12], dtype=torch.int32)
    good = dict(q=q, k=q, v=v, g=g, beta=g, cu_seqlens=cu,
                initial_state=torch.zeros(N, hv, d, d), o=torch.zeros(T, hv, d),
                final_state=torch.zeros(N, hv, d, d))
    with pytest.raises(ValueError, match="device tensors"):
        gdn.prefill(**good)
    bad = {
        "k": torch.zeros(T, hqk + 1, d), "v": torch.zeros(T - 1, hv, d),
        "g": torch.zeros(T, hv + 1), "beta": torch.zeros(T - 1, hv),
        "initial_state": torch.zeros(N - 1, hv, d, d),
        "final_state": torch.zeros(N, hv, d, d - 1), "o": torch.zeros(T, hv, d + 1),
    }
    for name, t in bad.items():
        with pytest.raises(ValueError, match="^%s must have shape" % name):
            gdn.prefill(**dict(good, **{name: t}))
    with pytest.raises(ValueError, match="cu_seqlens"):
        gdn.prefill(**dict(good, cu_seqlens=torch.zeros(0, dtype=torch.int32)))

    B = 3
    dq, dv = torch.zeros(B, hqk, d), torch.zeros(B, hv, d)
    dg = torch.zeros(B, hv)
    dgood = dict(q=dq, k=dq, v=dv, g=dg, beta=dg, state=torch.zeros(B, hv, d, d),
                 o=torch.zeros(B, hv, d))
    with pytest.raises(ValueError, match="device tensors"):
        gdn.decode(**dgood)
    dbad = {"k": torch.zeros(B, hqk, d + 1), "v": torch.zeros(B + 1, hv, d),
            "g": torch.zeros(B, hv - 1), "beta": torch.zeros(B + 1, hv),
            "state": torch.zeros(B - 1, hv, d, d), "o": torch.zeros(B, hv - 1, d)}
    for name, t in dbad.items():
        with pytest.raises(ValueError, match="^%s must have shape" % name):
            gdn.decode(**dict(dgood, **{name: t}))

    # the gated entry points check the same tensors (the gates by their own rule)
    a = torch.zeros(T, hv)
    hvec = torch.zeros(hv)
    with pytest.raises(ValueError, match="^final_state must have shape"):
        gdn.prefill_gated(q, q, v, a, a, hvec, hvec, cu,
                          final_state=torch.zeros(N + 1, hv, d, d))
    with pytest.raises(ValueError, match="^state must have shape"):
        gdn.decode_gated(dq, dq, dv, dg, dg, hvec, hvec, torch.zeros(B, hv, d, 2 * d))


def test_scratch_prefill_validation():
    """gdn_prefill_scratch refuses, before any HIP call, what gdn_prefill
    refuses, and sizes whose workspace exceeds the library's fixed array."""
    E = gdn

    def call(**kw):
        args = dict(q=FAKE, k=FAKE, v=FAKE, g=FAKE, beta=FAKE, cu_seqlens=FAKE,
                    initial_state=None, o=FAKE, final_state=FAKE, n_seqs=1, n_tokens=64,
                    hqk=1, hv=1, dk=32, dv=32, chunk=16, dtype=gdn.GDN_F32, stream=None)
        args.update(kw)
        return gdn.prefill_scratch_raw(**args)

    assert call(n_seqs=-1) == E.GDN_ERR_INVALID_ARG
    assert call(hqk=2, hv=3) == E.GDN_ERR_INVALID_ARG
    assert call(dk=96, dv=96) == E.GDN_ERR_UNSUPPORTED
    assert call(chunk=48) == E.GDN_ERR_UNSUPPORTED
    assert call(q=None) == E.GDN_ERR_INVALID_ARG
    assert call(final_state=None) == E.GDN_ERR_INVALID_ARG
    assert call(n_seqs=0, n_tokens=0, q=None, cu_seqlens=None) == E.GDN_OK
    # 16384 tokens at 16/32 heads, d = 128, chunk 64: 197 MiB > 128 MiB
    big = dict(n_tokens=16384, hqk=16, hv=32, dk=128, dv=128, chunk=64, dtype=gdn.GDN_BF16)
    assert gdn.prefill_workspace_size(1, 16384, 16, 32, 128, 128, 64) > \
        gdn.PREFILL_SCRATCH_MAX_BYTES
    assert call(**big) == E.GDN_ERR_WORKSPACE
    # chunk = 0 is held to the size of the chunk it resolves to: 32-token
    # chunks for one sequence of 32768 tokens (168 MiB)
    assert gdn.prefill_auto_chunk(1, 32768, 16, 32, 128, 128) == 32
    assert call(**dict(big, n_tokens=32768, chunk=0)) == E.GDN_ERR_WORKSPACE
    assert gdn.prefill_workspace_size(1, 4096, 16, 32, 128, 128, 64) <= \
        gdn.PREFILL_SCRATCH_MAX_BYTES
    # the header and the binding agree on the array's size
    text = open(HEADER).read()
    assert "#define GDN_PREFILL_SCRATCH_MAX_BYTES (128u << 20)" in text
    assert gdn.PREFILL_SCRATCH_MAX_BYTES == 128 << 20
