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
