"""ctypes binding for libgdn (C ABI in include/gdn.h).

Argument marshalling only: every step of prefill and decode runs in the HIP
kernels of ``libgdn.so``. PyTorch supplies device memory and the current HIP
stream. If the library has not been built, or the tensors are not on a GPU,
calls raise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgdn.so")

GDN_OK, GDN_ERR_INVALID_ARG, GDN_ERR_UNSUPPORTED, GDN_ERR_WORKSPACE, GDN_ERR_HIP = range(5)
GDN_BF16, GDN_F32 = 0, 1

EXPORTS = ("gdn_status_string", "gdn_version", "gdn_prefill_workspace_size",
           "gdn_prefill_auto_chunk", "gdn_prefill", "gdn_decode", "gdn_prefill_gated",
           "gdn_decode_gated", "gdn_prefill_scratch")

# Size of the library's fixed prefill workspace on each device
# (GDN_PREFILL_SCRATCH_MAX_BYTES in gdn.h).
PREFILL_SCRATCH_MAX_BYTES = 128 << 20

# Prefill chunk sizes: AUTO lets the library choose from the batch shape,
# SERIAL runs the token-serial path; 16, 32 and 64 run the chunked path.
CHUNK_AUTO, CHUNK_SERIAL = 0, 1
# OR-ed into a chunk size of 16, 32 or 64: diagonal blocks of the WY factor by
# the Neumann product instead of forward substitution.
CHUNK_NEUMANN = 0x100
# OR-ed into a chunk size of 0, 16, 32 or 64: the per-tile carry (instead of
# the library's choice between it and the whole-chain carry).
CHUNK_TILE_CARRY = 0x200
CHUNK_SEGMENT_SHIFT = 16


def CHUNK_SEGMENT(n_chunks: int) -> int:
    """OR-ed into a chunk size of 0, 16, 32 or 64: the whole-chain carry with
    segments of `n_chunks` chunks (1..4095) instead of the library's choice."""
    if not 1 <= n_chunks <= 4095:
        raise ValueError("segment length must be in [1, 4095] chunks")
    return n_chunks << CHUNK_SEGMENT_SHIFT

_lib = None


class GdnError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__("%s failed: %s (status %d)" % (fn, status_string(status), status))


def lib() -> ctypes.CDLL:
    """Load libgdn.so from the package directory (raises if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                "libgdn.so is not built (%s); run python -m paper_2607_16831_amd.build"
                % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        vp, fp, ip = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p
        i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.gdn_status_string.argtypes = [ctypes.c_int]
        L.gdn_status_string.restype = ctypes.c_char_p
        L.gdn_version.argtypes = []
        L.gdn_version.restype = ctypes.c_int
        L.gdn_prefill_workspace_size.argtypes = [i32, i64, i32, i32, i32, i32, i32]
        L.gdn_prefill_workspace_size.restype = sz
        L.gdn_prefill_auto_chunk.argtypes = [i32, i64, i32, i32, i32, i32]
        L.gdn_prefill_auto_chunk.restype = i32
        L.gdn_prefill.argtypes = [vp, vp, vp, fp, fp, ip, fp, vp, fp, i32, i64,
                                  i32, i32, i32, i32, i32, ctypes.c_int, vp, sz, vp]
        L.gdn_prefill.restype = ctypes.c_int
        L.gdn_decode.argtypes = [vp, vp, vp, fp, fp, fp, vp, i32, i32, i32, i32,
                                 i32, ctypes.c_int, vp]
        L.gdn_decode.restype = ctypes.c_int
        L.gdn_prefill_gated.argtypes = [vp, vp, vp, fp, fp, fp, fp, ip, fp, vp, fp, i32,
                                        i64, i32, i32, i32, i32, i32, ctypes.c_int, vp, sz,
                                        vp]
        L.gdn_prefill_gated.restype = ctypes.c_int
        L.gdn_decode_gated.argtypes = [vp, vp, vp, fp, fp, fp, fp, fp, vp, i32, i32, i32,
                                       i32, i32, ctypes.c_int, vp]
        L.gdn_decode_gated.restype = ctypes.c_int
        L.gdn_prefill_scratch.argtypes = [vp, vp, vp, fp, fp, ip, fp, vp, fp, i32, i64,
                                          i32, i32, i32, i32, i32, ctypes.c_int, vp]
        L.gdn_prefill_scratch.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().gdn_status_string(int(status)).decode()


def version() -> int:
    return int(lib().gdn_version())


def prefill_workspace_size(n_seqs, n_tokens, hqk, hv, dk, dv, chunk) -> int:
    return int(lib().gdn_prefill_workspace_size(n_seqs, n_tokens, hqk, hv, dk, dv, chunk))


def prefill_auto_chunk(n_seqs, n_tokens, hqk, hv, dk, dv) -> int:
    """Chunk size the library picks for chunk=CHUNK_AUTO (0 on invalid sizes)."""
    return int(lib().gdn_prefill_auto_chunk(n_seqs, n_tokens, hqk, hv, dk, dv))


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return GDN_BF16
    if t.dtype == torch.float32:
        return GDN_F32
    raise TypeError("q/k/v must be bfloat16 or float32, got %s" % t.dtype)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check_dev(*ts):
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("libgdn takes device tensors (got a %s tensor)" % t.device)
        if not t.is_contiguous():
            raise ValueError("libgdn takes contiguous tensors")


def _shape_error(name, t, want):
    raise ValueError("%s must have shape %s, got %s" % (name, tuple(want), tuple(t.shape)))


def _check_shapes(q, k, v, rows, n_states, gates, state_tensors, o):
    """Every tensor's shape against the sizes taken from q and v, before any
    launch: the C ABI receives bare pointers and cannot tell a short tensor
    from a full one, so a wrong shape would make the kernels read or write
    out of bounds."""
    if q.dim() != 3:
        raise ValueError("q must be [tokens, heads_qk, d_k], got %s" % (tuple(q.shape),))
    if v.dim() != 3:
        raise ValueError("v must be [tokens, heads_v, d_v], got %s" % (tuple(v.shape),))
    _, hqk, dk = q.shape
    hv, dv = v.shape[1], v.shape[2]
    if tuple(k.shape) != tuple(q.shape):
        _shape_error("k", k, q.shape)
    if v.shape[0] != rows:
        _shape_error("v", v, (rows, hv, dv))
    for name, t in gates:
        if t is not None and tuple(t.shape) != (rows, hv):
            _shape_error(name, t, (rows, hv))
    for name, t in state_tensors:
        if t is not None and tuple(t.shape) != (n_states, hv, dv, dk):
            _shape_error(name, t, (n_states, hv, dv, dk))
    if o is not None and tuple(o.shape) != (rows, hv, dv):
        _shape_error("o", o, (rows, hv, dv))


def _check_cu(cu_seqlens):
    if cu_seqlens.dim() != 1 or cu_seqlens.shape[0] < 1:
        raise ValueError("cu_seqlens must be a 1-D tensor of n_seqs + 1 offsets")


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def prefill_raw(q, k, v, g, beta, cu_seqlens, initial_state, o, final_state,
                n_seqs, n_tokens, hqk, hv, dk, dv, chunk, dtype, workspace,
                workspace_bytes, stream) -> int:
    """Direct call of gdn_prefill with integer pointers; returns the status."""
    return int(lib().gdn_prefill(q, k, v, g, beta, cu_seqlens, initial_state, o,
                                 final_state, n_seqs, n_tokens, hqk, hv, dk, dv,
                                 chunk, dtype, workspace, workspace_bytes, stream))


def prefill_scratch_raw(q, k, v, g, beta, cu_seqlens, initial_state, o, final_state,
                        n_seqs, n_tokens, hqk, hv, dk, dv, chunk, dtype, stream) -> int:
    """Direct call of gdn_prefill_scratch with integer pointers; returns the status."""
    return int(lib().gdn_prefill_scratch(q, k, v, g, beta, cu_seqlens, initial_state, o,
                                         final_state, n_seqs, n_tokens, hqk, hv, dk, dv,
                                         chunk, dtype, stream))


def decode_raw(q, k, v, g, beta, state, o, batch, hqk, hv, dk, dv, dtype,
               stream) -> int:
    """Direct call of gdn_decode with integer pointers; returns the status."""
    return int(lib().gdn_decode(q, k, v, g, beta, state, o, batch, hqk, hv, dk,
                                dv, dtype, stream))


def prefill_gated_raw(q, k, v, a, b, a_log, dt_bias, cu_seqlens, initial_state, o,
                      final_state, n_seqs, n_tokens, hqk, hv, dk, dv, chunk, dtype,
                      workspace, workspace_bytes, stream) -> int:
    """Direct call of gdn_prefill_gated with integer pointers; returns the status."""
    return int(lib().gdn_prefill_gated(q, k, v, a, b, a_log, dt_bias, cu_seqlens,
                                       initial_state, o, final_state, n_seqs, n_tokens,
                                       hqk, hv, dk, dv, chunk, dtype, workspace,
                                       workspace_bytes, stream))


def decode_gated_raw(q, k, v, a, b, a_log, dt_bias, state, o, batch, hqk, hv, dk, dv,
                     dtype, stream) -> int:
    """Direct call of gdn_decode_gated with integer pointers; returns the status."""
    return int(lib().gdn_decode_gated(q, k, v, a, b, a_log, dt_bias, state, o, batch,
                                      hqk, hv, dk, dv, dtype, stream))


def alloc_workspace(n_seqs, n_tokens, hqk, hv, d, chunk, device) -> torch.Tensor:
    nbytes = prefill_workspace_size(n_seqs, n_tokens, hqk, hv, d, d, chunk)
    if nbytes == 0:
        raise ValueError("unsupported prefill sizes")
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def prefill(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor,
            beta: torch.Tensor, cu_seqlens: torch.Tensor,
            initial_state: Optional[torch.Tensor] = None, chunk: int = 64,
            o: Optional[torch.Tensor] = None,
            final_state: Optional[torch.Tensor] = None,
            workspace: Optional[torch.Tensor] = None,
            stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Prefill; returns (o [T, HV, DV], final_state [N, HV, DV, DK]).

    chunk: 16, 32 or 64 (chunked path), CHUNK_SERIAL (token-serial path) or
    CHUNK_AUTO (the library's shape dispatch).
    """
    _check_cu(cu_seqlens)
    N = cu_seqlens.shape[0] - 1
    _check_shapes(q, k, v, q.shape[0] if q.dim() == 3 else -1, N,
                  (("g", g), ("beta", beta)),
                  (("initial_state", initial_state), ("final_state", final_state)), o)
    T, hqk, dk = q.shape
    hv, dv = v.shape[1], v.shape[2]
    if o is None:
        o = torch.empty((T, hv, dv), dtype=q.dtype, device=q.device)
    if final_state is None:
        final_state = torch.empty((N, hv, dv, dk), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = alloc_workspace(N, T, hqk, hv, dk, chunk, q.device)
    _check_dev(q, k, v, g, beta, cu_seqlens, initial_state, o, final_state, workspace)
    if cu_seqlens.dtype != torch.int32:
        raise TypeError("cu_seqlens must be int32")
    if g.dtype != torch.float32 or beta.dtype != torch.float32:
        raise TypeError("g and beta must be float32")
    if k.dtype != q.dtype or v.dtype != q.dtype or o.dtype != q.dtype:
        raise TypeError("q, k, v and o must share one dtype")
    st = prefill_raw(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(cu_seqlens),
                     _ptr(initial_state), _ptr(o), _ptr(final_state), N, T, hqk, hv,
                     dk, dv, chunk, _dtype_code(q), _ptr(workspace),
                     workspace.numel(), _stream(stream))
    if st != GDN_OK:
        raise GdnError("gdn_prefill", st)
    return o, final_state


def prefill_scratch(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor,
                    beta: torch.Tensor, cu_seqlens: torch.Tensor,
                    initial_state: Optional[torch.Tensor] = None, chunk: int = 64,
                    o: Optional[torch.Tensor] = None,
                    final_state: Optional[torch.Tensor] = None,
                    stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """prefill() on the library's fixed per-device workspace (gdn_prefill_scratch):
    no workspace argument, and nothing allocated when o and final_state are
    given. Sizes whose workspace exceeds PREFILL_SCRATCH_MAX_BYTES raise
    GdnError (GDN_ERR_WORKSPACE)."""
    _check_cu(cu_seqlens)
    N = cu_seqlens.shape[0] - 1
    _check_shapes(q, k, v, q.shape[0] if q.dim() == 3 else -1, N,
                  (("g", g), ("beta", beta)),
                  (("initial_state", initial_state), ("final_state", final_state)), o)
    T, hqk, dk = q.shape
    hv, dv = v.shape[1], v.shape[2]
    if o is None:
        o = torch.empty((T, hv, dv), dtype=q.dtype, device=q.device)
    if final_state is None:
        final_state = torch.empty((N, hv, dv, dk), dtype=torch.float32, device=q.device)
    _check_dev(q, k, v, g, beta, cu_seqlens, initial_state, o, final_state)
    if cu_seqlens.dtype != torch.int32:
        raise TypeError("cu_seqlens must be int32")
    if g.dtype != torch.float32 or beta.dtype != torch.float32:
        raise TypeError("g and beta must be float32")
    if k.dtype != q.dtype or v.dtype != q.dtype or o.dtype != q.dtype:
        raise TypeError("q, k, v and o must share one dtype")
    st = prefill_scratch_raw(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(cu_seqlens),
                             _ptr(initial_state), _ptr(o), _ptr(final_state), N, T, hqk, hv,
                             dk, dv, chunk, _dtype_code(q), _stream(stream))
    if st != GDN_OK:
        raise GdnError("gdn_prefill_scratch", st)
    return o, final_state


def decode(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, g: torch.Tensor,
           beta: torch.Tensor, state: torch.Tensor,
           o: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """One decode step; advances ``state`` in place and returns o [B, HV, DV]."""
    B = q.shape[0] if q.dim() == 3 else -1
    _check_shapes(q, k, v, B, B, (("g", g), ("beta", beta)), (("state", state),), o)
    B, hqk, dk = q.shape
    hv, dv = v.shape[1], v.shape[2]
    if o is None:
        o = torch.empty((B, hv, dv), dtype=q.dtype, device=q.device)
    _check_dev(q, k, v, g, beta, state, o)
    if g.dtype != torch.float32 or beta.dtype != torch.float32 or state.dtype != torch.float32:
        raise TypeError("g, beta and state must be float32")
    if k.dtype != q.dtype or v.dtype != q.dtype or o.dtype != q.dtype:
        raise TypeError("q, k, v and o must share one dtype")
    st = decode_raw(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(state),
                    _ptr(o), B, hqk, hv, dk, dv, _dtype_code(q), _stream(stream))
    if st != GDN_OK:
        raise GdnError("gdn_decode", st)
    return o


def _check_gate(a, b, a_log, dt_bias, rows, hv):
    for name, t in (("a", a), ("b", b), ("A_log", a_log), ("dt_bias", dt_bias)):
        if t.dtype != torch.float32:
            raise TypeError("%s must be float32" % name)
    if tuple(a.shape) != (rows, hv) or tuple(b.shape) != (rows, hv):
        raise ValueError("a and b must be [%d, %d]" % (rows, hv))
    if tuple(a_log.shape) != (hv,) or tuple(dt_bias.shape) != (hv,):
        raise ValueError("A_log and dt_bias must be [%d]" % hv)


def prefill_gated(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, a: torch.Tensor,
                  b: torch.Tensor, a_log: torch.Tensor, dt_bias: torch.Tensor,
                  cu_seqlens: torch.Tensor, initial_state: Optional[torch.Tensor] = None,
                  chunk: int = 64, o: Optional[torch.Tensor] = None,
                  final_state: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None,
                  stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Chunked prefill from the raw gate inputs a, b [T, HV], A_log, dt_bias [HV]."""
    _check_cu(cu_seqlens)
    N = cu_seqlens.shape[0] - 1
    _check_shapes(q, k, v, q.shape[0] if q.dim() == 3 else -1, N, (),
                  (("initial_state", initial_state), ("final_state", final_state)), o)
    T, hqk, dk = q.shape
    hv, dv = v.shape[1], v.shape[2]
    _check_gate(a, b, a_log, dt_bias, T, hv)
    if o is None:
        o = torch.empty((T, hv, dv), dtype=q.dtype, device=q.device)
    if final_state is None:
        final_state = torch.empty((N, hv, dv, dk), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = alloc_workspace(N, T, hqk, hv, dk, chunk, q.device)
    _check_dev(q, k, v, a, b, a_log, dt_bias, cu_seqlens, initial_state, o, final_state,
               workspace)
    if cu_seqlens.dtype != torch.int32:
        raise TypeError("cu_seqlens must be int32")
    if k.dtype != q.dtype or v.dtype != q.dtype or o.dtype != q.dtype:
        raise TypeError("q, k, v and o must share one dtype")
    st = prefill_gated_raw(_ptr(q), _ptr(k), _ptr(v), _ptr(a), _ptr(b), _ptr(a_log),
                           _ptr(dt_bias), _ptr(cu_seqlens), _ptr(initial_state), _ptr(o),
                           _ptr(final_state), N, T, hqk, hv, dk, dv, chunk, _dtype_code(q),
                           _ptr(workspace), workspace.numel(), _stream(stream))
    if st != GDN_OK:
        raise GdnError("gdn_prefill_gated", st)
    return o, final_state


def decode_gated(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, a: torch.Tensor,
                 b: torch.Tensor, a_log: torch.Tensor, dt_bias: torch.Tensor,
                 state: torch.Tensor, o: Optional[torch.Tensor] = None,
                 stream=None) -> torch.Tensor:
    """One decode step from the raw gate inputs; advances ``state`` in place."""
    B = q.shape[0] if q.dim() == 3 else -1
    _check_shapes(q, k, v, B, B, (), (("state", state),), o)
    B, hqk, dk = q.shape
    hv, dv = v.shape[1], v.shape[2]
    _check_gate(a, b, a_log, dt_bias, B, hv)
    if o is None:
        o = torch.empty((B, hv, dv), dtype=q.dtype, device=q.device)
    _check_dev(q, k, v, a, b, a_log, dt_bias, state, o)
    if state.dtype != torch.float32:
        raise TypeError("state must be float32")
    if k.dtype != q.dtype or v.dtype != q.dtype or o.dtype != q.dtype:
        raise TypeError("q, k, v and o must share one dtype")
    st = decode_gated_raw(_ptr(q), _ptr(k), _ptr(v), _ptr(a), _ptr(b), _ptr(a_log),
                          _ptr(dt_bias), _ptr(state), _ptr(o), B, hqk, hv, dk, dv,
                          _dtype_code(q), _stream(stream))
    if st != GDN_OK:
        raise GdnError("gdn_decode_gated", st)
    return o
