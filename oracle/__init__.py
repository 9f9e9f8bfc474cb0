"""CPU oracle for the Gated DeltaNet recurrence -- test infrastructure only.

Only the test suite, the smoke check and the CPU-baseline leg of the benchmark
may import this package. The product library never links or calls it, and it
shares no code with the HIP path.

The arithmetic lives in ``gdn_ref.c`` (fp64, token-serial, OpenMP over
(sequence, value head) chains); this module only compiles it with gcc,
converts inputs to contiguous float64 arrays and marshals the call. The
computed quantity is the gated delta rule of the paper's Section 3.2 (the
display equations for old_v, delta and S'), with ``g`` taken as the log of the
paper's multiplicative gate, so alpha = exp(g); see ``gdn_ref.c``.

Pins: every function here is checked in ``tests/test_oracle_pins.py`` against
the explicit matrix form S_t = alpha S (I - beta k k^T) + beta v k^T, the
paper's one-pass output rewrite, closed forms (beta = 0 decay, key replacement
with orthonormal keys), exact rational arithmetic and an independent chunked
fp64 evaluation; the gate activation against numpy's logaddexp and scipy's
expit, exact values (softplus(0) = ln 2, sigmoid(0) = 1/2), the identities
softplus(x) - softplus(-x) = x and sigmoid(x) + sigmoid(-x) = 1, and its
limits (A_log -> -inf gives no decay).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gdn_ref.c")
_LIB_PATH = os.path.join(_HERE, "libgdn_ref.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile gdn_ref.c into oracle/libgdn_ref.so with gcc (-O2, OpenMP).

    -ffp-contract=off keeps every product and sum a separately rounded fp64
    operation, exactly as written in the source.
    """
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-shared",
               "-fPIC", "-std=c99", _SRC, "-o", tmp, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                build(force=True)
            lib = ctypes.CDLL(_LIB_PATH)
            dp = ctypes.POINTER(ctypes.c_double)
            ip = ctypes.POINTER(ctypes.c_int32)
            i32, i64 = ctypes.c_int32, ctypes.c_int64
            lib.gdn_ref_prefill.argtypes = [dp, dp, dp, dp, dp, ip, dp, dp, dp,
                                            i32, i64, i32, i32, i32, i32]
            lib.gdn_ref_prefill.restype = ctypes.c_int
            lib.gdn_ref_decode.argtypes = [dp, dp, dp, dp, dp, dp, dp,
                                           i32, i32, i32, i32, i32]
            lib.gdn_ref_decode.restype = ctypes.c_int
            lib.gdn_ref_gate.argtypes = [dp, dp, dp, dp, dp, dp, i64, i32]
            lib.gdn_ref_gate.restype = ctypes.c_int
            lib.gdn_ref_num_threads.argtypes = []
            lib.gdn_ref_num_threads.restype = ctypes.c_int
            _lib = lib
    return _lib


def _f64(x) -> np.ndarray:
    """Exact upcast of a numpy array or CPU torch tensor (bf16/f32/f64) to f64."""
    if hasattr(x, "detach"):  # torch tensor: bf16 widens exactly to f32
        x = x.detach().cpu()
        if str(x.dtype) == "torch.bfloat16":
            x = x.float()
        x = x.double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def num_threads() -> int:
    return int(_load().gdn_ref_num_threads())


def prefill(q, k, v, g, beta, cu_seqlens, initial_state=None):
    """Token-serial prefill over packed sequences.

    q, k: [T, HQK, DK]; v: [T, HV, DV]; g, beta: [T, HV]; cu_seqlens: [N+1];
    initial_state: [N, HV, DV, DK] or None (zeros).
    Returns (o [T, HV, DV] float64, final_state [N, HV, DV, DK] float64).
    """
    lib = _load()
    q, k, v, g, beta = (_f64(a) for a in (q, k, v, g, beta))
    if hasattr(cu_seqlens, "detach"):
        cu_seqlens = cu_seqlens.detach().cpu().numpy()
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    T, HQK, DK = q.shape
    HV, DV = v.shape[1], v.shape[2]
    N = cu.shape[0] - 1
    if k.shape != q.shape or v.shape[0] != T or g.shape != (T, HV) \
            or beta.shape != (T, HV):
        raise ValueError("oracle.prefill: inconsistent shapes")
    s0 = None
    if initial_state is not None:
        s0 = _f64(initial_state)
        if s0.shape != (N, HV, DV, DK):
            raise ValueError("oracle.prefill: initial_state shape")
    o = np.zeros((T, HV, DV), dtype=np.float64)
    sf = np.zeros((N, HV, DV, DK), dtype=np.float64)
    rc = lib.gdn_ref_prefill(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                             cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                             _ptr(s0) if s0 is not None else None,
                             _ptr(o), _ptr(sf), N, T, HQK, HV, DK, DV)
    if rc != 0:
        raise ValueError("oracle.prefill: rejected arguments (code %d)" % rc)
    return o, sf


def decode(q, k, v, g, beta, state):
    """One decode step for B single-token sequences.

    q, k: [B, HQK, DK]; v: [B, HV, DV]; g, beta: [B, HV];
    state: [B, HV, DV, DK] (not modified; the advanced copy is returned).
    Returns (o [B, HV, DV], new_state [B, HV, DV, DK]), both float64.
    """
    lib = _load()
    q, k, v, g, beta = (_f64(a) for a in (q, k, v, g, beta))
    s = _f64(state).copy()
    B, HQK, DK = q.shape
    HV, DV = v.shape[1], v.shape[2]
    if s.shape != (B, HV, DV, DK) or g.shape != (B, HV):
        raise ValueError("oracle.decode: inconsistent shapes")
    o = np.zeros((B, HV, DV), dtype=np.float64)
    rc = lib.gdn_ref_decode(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                            _ptr(s), _ptr(o), B, HQK, HV, DK, DV)
    if rc != 0:
        raise ValueError("oracle.decode: rejected arguments (code %d)" % rc)
    return o, s


def gate(a, b, a_log, dt_bias):
    """Gate activation of the raw inputs (paper, Section 3.2, see gdn_ref.c).

    a, b: [T, HV]; a_log, dt_bias: [HV]. Returns (g, beta), both [T, HV]
    float64: g = -exp(A_log) softplus(a + dt_bias) (the log of the paper's
    gate), beta = sigmoid(b).
    """
    lib = _load()
    a, b, a_log, dt_bias = (_f64(x) for x in (a, b, a_log, dt_bias))
    T, HV = a.shape
    if b.shape != (T, HV) or a_log.shape != (HV,) or dt_bias.shape != (HV,):
        raise ValueError("oracle.gate: inconsistent shapes")
    g = np.zeros((T, HV), dtype=np.float64)
    beta = np.zeros((T, HV), dtype=np.float64)
    rc = lib.gdn_ref_gate(_ptr(a), _ptr(b), _ptr(a_log), _ptr(dt_bias), _ptr(g),
                          _ptr(beta), T, HV)
    if rc != 0:
        raise ValueError("oracle.gate: rejected arguments (code %d)" % rc)
    return g, beta


def prefill_gated(q, k, v, a, b, a_log, dt_bias, cu_seqlens, initial_state=None):
    """prefill() with g and beta formed from the raw gate inputs by gate()."""
    g, beta = gate(a, b, a_log, dt_bias)
    return prefill(q, k, v, g, beta, cu_seqlens, initial_state)


def decode_gated(q, k, v, a, b, a_log, dt_bias, state):
    """decode() with g and beta formed from the raw gate inputs by gate()."""
    g, beta = gate(a, b, a_log, dt_bias)
    return decode(q, k, v, g, beta, state)
