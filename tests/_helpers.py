"""Shared test helpers: error metrics, GPU staging, oracle slicing."""
import numpy as np
import torch

# Parity bars (rel-L2 against the fp64 oracle): bf16 outputs and fp32 state.
O_BAR = 2e-2
STATE_BAR = 5e-3
# float32 inputs on the chunked path: float32 products and tables throughout,
# held to the canary bar on o and on the state.
F32_BAR = 1e-4


def chunked_bars(dtype):
    """(o bar, state bar) of the chunked path for an input dtype."""
    return (O_BAR, STATE_BAR) if dtype == "bf16" else (F32_BAR, F32_BAR)


def rel_l2(x, y) -> float:
    """||x - y||_2 / ||y||_2 in fp64 over the whole tensor (y = reference)."""
    x = x.detach().cpu().double().numpy() if hasattr(x, "detach") else np.asarray(x, np.float64)
    y = y.detach().cpu().double().numpy() if hasattr(y, "detach") else np.asarray(y, np.float64)
    ny = np.linalg.norm(y)
    if ny == 0:
        return float(np.linalg.norm(x))
    return float(np.linalg.norm(x - y) / ny)


def gates_from_raw(x: dict):
    """fp32 g and beta of a raw-gate input set, formed by the oracle's gate
    activation (fp64, then rounded to fp32): the input of the plain entry
    points that the gated ones are compared with."""
    import oracle
    g, beta = oracle.gate(x["a"], x["b"], x["A_log"], x["dt_bias"])
    return (torch.from_numpy(g).float().contiguous(),
            torch.from_numpy(beta).float().contiguous())


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU test run without a visible GPU")
    return torch.device("cuda:0")


def to_dev(x: dict, dev):
    out = {}
    for k, v in x.items():
        out[k] = v.to(dev).contiguous() if isinstance(v, torch.Tensor) else v
    return out


def chain_slice(x: dict, n: int, h: int):
    """Inputs of one (sequence, value head) chain as a 1-head oracle problem."""
    w = x["w"]
    grp = w.hv // w.hqk
    cu = x["cu_seqlens"].numpy()
    t0, t1 = int(cu[n]), int(cu[n + 1])
    hk = h // grp
    s0 = x["initial_state"]
    g, beta = x["g"], x["beta"]  # None for raw-gate input sets
    return dict(q=x["q"][t0:t1, hk:hk + 1], k=x["k"][t0:t1, hk:hk + 1],
                v=x["v"][t0:t1, h:h + 1], g=None if g is None else g[t0:t1, h:h + 1],
                beta=None if beta is None else beta[t0:t1, h:h + 1],
                cu_seqlens=np.array([0, t1 - t0], np.int32),
                initial_state=None if s0 is None else s0[n:n + 1, h:h + 1])


def chain_errors(o, sT, o_ref, s_ref, cu):
    """Whole-tensor and per-(sequence, value head) rel-L2 of a prefill result.

    o, o_ref: [T, HV, DV]; sT, s_ref: [N, HV, DV, DK]; cu: cu_seqlens.
    Returns dict(o=, state=, o_max=, state_max=, worst=(n, h)) where o_max and
    state_max are the largest per-chain errors (sequences of length 0 count
    only for the state).
    """
    o = _np(o)
    sT = _np(sT)
    o_ref = np.asarray(o_ref, dtype=np.float64)
    s_ref = np.asarray(s_ref, dtype=np.float64)
    cu = np.asarray(cu).astype(np.int64)
    N, HV = s_ref.shape[0], s_ref.shape[1]
    o_max = s_max = 0.0
    worst = (-1, -1)
    for n in range(N):
        t0, t1 = cu[n], cu[n + 1]
        for h in range(HV):
            es = rel_l2(sT[n, h], s_ref[n, h])
            eo = rel_l2(o[t0:t1, h], o_ref[t0:t1, h]) if t1 > t0 else 0.0
            if max(eo / 2e-2, es / 5e-3) > max(o_max / 2e-2, s_max / 5e-3):
                worst = (n, h)
            o_max, s_max = max(o_max, eo), max(s_max, es)
    return dict(o=rel_l2(o, o_ref), state=rel_l2(sT, s_ref), o_max=o_max,
                state_max=s_max, worst=worst)


def _np(x):
    if hasattr(x, "detach"):
        return x.detach().cpu().double().numpy()
    return np.asarray(x, dtype=np.float64)
