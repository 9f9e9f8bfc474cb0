"""Pins for the CPU oracle (runs without a GPU).

The paper prints no worked numeric example, so the oracle is pinned by what the
mathematics fixes:

* the explicit matrix form S_t = alpha S (I - beta k k^T) + beta v k^T,
  o_t = S_t q_t with d_k != d_v and grouped heads (catches transposes and
  index mistakes);
* exact rational arithmetic on dyadic inputs (every fp64 step is exact there,
  so the oracle must agree bit for bit);
* the paper's one-pass output rewrite q^T(gS) + delta (q^T k) (Section 3.2);
* closed forms: beta = 0 pure decay; beta = 1 key replacement; orthonormal
  keys with g = 0, beta = 1 writing S = sum v_i k_i^T;
* an independent chunked (WY / UT) fp64 evaluation, chunk sizes 1..64,
  ragged last chunks;
* structure: split composition, packing invariance with empty sequences,
  grouped-head equivalence, linearity in (S0, V), the Frobenius norm bound,
  decode == one-token prefill.

Each pin is a function of an implementation, and ``test_pins_reject_mutants``
plants plausible mistakes (on the CPU, in numpy copies) to show that every
mutant fails at least one pin.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle

RTOL = 1e-12


def _rand_inputs(rng, lens, hqk, hv, dk, dv, g_mu=0.0, s0=True, unit=True):
    T = int(sum(lens))
    q = rng.standard_normal((T, hqk, dk))
    k = rng.standard_normal((T, hqk, dk))
    if unit:
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
        q /= np.linalg.norm(q, axis=-1, keepdims=True)
    v = rng.standard_normal((T, hv, dv))
    g = -np.logaddexp(0.0, rng.standard_normal((T, hv)) + g_mu)
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((T, hv))))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    st = rng.standard_normal((len(lens), hv, dv, dk)) * 0.3 if s0 else None
    return q, k, v, g, beta, cu, st


def _rel(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


# ---------------------------------------------------------------- references
def matrix_form(q, k, v, g, beta, cu, s0):
    """S_t = alpha S (I - beta k k^T) + beta v k^T, o_t = S_t q_t, with the
    (d_k x d_k) projector formed explicitly for every token."""
    T, hqk, dk = q.shape
    hv, dv = v.shape[1], v.shape[2]
    N = len(cu) - 1
    grp = hv // hqk
    o = np.zeros((T, hv, dv))
    sf = np.zeros((N, hv, dv, dk))
    for n in range(N):
        for h in range(hv):
            S = np.zeros((dv, dk)) if s0 is None else s0[n, h].copy()
            for t in range(cu[n], cu[n + 1]):
                kk = k[t, h // grp]
                proj = np.eye(dk) - beta[t, h] * np.outer(kk, kk)
                S = np.exp(g[t, h]) * S @ proj + beta[t, h] * np.outer(v[t, h], kk)
                o[t, h] = S @ q[t, h // grp]
            sf[n, h] = S
    return o, sf


def chunked_form(q, k, v, g, beta, cu, s0, C):
    """Chunked WY/UT evaluation in fp64, written independently of the oracle.

    Per chunk of n <= C tokens with incoming state S0 (d_v x d_k):
      gamma = cumsum(g), E_ij = exp(gamma_i - gamma_j) for i >= j,
      A = strict_lower(beta_i E_ij k_i.k_j), T = (I + A)^-1,
      U = T (beta V) - T (beta exp(gamma) K) S0^T,
      O = (exp(gamma) Q) S0^T + (E * Q K^T) U,
      S = exp(gamma_n) S0 + U^T (exp(gamma_n - gamma) K).
    """
    T_, hqk, dk = q.shape
    hv, dv = v.shape[1], v.shape[2]
    N = len(cu) - 1
    grp = hv // hqk
    o = np.zeros((T_, hv, dv))
    sf = np.zeros((N, hv, dv, dk))
    for n in range(N):
        for h in range(hv):
            S = np.zeros((dv, dk)) if s0 is None else s0[n, h].copy()
            for c0 in range(cu[n], cu[n + 1], C):
                c1 = min(c0 + C, cu[n + 1])
                K = k[c0:c1, h // grp]
                Q = q[c0:c1, h // grp]
                V = v[c0:c1, h]
                b = beta[c0:c1, h]
                gam = np.cumsum(g[c0:c1, h])
                diff = gam[:, None] - gam[None, :]
                low = np.tril(np.ones_like(diff, dtype=bool))
                E = np.where(low, np.exp(np.where(low, diff, 0.0)), 0.0)
                A = np.tril(b[:, None] * E * (K @ K.T), -1)
                Tm = np.linalg.inv(np.eye(len(b)) + A)
                W = Tm @ (b[:, None] * np.exp(gam)[:, None] * K)
                U = Tm @ (b[:, None] * V) - W @ S.T
                o[c0:c1, h] = (np.exp(gam)[:, None] * Q) @ S.T + (E * (Q @ K.T)) @ U
                S = np.exp(gam[-1]) * S + U.T @ (np.exp(gam[-1] - gam)[:, None] * K)
            sf[n, h] = S
    return o, sf


# ---------------------------------------------------------------- pin checks
def pin_matrix_form(impl, rng):
    args = _rand_inputs(rng, [7, 0, 5], hqk=2, hv=4, dk=5, dv=3)
    o, sf = impl(*args)
    o2, sf2 = matrix_form(*args)
    return _rel(o, o2) < RTOL and _rel(sf, sf2) < RTOL


def pin_exact_rational(impl, rng):
    """Dyadic inputs, g = 0: every fp64 product and sum is exact."""
    dk, dv, T = 3, 2, 6
    pick = lambda vals, shape: rng.choice(vals, size=shape)
    q = pick([-1.0, -0.5, 0.0, 0.5, 1.0], (T, 1, dk))
    k = pick([-1.0, -0.5, 0.0, 0.5, 1.0], (T, 1, dk))
    v = pick([-2.0, -1.0, 0.0, 1.0, 0.5], (T, 1, dv))
    beta = pick([0.0, 0.25, 0.5, 1.0], (T, 1))
    g = np.zeros((T, 1))
    s0 = pick([-1.0, 0.0, 0.5, 1.0], (1, 1, dv, dk))
    cu = np.array([0, T], dtype=np.int32)
    o, sf = impl(q, k, v, g, beta, cu, s0)
    F = Fraction
    S = [[F(float(s0[0, 0, r, c])) for c in range(dk)] for r in range(dv)]
    ok = True
    for t in range(T):
        kk = [F(float(x)) for x in k[t, 0]]
        qq = [F(float(x)) for x in q[t, 0]]
        b = F(float(beta[t, 0]))
        # S (I - b k k^T) + b v k^T, entry by entry
        Sk = [sum(S[r][c] * kk[c] for c in range(dk)) for r in range(dv)]
        S = [[S[r][c] - b * Sk[r] * kk[c] + b * F(float(v[t, 0, r])) * kk[c]
              for c in range(dk)] for r in range(dv)]
        for r in range(dv):
            ok &= float(sum(S[r][c] * qq[c] for c in range(dk))) == o[t, 0, r]
    for r in range(dv):
        for c in range(dk):
            ok &= float(S[r][c]) == sf[0, 0, r, c]
    return bool(ok)


def pin_one_pass_rewrite(impl, rng):
    """o_t = q^T (alpha S_{t-1}) + delta (q^T k): the paper's output rewrite,
    evaluated here against the OLD state, must equal the implementation's
    output (which reads the new state)."""
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, [9], hqk=1, hv=2, dk=4, dv=4)
    o, _ = impl(q, k, v, g, beta, cu, s0)
    ok = True
    for h in range(2):
        S = s0[0, h].copy()
        for t in range(9):
            aS = np.exp(g[t, h]) * S
            delta = beta[t, h] * (v[t, h] - aS @ k[t, 0])
            out = aS @ q[t, 0] + delta * (q[t, 0] @ k[t, 0])
            ok &= _rel(o[t, h], out) < RTOL
            S = aS + np.outer(delta, k[t, 0])
    return bool(ok)


def pin_beta_zero(impl, rng):
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, [6, 4], hqk=1, hv=1, dk=3, dv=3)
    beta = np.zeros_like(beta)
    o, sf = impl(q, k, v, g, beta, cu, s0)
    ok = True
    for n in range(2):
        gam = np.cumsum(g[cu[n]:cu[n + 1], 0])
        for i, t in enumerate(range(cu[n], cu[n + 1])):
            ok &= _rel(o[t, 0], np.exp(gam[i]) * s0[n, 0] @ q[t, 0]) < RTOL
        ok &= _rel(sf[n, 0], np.exp(gam[-1]) * s0[n, 0]) < RTOL
    return bool(ok)


def pin_key_replacement(impl, rng):
    """beta = 1, unit key: the new state maps k_t to v_t exactly, any alpha."""
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, [5], hqk=1, hv=1, dk=4, dv=3)
    ok = True
    for t_end in range(1, 6):
        sub = lambda a: a[:t_end]
        cu2 = np.array([0, t_end], dtype=np.int32)
        _, sf = impl(sub(q), sub(k), sub(v), sub(g), np.ones((t_end, 1)), cu2, s0)
        ok &= _rel(sf[0, 0] @ k[t_end - 1, 0], v[t_end - 1, 0]) < 1e-12
    return bool(ok)


def pin_orthonormal_keys(impl, rng):
    d = 4
    Qm, _ = np.linalg.qr(rng.standard_normal((d, d)))
    k = Qm.T.reshape(d, 1, d)             # k_i = i-th orthonormal vector
    q = rng.standard_normal((d, 1, d))
    v = rng.standard_normal((d, 1, d))
    g = np.zeros((d, 1))
    beta = np.ones((d, 1))
    cu = np.array([0, d], dtype=np.int32)
    s0 = rng.standard_normal((1, 1, d, d))
    _, sf = impl(q, k, v, g, beta, cu, s0)
    expect = sum(np.outer(v[i, 0], k[i, 0]) for i in range(d))
    ok = _rel(sf[0, 0], expect) < 1e-12
    # k' orthogonal to k_t passes through unchanged by token t
    cu1 = np.array([0, 1], dtype=np.int32)
    _, s1 = impl(q[:1], k[:1], v[:1], g[:1], beta[:1], cu1, s0)
    for j in range(1, d):
        ok &= _rel(s1[0, 0] @ k[j, 0], s0[0, 0] @ k[j, 0]) < 1e-12
    return bool(ok)


def pin_chunked(impl, rng):
    args = _rand_inputs(rng, [70, 33, 1], hqk=1, hv=2, dk=6, dv=5)
    o, sf = impl(*args)
    ok = True
    for C in (1, 2, 3, 16, 64):
        o2, sf2 = chunked_form(*args, C)
        ok &= _rel(o, o2) < 1e-11 and _rel(sf, sf2) < 1e-11
    return bool(ok)


def pin_split_composition(impl, rng):
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, [20], hqk=1, hv=2, dk=4, dv=4)
    o, sf = impl(q, k, v, g, beta, cu, s0)
    m = 13
    a = lambda x: x[:m]
    b = lambda x: x[m:]
    oa, sa = impl(a(q), a(k), a(v), a(g), a(beta), np.array([0, m], np.int32), s0)
    ob, sb = impl(b(q), b(k), b(v), b(g), b(beta), np.array([0, 20 - m], np.int32), sa)
    return _rel(np.concatenate([oa, ob]), o) < RTOL and _rel(sb, sf) < RTOL


def pin_packing(impl, rng):
    lens = [5, 0, 8, 3, 0]
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, lens, hqk=1, hv=2, dk=3, dv=3)
    o, sf = impl(q, k, v, g, beta, cu, s0)
    ok = True
    for n in range(len(lens)):
        sl = slice(cu[n], cu[n + 1])
        on, sn = impl(q[sl], k[sl], v[sl], g[sl], beta[sl],
                      np.array([0, lens[n]], np.int32), s0[n:n + 1])
        ok &= _rel(o[sl], on) < RTOL and _rel(sf[n:n + 1], sn) < RTOL
        if lens[n] == 0:
            ok &= np.array_equal(sf[n], s0[n])
    return bool(ok)


def pin_gqa(impl, rng):
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, [6, 3], hqk=2, hv=4, dk=3, dv=3)
    o, sf = impl(q, k, v, g, beta, cu, s0)
    idx = np.arange(4) // 2
    o2, sf2 = impl(q[:, idx], k[:, idx], v, g, beta, cu, s0)
    return _rel(o, o2) < RTOL and _rel(sf, sf2) < RTOL


def pin_linearity(impl, rng):
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, [7], hqk=1, hv=1, dk=3, dv=3)
    v2 = rng.standard_normal(v.shape)
    s02 = rng.standard_normal(s0.shape)
    a, b = 0.7, -1.3
    o1, f1 = impl(q, k, v, g, beta, cu, s0)
    o2, f2 = impl(q, k, v2, g, beta, cu, s02)
    o3, f3 = impl(q, k, a * v + b * v2, g, beta, cu, a * s0 + b * s02)
    return _rel(o3, a * o1 + b * o2) < 1e-11 and _rel(f3, a * f1 + b * f2) < 1e-11


def pin_norm_bound(impl, rng):
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, [12], hqk=1, hv=1, dk=4, dv=4)
    ok = True
    prev = s0[0, 0]
    for t in range(12):
        _, sf = impl(q[:t + 1], k[:t + 1], v[:t + 1], g[:t + 1], beta[:t + 1],
                     np.array([0, t + 1], np.int32), s0)
        bound = np.exp(g[t, 0]) * np.linalg.norm(prev) + beta[t, 0] * np.linalg.norm(v[t, 0])
        ok &= np.linalg.norm(sf[0, 0]) <= bound * (1 + 1e-12)
        prev = sf[0, 0]
    return bool(ok)


PINS = [pin_matrix_form, pin_exact_rational, pin_one_pass_rewrite, pin_beta_zero,
        pin_key_replacement, pin_orthonormal_keys, pin_chunked,
        pin_split_composition, pin_packing, pin_gqa, pin_linearity,
        pin_norm_bound]


def oracle_impl(q, k, v, g, beta, cu, s0):
    return oracle.prefill(q, k, v, g, beta, cu, s0)


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin):
    assert pin(oracle_impl, np.random.default_rng(7))


# ---------------------------------------------------------------- mutants
def _mutant(kind):
    """Sequential numpy recurrence with one planted mistake."""
    def impl(q, k, v, g, beta, cu, s0):
        T, hqk, dk = q.shape
        hv, dv = v.shape[1], v.shape[2]
        N = len(cu) - 1
        grp = hv // hqk
        o = np.zeros((T, hv, dv))
        sf = np.zeros((N, hv, dv, dk))
        for n in range(N):
            for h in range(hv):
                hk = (h % hqk) if kind == "gqa_modulo" else h // grp
                S = np.zeros((dv, dk)) if (s0 is None or kind == "no_s0") else s0[n, h].copy()
                for t in range(cu[n], cu[n + 1]):
                    a = np.exp(g[t, h])
                    kk, qq, b = k[t, hk], q[t, hk], beta[t, h]
                    if kind == "old_not_decayed":
                        old = S @ kk
                    elif kind == "transposed":
                        old = a * (S.T @ kk)    # state read along the wrong axis
                    else:
                        old = a * (S @ kk)
                    delta = b * (v[t, h] - old)
                    if kind == "sign":
                        delta = b * (old - v[t, h])
                    if kind == "beta_missing":
                        delta = v[t, h] - old
                    Sn = a * S + np.outer(delta, kk)
                    if kind == "decay_after":
                        Sn = a * (S + np.outer(delta, kk))
                    o[t, h] = (a * S) @ qq if kind == "output_old_state" else Sn @ qq
                    S = Sn
                sf[n, h] = S
        return o, sf
    return impl


MUTANTS = ["old_not_decayed", "sign", "beta_missing", "decay_after",
           "output_old_state", "gqa_modulo", "no_s0", "transposed"]


def test_mutant_harness_is_faithful():
    """The unmutated numpy copy passes every pin (so failures below come from
    the planted mistakes, not from the harness)."""
    impl = _mutant("none")
    for pin in PINS:
        assert pin(impl, np.random.default_rng(7)), pin.__name__


@pytest.mark.parametrize("kind", MUTANTS)
def test_pins_reject_mutants(kind):
    impl = _mutant(kind)
    failed = []
    for pin in PINS:
        try:
            ok = pin(impl, np.random.default_rng(7))
        except Exception:
            ok = False
        if not ok:
            failed.append(pin.__name__)
    assert failed, "mutant %s passed every pin" % kind


# ---------------------------------------------------------------- plumbing
def test_decode_equals_one_token_prefill():
    rng = np.random.default_rng(3)
    B, hqk, hv, d = 5, 2, 4, 6
    q, k, v, g, beta, cu, s0 = _rand_inputs(rng, [1] * B, hqk, hv, d, d)
    o1, s1 = oracle.decode(q, k, v, g, beta, s0)
    o2, s2 = oracle.prefill(q, k, v, g, beta, cu, s0)
    assert np.array_equal(o1, o2) and np.array_equal(s1, s2)


def test_empty_batch_and_zero_state():
    q = np.zeros((0, 1, 4)); v = np.zeros((0, 2, 4)); g = np.zeros((0, 2))
    o, sf = oracle.prefill(q, q, v, g, g, np.array([0, 0, 0], np.int32), None)
    assert o.shape == (0, 2, 4) and sf.shape == (2, 2, 4, 4) and not sf.any()
    o, sf = oracle.prefill(q, q, v, g, g, np.array([0], np.int32), None)
    assert sf.shape == (0, 2, 4, 4)


def test_rejects_malformed():
    q = np.zeros((3, 1, 4)); v = np.zeros((3, 2, 4)); g = np.zeros((3, 2))
    with pytest.raises(ValueError):
        oracle.prefill(q, q, v, g, g, np.array([0, 2], np.int32))   # cu[N] != T
    with pytest.raises(ValueError):
        oracle.prefill(q, q, v, g, g, np.array([0, 2, 1, 3], np.int32))
    with pytest.raises(ValueError):
        q2 = np.zeros((3, 2, 4))                                    # HV % HQK != 0
        oracle.prefill(q2, q2, np.zeros((3, 3, 4)), np.zeros((3, 3)),
                       np.zeros((3, 3)), np.array([0, 3], np.int32))
