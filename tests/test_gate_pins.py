"""Pins for the oracle's gate activation (runs without a GPU).

The paper's gate (Section 3.2) is exp(-exp(A_log) softplus(a + b_dt)) with
beta = sigmoid(b); the oracle forms its log, g = -exp(A_log) softplus(a +
dt_bias). Pinned against library routines (numpy.logaddexp(0, x) is
softplus(x), scipy.special.expit is the logistic sigmoid), exact values, two
identities and the limits of the parameters, and wired into the recurrence:
oracle.prefill_gated / decode_gated must equal prefill / decode run on gates
formed independently here.
"""
import numpy as np
import pytest
from scipy.special import expit

import oracle


def _lib_gate(a, b, a_log, dt_bias):
    return -np.exp(a_log)[None, :] * np.logaddexp(0.0, a + dt_bias[None, :]), expit(b)


def test_gate_matches_library_routines():
    rng = np.random.default_rng(7)
    T, HV = 257, 6
    a = rng.standard_normal((T, HV)) * 4.0
    a[0, :] = [-700.0, -40.0, -1e-9, 1e-9, 40.0, 700.0]  # far tails on both sides
    b = rng.standard_normal((T, HV)) * 4.0
    b[0, :] = [-700.0, -40.0, -1e-9, 1e-9, 40.0, 700.0]
    a_log = np.log(rng.uniform(1.0, 16.0, HV))
    dt_bias = rng.uniform(-7.0, 1.0, HV)
    g, beta = oracle.gate(a, b, a_log, dt_bias)
    g_ref, beta_ref = _lib_gate(a, b, a_log, dt_bias)
    assert np.all(g <= 0.0) and np.all((beta >= 0.0) & (beta <= 1.0))
    np.testing.assert_allclose(g, g_ref, rtol=1e-14, atol=1e-300)
    np.testing.assert_allclose(beta, beta_ref, rtol=1e-14, atol=1e-300)


def test_gate_exact_values():
    HV = 3
    dt_bias = np.array([-2.5, 0.0, 1.25])
    a_log = np.array([0.0, np.log(2.0), np.log(16.0)])
    a = -dt_bias[None, :].repeat(2, 0)  # softplus(0) = ln 2
    b = np.zeros((2, HV))
    g, beta = oracle.gate(a, b, a_log, dt_bias)
    np.testing.assert_allclose(g, np.broadcast_to(-np.exp(a_log) * np.log(2.0), g.shape), rtol=2e-15)
    assert np.all(beta == 0.5)


def test_gate_identities():
    # A_log = 0, dt_bias = 0: g(a) = -softplus(a), and
    # softplus(x) - softplus(-x) = x, sigmoid(x) + sigmoid(-x) = 1.
    x = np.linspace(-30.0, 30.0, 121)[:, None]
    zero = np.zeros(1)
    g_pos, b_pos = oracle.gate(x, x, zero, zero)
    g_neg, b_neg = oracle.gate(-x, -x, zero, zero)
    np.testing.assert_allclose(g_neg - g_pos, x, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(b_pos + b_neg, 1.0, rtol=0, atol=1e-15)


def test_gate_limits():
    a = np.array([[100.0, -100.0, 0.3]])
    g, _ = oracle.gate(a, np.zeros((1, 3)), np.array([-1e3, 0.0, 0.0]), np.zeros(3))
    assert g[0, 0] == 0.0                       # exp(A_log) underflows: no decay
    np.testing.assert_allclose(g[0, 1], -np.exp(-100.0), rtol=1e-14)  # softplus ~ e^x
    g2, _ = oracle.gate(np.array([[100.0]]), np.zeros((1, 1)), np.zeros(1), np.zeros(1))
    np.testing.assert_allclose(g2[0, 0], -100.0, rtol=1e-15)        # softplus ~ x


def _raw(rng, T, hqk, hv, d, n_state=None):
    q = rng.standard_normal((T, hqk, d)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = rng.standard_normal((T, hqk, d)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, hv, d))
    a, b = rng.standard_normal((T, hv)), rng.standard_normal((T, hv))
    a_log = np.log(rng.uniform(1.0, 16.0, hv))
    dt_bias = rng.uniform(-6.0, -1.0, hv)
    return q, k, v, a, b, a_log, dt_bias


def test_gated_recurrence_wiring():
    rng = np.random.default_rng(11)
    q, k, v, a, b, a_log, dt_bias = _raw(rng, 40, 2, 4, 8)
    cu = np.array([0, 17, 17, 40], np.int32)
    s0 = rng.standard_normal((3, 4, 8, 8)) * 0.1
    g, beta = _lib_gate(a, b, a_log, dt_bias)
    o_ref, s_ref = oracle.prefill(q, k, v, g, beta, cu, s0)
    o, s = oracle.prefill_gated(q, k, v, a, b, a_log, dt_bias, cu, s0)
    np.testing.assert_allclose(o, o_ref, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(s, s_ref, rtol=1e-12, atol=1e-14)
    # decode: one token per sequence
    q1, k1, v1, a1, b1 = q[:3], k[:3], v[:3], a[:3], b[:3]
    g1, beta1 = _lib_gate(a1, b1, a_log, dt_bias)
    o_ref, s_ref = oracle.decode(q1, k1, v1, g1, beta1, s0)
    o, s = oracle.decode_gated(q1, k1, v1, a1, b1, a_log, dt_bias, s0)
    np.testing.assert_allclose(o, o_ref, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(s, s_ref, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("mistake", ["swap_ab", "no_exp_alog", "bias_outside", "sigmoid_sign"])
def test_gate_pins_reject_mutants(mistake):
    """Plausible slips in a gate implementation fail the library comparison."""
    rng = np.random.default_rng(3)
    a, b = rng.standard_normal((64, 4)), rng.standard_normal((64, 4))
    a_log, dt_bias = np.log(rng.uniform(1, 16, 4)), rng.uniform(-6, 1, 4)
    sp = lambda x: np.logaddexp(0.0, x)
    if mistake == "swap_ab":
        g, beta = -np.exp(a_log) * sp(b + dt_bias), expit(a)
    elif mistake == "no_exp_alog":
        g, beta = -a_log * sp(a + dt_bias), expit(b)
    elif mistake == "bias_outside":
        g, beta = -np.exp(a_log) * (sp(a) + dt_bias), expit(b)
    else:
        g, beta = -np.exp(a_log) * sp(a + dt_bias), expit(-b)
    g_o, beta_o = oracle.gate(a, b, a_log, dt_bias)
    assert not (np.allclose(g, g_o, rtol=1e-12) and np.allclose(beta, beta_o, rtol=1e-12))
