"""The Neumann product form of the chunk solve, checked on the CPU in fp64.

The chunked prefill can form the diagonal 16 x 16 blocks of (I + A)^-1 by
(I - N)(I + N^2)(I + N^4)(I + N^8), N strictly lower (the Neumann series,
finite because N^16 = 0; the chunk-solve variant named in the paper's Section
5.1). This checks the identity itself, independently of any kernel: against
numpy's inverse and against the truncated series, on blocks with the entry
distribution of the method's A = strict_lower(beta E K K^T) (unit keys,
beta in (0, 1), decays in (0, 1]), and on the full 64 x 64 chunk matrix with
six factors.
"""
import numpy as np


def _strict_lower_a(n, rng, d=128):
    k = rng.standard_normal((n, d))
    k /= np.linalg.norm(k, axis=1, keepdims=True)
    g = -np.logaddexp(0.0, rng.standard_normal(n))   # log-decay, <= 0
    gam = np.cumsum(g)
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal(n)))
    E = np.exp(np.minimum(gam[:, None] - gam[None, :], 0.0))
    return np.tril(beta[:, None] * E * (k @ k.T), -1)


def _neumann_product(N, factors):
    inv = np.eye(N.shape[0]) - N
    P = -N
    for _ in range(1, factors):
        P = P @ P
        inv = (np.eye(N.shape[0]) + P) @ inv
    return inv


def test_product_form_matches_inverse_16():
    rng = np.random.default_rng(0)
    for _ in range(50):
        N = _strict_lower_a(16, rng)
        ref = np.linalg.inv(np.eye(16) + N)
        got = _neumann_product(N, 4)
        assert np.max(np.abs(got - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


def test_product_form_matches_truncated_series():
    rng = np.random.default_rng(1)
    N = _strict_lower_a(16, rng)
    series = sum(np.linalg.matrix_power(-N, j) for j in range(16))
    np.testing.assert_allclose(_neumann_product(N, 4), series, rtol=0, atol=1e-12)
    assert np.count_nonzero(np.linalg.matrix_power(N, 16)) == 0  # nilpotent


def test_product_form_full_chunk_64():
    rng = np.random.default_rng(2)
    N = _strict_lower_a(64, rng)
    ref = np.linalg.inv(np.eye(64) + N)
    got = _neumann_product(N, 6)
    assert np.max(np.abs(got - ref)) <= 1e-11 * max(1.0, np.max(np.abs(ref)))


def test_too_few_factors_is_wrong():
    """Three factors cover N^0..N^7 only: a strictly lower block with a long
    chain of nonzeros then differs from the inverse."""
    N = np.diag(np.full(15, 0.9), -1)
    ref = np.linalg.inv(np.eye(16) + N)
    assert np.max(np.abs(_neumann_product(N, 3) - ref)) > 1e-3
    assert np.max(np.abs(_neumann_product(N, 4) - ref)) < 1e-14
