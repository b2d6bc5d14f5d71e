"""Pins for the oracle's query-side transform (no GPU): Algorithm 1 steps
4-6, z-score normalisation (Eq. 1), PCA projection (Section 3.3) and L2
normalisation (Eq. 2).  Checks use closed forms and properties the
mathematics fixes, not a retyping of the formula: identity projection of
standardised data, orthogonal invariance, scale invariance, the effect of
eps in each equation, and an exact rational computation on a tiny case."""
from fractions import Fraction
import math

import numpy as np
import pytest

import oracle


def test_identity_projection_of_standard_data():
    """mean 0, var = 1 - eps, W = first l columns of I: the output is the
    first l coordinates of x, scaled to unit length."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 12))
    eps = 1e-5
    W = np.eye(12)[:, :4]
    y = oracle.transform(x, np.zeros(12), np.full(12, 1 - eps), W, eps_z=eps)
    want = x[:, :4] / np.linalg.norm(x[:, :4], axis=1, keepdims=True)
    assert np.allclose(y, want, rtol=0, atol=1e-15)


def test_orthogonal_projection_keeps_unit_norm_and_angles():
    """With an orthonormal W spanning all dims the output norm is 1 and inner
    products between outputs equal those of the standardised inputs / norms."""
    rng = np.random.default_rng(2)
    D = 9
    Q, _ = np.linalg.qr(rng.standard_normal((D, D)))
    x = rng.standard_normal((4, D))
    mu = rng.standard_normal(D)
    var = rng.uniform(0.5, 2.0, D)
    y = oracle.transform(x, mu, var, Q, eps_z=0.0)
    z = (x - mu) / np.sqrt(var)
    zn = z / np.linalg.norm(z, axis=1, keepdims=True)
    assert np.allclose(np.linalg.norm(y, axis=1), 1.0, atol=1e-14)
    assert np.allclose(y @ y.T, zn @ zn.T, atol=1e-14)


def test_scaling_the_input_direction_does_not_matter_after_centring():
    """(x - mu) scaled by c > 0 gives the same unit output (Eq. 2 removes it)."""
    rng = np.random.default_rng(3)
    x = rng.standard_normal((3, 7))
    mu = rng.standard_normal(7)
    var = rng.uniform(0.2, 3.0, 7)
    W = rng.standard_normal((7, 5))
    a = oracle.transform(x, mu, var, W)
    b = oracle.transform(mu + 3.5 * (x - mu), mu, var, W)
    assert np.allclose(a, b, atol=1e-14)


def test_eps_of_eq2_guards_the_zero_vector():
    """x == mean: z = 0, the projection is 0 and Eq. 2 returns 0 (not NaN)."""
    mu = np.arange(6, dtype=np.float64)
    y = oracle.transform(mu[None, :], mu, np.ones(6), np.ones((6, 2)))
    assert np.array_equal(y, np.zeros((1, 2)))


def test_eps_of_eq1_enters_under_the_square_root():
    """var = 0 on one dim: that dim is scaled by 1/sqrt(eps) exactly."""
    x = np.array([[2.0, 0.0]])
    W = np.array([[1.0], [0.0]])
    eps = 0.25
    y_unnorm_dir = oracle.transform(x, np.zeros(2), np.zeros(2), W, eps_z=eps)
    assert y_unnorm_dir[0, 0] == 1.0  # sign survives normalisation
    W2 = np.array([[1.0, 0.0], [0.0, 1.0]])
    y = oracle.transform(np.array([[2.0, 3.0]]), np.zeros(2), np.array([0.0, 0.75]), W2, eps_z=eps)
    z = np.array([2.0 / math.sqrt(0.25), 3.0 / math.sqrt(1.0)])
    assert np.allclose(y[0], z / np.linalg.norm(z), atol=1e-15)


def test_exact_rational_tiny_case():
    """Exact arithmetic with var + eps perfect squares: every step rational."""
    x = [[3, -1, 2], [0, 4, 1]]
    mu = [1, 1, -1]
    var = [4 - Fraction(1, 4), 1 - Fraction(1, 4), 9 - Fraction(1, 4)]  # + eps = 4, 1, 9
    W = [[1, 2], [0, -1], [3, 1]]
    for r in range(2):
        z = [Fraction(x[r][j] - mu[j]) / [2, 1, 3][j] for j in range(3)]
        v = [sum(z[j] * W[j][c] for j in range(3)) for c in range(2)]
        n = math.sqrt(float(sum(t * t for t in v)))
        want = [float(t) / n for t in v]
        got = oracle.transform(np.array([x[r]], float), np.array(mu, float),
                               np.array([float(v_) for v_ in var]), np.array(W, float),
                               eps_z=0.25)[0]
        assert np.allclose(got, want, rtol=0, atol=2e-16 * 8)


def test_argument_errors():
    with pytest.raises(ValueError):
        oracle.transform(np.zeros((2, 3)), np.zeros(3), np.ones(3), np.zeros((4, 2)))
    with pytest.raises(ValueError):
        oracle.transform(np.zeros((2, 3)), np.zeros(2), np.ones(3), np.zeros((3, 2)))
