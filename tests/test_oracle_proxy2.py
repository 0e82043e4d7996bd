"""Pins of the paper-shape pipeline's two observables y0 = x1 + x3, y1 = x2 + x3
(the oracle's reading of the six-parameter, two-observable proxy)."""
import numpy as np
from scipy.special import beta as B

import oracle

THETA = np.array([[2.0, 5.0, 1.5, 3.0, 3.0, 2.0]])


def _moment(a, b, n):
    """E[x^n] of Kumaraswamy(a, b) = b B(1 + n/a, b)."""
    return b * B(1.0 + n / a, b)


def test_jacobian_finite_differences():
    rng = np.random.default_rng(3)
    x = rng.uniform(0.05, 0.95, (50, 3))
    J = oracle.features_proxy2_jacobian(x)
    h = 1e-6
    for j in range(3):
        e = np.zeros(3)
        e[j] = h
        fd = (oracle.features_proxy2(x + e) - oracle.features_proxy2(x - e)) / (2 * h)
        np.testing.assert_allclose(J[:, :, j], fd, atol=1e-9)


def test_means_and_covariance_of_observables():
    """E[y0] = E[x1] + E[x3], E[y1] = E[x2] + E[x3], Cov(y0, y1) = Var(x3), with the
    closed-form Kumaraswamy moments, within 5 standard errors on 400k events."""
    y = oracle.features_proxy2(oracle.sample(THETA, 400_000, seed=11))
    a, b = THETA[0, 0::2], THETA[0, 1::2]
    m1 = [_moment(a[j], b[j], 1) for j in range(3)]
    var3 = _moment(a[2], b[2], 2) - m1[2] ** 2
    n = y.shape[0]
    for k, expect in ((0, m1[0] + m1[2]), (1, m1[1] + m1[2])):
        se = y[:, k].std() / np.sqrt(n)
        assert abs(y[:, k].mean() - expect) < 5 * se, (k, y[:, k].mean(), expect)
    c = (y[:, 0] - y[:, 0].mean()) * (y[:, 1] - y[:, 1].mean())
    assert abs(c.mean() - var3) < 5 * c.std() / np.sqrt(n), (c.mean(), var3)
    # the observables are not the identity map of any two coordinates
    assert var3 > 0.01


def test_observables_stay_in_range():
    y = oracle.features_proxy2(oracle.sample(THETA, 10_000, seed=2))
    assert (y > 0).all() and (y < 2).all()
