"""Pins the oracle's whole step: the per-parameter reduction, the quadratic
critic, and dL/dtheta against finite differences through sampler and network."""
import numpy as np
import pytest

import oracle
from oracle.sampler import uniform_from_words
from workloads import gen


def test_param_grad_brute_force():
    rng = np.random.default_rng(0)
    n_theta, E, d = 3, 7, 2
    g = rng.standard_normal((n_theta * E, d))
    da = rng.standard_normal((n_theta * E, d))
    db = rng.standard_normal((n_theta * E, d))
    out, cond = oracle.param_grad(g, da, db, n_theta, E)
    for i in range(n_theta):
        for j in range(d):
            sa = sum(g[i * E + k, j] * da[i * E + k, j] for k in range(E))
            sb = sum(g[i * E + k, j] * db[i * E + k, j] for k in range(E))
            ca = sum(abs(g[i * E + k, j] * da[i * E + k, j]) for k in range(E))
            assert abs(out[i, 2 * j] - sa) < 1e-12 and abs(out[i, 2 * j + 1] - sb) < 1e-12
            assert abs(cond[i, 2 * j] - ca) < 1e-12


def test_quadratic_critic_unit_theta_closed_form():
    """At theta = 1 the sampler is the identity: x = u, dx/da = -u ln u,
    dx/db = (1-u) ln(1-u), so loss and gradient are sums over the u grid."""
    E = 5000
    theta = np.ones((2, 4))
    r = oracle.run_step(theta, E, fake_seed=3, critic="quadratic", counter_base=77)
    u = uniform_from_words(oracle.event_words(3, 77 + np.arange(2 * E, dtype=np.uint64))[:, :2])
    assert abs(r["loss"] - ((u - 0.5) ** 2).sum()) < 1e-9
    for i in range(2):
        uu = u[i * E:(i + 1) * E]
        np.testing.assert_allclose(r["dL_dtheta"][i, 0::2], (2 * (uu - 0.5) * (-uu * np.log(uu))).sum(0), rtol=1e-10)
        np.testing.assert_allclose(r["dL_dtheta"][i, 1::2], (2 * (uu - 0.5) * (1 - uu) * np.log1p(-uu)).sum(0), rtol=1e-9)


def test_quadratic_critic_expectation():
    """E[dL/dtheta] per event = d/dtheta (m2 - m1) per coordinate (Kumaraswamy moments)."""
    from scipy import special
    theta = np.array([[2.0, 5.0, 1.5, 3.0]])
    E = 300_000
    r = oracle.run_step(theta, E, fake_seed=4, critic="quadratic")
    terms_a = r["dL_dx"] * r["dxda"]
    for j in range(2):
        a, b = theta[0, 2 * j], theta[0, 2 * j + 1]
        m = lambda aa, bb, n: bb * special.beta(1 + n / aa, bb)
        h = 1e-6
        ref = ((m(a + h, b, 2) - m(a + h, b, 1)) - (m(a - h, b, 2) - m(a - h, b, 1))) / (2 * h)
        t = terms_a[:, j]
        assert abs(r["dL_dtheta"][0, 2 * j] / E - ref) < 5 * t.std() / np.sqrt(E)


def _fd_theta(fun, theta, h=1e-6):
    g = np.zeros_like(theta)
    for idx in np.ndindex(*theta.shape):
        tp = theta.copy(); tm = theta.copy()
        tp[idx] += h; tm[idx] -= h
        g[idx] = (fun(tp) - fun(tm)) / (2 * h)
    return g


@pytest.mark.parametrize("features,d,widths", [("identity", 2, (2, 8, 8, 1)), ("hd8", 3, (8, 6, 6, 1)),
                                              ("proxy2", 3, (2, 8, 8, 1))])
def test_generator_loss_gradient_vs_finite_differences(features, d, widths):
    theta = gen.theta_uniform(2, d, seed=9).astype(np.float64)
    E = 40
    W, b = gen.xavier_mlp(widths, seed=2)
    real = oracle.sample(np.array([[2.0, 5.0, 1.5, 3.0, 3.0, 2.0][:2 * d]]), 2 * E, seed=1)
    r = oracle.run_step(theta, E, 0, W, b, real, features=features)
    fd = _fd_theta(lambda t: oracle.run_step(t, E, 0, W, b, real, features=features)["loss_g"], theta)
    np.testing.assert_allclose(r["dL_dtheta"], fd, rtol=2e-5, atol=1e-10)


def test_quadratic_gradient_vs_finite_differences():
    theta = gen.theta_uniform(3, 2, seed=1).astype(np.float64)
    r = oracle.run_step(theta, 30, 8, critic="quadratic")
    fd = _fd_theta(lambda t: oracle.run_step(t, 30, 8, critic="quadratic")["loss"], theta)
    np.testing.assert_allclose(r["dL_dtheta"], fd, rtol=1e-6, atol=1e-9)


def test_param_grad_condition_sums():
    """dL_dtheta_cond bounds |dL/dtheta| entrywise, and with one event per
    parameter row each entry has a single term (dL/dx_j dx_j/da_j or
    dx_j/db_j), so the condition sum is exactly its magnitude."""
    rng = np.random.default_rng(3)
    theta = rng.uniform(1.0, 6.0, (5, 4))
    r = oracle.run_step(theta, 300, 7, critic="quadratic")
    assert np.all(np.abs(r["dL_dtheta"]) <= r["dL_dtheta_cond"] * (1 + 1e-12))
    assert np.any(np.abs(r["dL_dtheta"]) < 0.5 * r["dL_dtheta_cond"])
    r1 = oracle.run_step(theta, 1, 7, critic="quadratic")
    np.testing.assert_allclose(r1["dL_dtheta_cond"], np.abs(r1["dL_dtheta"]), rtol=1e-13)
