"""Pins of the generator (noise -> parameters) and of the ensemble response."""
import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")


def _gen_weights(widths, seed):
    rng = np.random.default_rng(seed)
    W = [rng.standard_normal((o, i)) * np.sqrt(2.0 / i) for i, o in zip(widths[:-1], widths[1:])]
    b = [rng.uniform(-0.1, 0.1, o) for o in widths[1:]]
    return W, b


def _torch_gen(W, b):
    layers = []
    for l, (w, bb) in enumerate(zip(W, b)):
        lin = torch.nn.Linear(w.shape[1], w.shape[0]).double()
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(w))
            lin.bias.copy_(torch.from_numpy(bb))
        layers.append(lin)
        if l < len(W) - 1:
            layers.append(torch.nn.LeakyReLU(0.2))
    layers.append(torch.nn.Softplus())
    return torch.nn.Sequential(*layers)


def test_paper_generator_parameter_count():
    w = oracle.G_WIDTHS
    assert sum(i * o + o for i, o in zip(w[:-1], w[1:])) == 51206


def test_forward_matches_torch_modules():
    W, b = _gen_weights(oracle.G_WIDTHS, 1)
    n = np.random.default_rng(2).standard_normal((300, 6))
    ref = 1.0 + _torch_gen(W, b)(torch.from_numpy(n)).detach().numpy()
    np.testing.assert_allclose(oracle.generator_forward(W, b, n), ref, rtol=1e-13, atol=1e-13)


def test_backward_matches_torch_autograd():
    W, b = _gen_weights(oracle.G_WIDTHS, 3)
    rng = np.random.default_rng(4)
    n = rng.standard_normal((64, 6))
    g = rng.standard_normal((64, 6))
    net = _torch_gen(W, b)
    out = 1.0 + net(torch.from_numpy(n))
    (out * torch.from_numpy(g)).sum().backward()
    dW, db = oracle.generator_backward(W, b, n, g)
    lins = [m for m in net if isinstance(m, torch.nn.Linear)]
    for l, lin in enumerate(lins):
        np.testing.assert_allclose(dW[l], lin.weight.grad.numpy(), rtol=1e-11, atol=1e-12)
        np.testing.assert_allclose(db[l], lin.bias.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_backward_finite_differences():
    widths = (6, 5, 4, 6)
    W, b = _gen_weights(widths, 5)
    rng = np.random.default_rng(6)
    n = rng.standard_normal((7, 6))
    g = rng.standard_normal((7, 6))
    dW, db = oracle.generator_backward(W, b, n, g)
    f = lambda W_, b_: float((oracle.generator_forward(W_, b_, n) * g).sum())
    h = 1e-6
    for l in range(len(W)):
        for (i, j) in [(0, 0), (W[l].shape[0] - 1, W[l].shape[1] - 1), (1, 2)]:
            Wp = [w.copy() for w in W]; Wm = [w.copy() for w in W]
            Wp[l][i, j] += h; Wm[l][i, j] -= h
            assert abs((f(Wp, b) - f(Wm, b)) / (2 * h) - dW[l][i, j]) < 1e-7 * max(1, abs(dW[l][i, j]))
        bp = [v.copy() for v in b]; bm = [v.copy() for v in b]
        bp[l][1] += h; bm[l][1] -= h
        assert abs((f(W, bp) - f(W, bm)) / (2 * h) - db[l][1]) < 1e-7 * max(1, abs(db[l][1]))


def test_outputs_above_one():
    W, b = _gen_weights(oracle.G_WIDTHS, 7)
    t = oracle.generator_forward(W, b, 5 * np.random.default_rng(8).standard_normal((500, 6)))
    assert (t >= 1.0).all() and np.isfinite(t).all()


def test_ensemble_single_member_and_identical_members():
    rng = np.random.default_rng(9)
    t = 1 + rng.random((1, 50, 6))
    p, s = oracle.ensemble_response(t)
    np.testing.assert_array_equal(s, 0.0)
    np.testing.assert_allclose(p, t[0].mean(axis=0), rtol=1e-15)
    p, s = oracle.ensemble_response(np.repeat(t, 7, axis=0))
    np.testing.assert_allclose(s, 0.0, atol=1e-15)
    np.testing.assert_allclose(p, t[0].mean(axis=0), rtol=1e-14)


def test_ensemble_two_members_closed_form():
    rng = np.random.default_rng(10)
    t = 1 + rng.random((2, 30, 6))
    p, s = oracle.ensemble_response(t)
    np.testing.assert_allclose(p, ((t[0] + t[1]) / 2).mean(axis=0), rtol=1e-14)
    np.testing.assert_allclose(s, (np.abs(t[0] - t[1]) / 2).mean(axis=0), rtol=1e-13)


def test_ensemble_population_std_and_member_order():
    rng = np.random.default_rng(11)
    t = 1 + rng.random((20, 40, 6))
    p, s = oracle.ensemble_response(t)
    np.testing.assert_allclose(s, np.std(t, axis=0, ddof=0).mean(axis=0), rtol=1e-12)
    np.testing.assert_allclose(p, np.mean(t, axis=0).mean(axis=0), rtol=1e-13)
    p2, s2 = oracle.ensemble_response(t[rng.permutation(20)])
    np.testing.assert_allclose(p2, p, rtol=1e-14)
    np.testing.assert_allclose(s2, s, rtol=1e-12)


def test_residual():
    p = np.array([2.0, 5.0, 1.5, 3.0, 3.0, 2.0])
    np.testing.assert_array_equal(oracle.residual(p, p), 0.0)
    np.testing.assert_allclose(oracle.residual(p, 1.1 * p), -0.1, rtol=1e-14)
