"""Pins of the optimiser step (Adam) against torch.optim.Adam and its first-step closed form."""
import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")


def test_adam_matches_torch_over_steps():
    rng = np.random.default_rng(0)
    p0 = rng.standard_normal((7, 5))
    grads = [rng.standard_normal((7, 5)) * 10.0 ** rng.uniform(-4, 1) for _ in range(6)]
    tp = torch.nn.Parameter(torch.from_numpy(p0.copy()))
    opt = torch.optim.Adam([tp], lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    p, m, v = p0, np.zeros_like(p0), np.zeros_like(p0)
    for t, g in enumerate(grads, start=1):
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
        p, m, v = oracle.adam_step(p, g, m, v, t, 1e-3)
        np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_adam_first_step_closed_form():
    rng = np.random.default_rng(1)
    g = rng.standard_normal(1000) * 10.0 ** rng.uniform(-9, 2, 1000)
    p, m, v = oracle.adam_step(np.zeros(1000), g, np.zeros(1000), np.zeros(1000), 1, 1e-4)
    np.testing.assert_allclose(p, -1e-4 * g / (np.abs(g) + 1e-8), rtol=1e-12)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-14)   # 1 - 0.999 is 0.001 to 1e-15


def test_adam_zero_gradient_keeps_parameters():
    p, m, v = oracle.adam_step(np.ones(4), np.zeros(4), np.zeros(4), np.zeros(4), 3, 1e-2)
    np.testing.assert_array_equal(p, 1.0)
