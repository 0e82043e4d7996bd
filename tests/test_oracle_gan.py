"""Pins of the oracle's GAN step: the generator's gradient through the whole
chain by finite differences, and the optimiser wiring."""
import numpy as np

import oracle
from workloads import gen

TH = np.array([[2.0, 5.0, 1.5, 3.0, 3.0, 2.0]])


def _setup(k=3, E=70):
    GW, Gb = gen.generator_stack((6, 8, 8, 6), 1, seed=3)
    GW, Gb = [w[0] for w in GW], [v[0] for v in Gb]
    DW, Db = gen.xavier_mlp((2, 8, 8, 1), seed=4)
    n = gen.noise(k, 6, seed=5).astype(np.float64)
    pool = oracle.sample(TH, 2 * k * E, seed=1)
    return oracle.initial_state(GW, Gb, DW, Db), n, pool


def _loss_g(state, n, E, t):
    k = n.shape[0]
    theta = oracle.generator_forward(state["G_W"], state["G_b"], n)
    real = np.full((4, 3), 0.5)   # the reference batch does not enter L_G
    return oracle.run_step(theta, E, 0, state["D_W"], state["D_b"], real, features="proxy2",
                           counter_base=(t - 1) * k * E)["loss_g"]


def test_generator_gradient_finite_differences():
    state, n, pool = _setup()
    E, t = 70, 2
    r = oracle.gan_step(state, n, pool, t, E, fake_seed=0, boot_seed=5)
    h = 1e-6
    for l, (i, j) in [(0, (2, 3)), (1, (5, 1)), (2, (4, 7)), (2, (0, 0))]:
        sp = {**state, "G_W": [w.copy() for w in state["G_W"]]}
        sm = {**state, "G_W": [w.copy() for w in state["G_W"]]}
        sp["G_W"][l][i, j] += h
        sm["G_W"][l][i, j] -= h
        fd = (_loss_g(sp, n, E, t) - _loss_g(sm, n, E, t)) / (2 * h)
        assert abs(fd - r["dW_G"][l][i, j]) <= 1e-6 * max(1.0, abs(fd)) + 1e-9, (l, i, j, fd, r["dW_G"][l][i, j])
    for l in range(3):
        sp = {**state, "G_b": [v.copy() for v in state["G_b"]]}
        sm = {**state, "G_b": [v.copy() for v in state["G_b"]]}
        sp["G_b"][l][1] += h
        sm["G_b"][l][1] -= h
        fd = (_loss_g(sp, n, E, t) - _loss_g(sm, n, E, t)) / (2 * h)
        assert abs(fd - r["db_G"][l][1]) <= 1e-6 * max(1.0, abs(fd)) + 1e-9


def test_zero_learning_rate_keeps_parameters_and_fills_moments():
    state, n, pool = _setup()
    r = oracle.gan_step(state, n, pool, 1, 70, 0, 5, lr_g=0.0, lr_d=0.0)
    s = r["state"]
    for a, b in zip(s["G_W"] + s["D_W"], state["G_W"] + state["D_W"]):
        np.testing.assert_array_equal(a, b)
    grads_d = [g for pair in zip(r["dW_D"], r["db_D"]) for g in pair]
    grads_g = [g for pair in zip(r["dW_G"], r["db_G"]) for g in pair]
    for m, v, g in zip(s["D_m"] + s["G_m"], s["D_v"] + s["G_v"], grads_d + grads_g):
        np.testing.assert_allclose(m, 0.1 * g, rtol=1e-14)
        np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-12)


def test_parameters_move_against_their_gradients():
    state, n, pool = _setup()
    r = oracle.gan_step(state, n, pool, 1, 70, 0, 5)
    s = r["state"]
    for new, old, g in zip(s["D_W"] + s["G_W"], state["D_W"] + state["G_W"], r["dW_D"] + r["dW_G"]):
        big = np.abs(g) > 1e-6 * np.abs(g).max()
        assert (np.sign(new - old)[big] == -np.sign(g)[big]).all()


def test_reference_batch_is_the_steps_bootstrap():
    state, n, pool = _setup()
    r = oracle.gan_step(state, n, pool, 4, 70, 0, 5)
    real, _ = oracle.bootstrap(pool, 3 * 70, 5, 4)
    np.testing.assert_array_equal(r["real"], real)
