"""Pins the oracle's discriminator forward/backward and BCE losses."""
import numpy as np
import pytest
import torch

from oracle.mlp import bce_losses, disc_fwd_bwd, mlp_forward, round_bf16, sigmoid


def _net(widths, seed):
    rng = np.random.default_rng(seed)
    W = [rng.standard_normal((o, i)) * 0.7 for i, o in zip(widths[:-1], widths[1:])]
    b = [rng.standard_normal(o) * 0.3 for o in widths[1:]]
    return W, b


def _batches(F, n, seed):
    rng = np.random.default_rng(seed)
    return rng.uniform(0.05, 0.95, (n, F)), rng.uniform(0.05, 0.95, (n + 3, F))


@pytest.mark.parametrize("widths", [(2, 8, 8, 1), (3, 5, 7, 4, 1), (8, 6, 1)])
def test_backward_vs_finite_differences(widths):
    W, b = _net(widths, 1)
    xf, xr = _batches(widths[0], 13, 2)
    r = disc_fwd_bwd(W, b, xf, xr)
    h = 1e-6

    def LD(W_, b_):
        zf, _, _ = mlp_forward(W_, b_, xf)
        zr, _, _ = mlp_forward(W_, b_, xr)
        return bce_losses(zf, zr)[0]

    for l in range(len(W)):
        for idx in [(0, 0), (W[l].shape[0] - 1, W[l].shape[1] - 1), (W[l].shape[0] // 2, 0)]:
            Wp = [w.copy() for w in W]; Wm = [w.copy() for w in W]
            Wp[l][idx] += h; Wm[l][idx] -= h
            fd = (LD(Wp, b) - LD(Wm, b)) / (2 * h)
            assert abs(r["dW"][l][idx] - fd) < 1e-7 + 1e-6 * abs(fd)
        bp = [v.copy() for v in b]; bm = [v.copy() for v in b]
        bp[l][-1] += h; bm[l][-1] -= h
        fd = (LD(W, bp) - LD(W, bm)) / (2 * h)
        assert abs(r["db"][l][-1] - fd) < 1e-7 + 1e-6 * abs(fd)
    # dL_G / d fake input
    for k in (0, 5, 12):
        for j in range(widths[0]):
            xp = xf.copy(); xm = xf.copy()
            xp[k, j] += h; xm[k, j] -= h
            fd = (bce_losses(mlp_forward(W, b, xp)[0], mlp_forward(W, b, xr)[0])[1]
                  - bce_losses(mlp_forward(W, b, xm)[0], mlp_forward(W, b, xr)[0])[1]) / (2 * h)
            assert abs(r["dLg_din"][k, j] - fd) < 1e-8 + 1e-6 * abs(fd)


def test_against_torch_float64_autograd():
    widths = (2, 16, 16, 16, 1)
    W, b = _net(widths, 3)
    xf, xr = _batches(2, 40, 4)
    r = disc_fwd_bwd(W, b, xf, xr)
    tW = [torch.tensor(w, requires_grad=True) for w in W]
    tb = [torch.tensor(v, requires_grad=True) for v in b]
    tf = torch.tensor(xf, requires_grad=True)
    tr = torch.tensor(xr)

    def fwd(h):
        for l in range(len(tW)):
            h = h @ tW[l].T + tb[l]
            if l < len(tW) - 1:
                h = torch.nn.functional.leaky_relu(h, 0.2)
        return h[:, 0]

    zf, zr = fwd(tf), fwd(tr)
    bce = torch.nn.functional.binary_cross_entropy_with_logits
    LD = bce(zr, torch.ones_like(zr)) + bce(zf, torch.zeros_like(zf))
    gW = torch.autograd.grad(LD, tW + tb, retain_graph=True)
    LG = bce(zf, torch.ones_like(zf))
    gx, = torch.autograd.grad(LG, [tf])
    assert abs(float(LD) - r["loss_d"]) < 1e-12 and abs(float(LG) - r["loss_g"]) < 1e-12
    for l in range(len(W)):
        np.testing.assert_allclose(r["dW"][l], gW[l].numpy(), rtol=1e-10, atol=1e-14)
        np.testing.assert_allclose(r["db"][l], gW[len(W) + l].numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(r["dLg_din"], gx.numpy(), rtol=1e-10, atol=1e-16)
    np.testing.assert_allclose(r["logits_fake"], zf.detach().numpy(), rtol=1e-12)


def test_zero_last_layer():
    W, b = _net((2, 8, 8, 1), 5)
    W[-1][:] = 0
    b[-1][:] = 0
    xf, xr = _batches(2, 17, 6)
    r = disc_fwd_bwd(W, b, xf, xr)
    assert abs(r["loss_d"] - 2 * np.log(2)) < 1e-15 and abs(r["loss_g"] - np.log(2)) < 1e-15
    assert np.all(r["dLg_din"] == 0)
    assert all(np.all(r["dW"][l] == 0) for l in range(len(W) - 1))
    # logit layer gradient: 1/2 mean over fakes of h minus 1/2 mean over reals of h
    _, _, hf = mlp_forward(W, b, xf)
    _, _, hr = mlp_forward(W, b, xr)
    np.testing.assert_allclose(r["dW"][-1][0], 0.5 * hf[-1].mean(0) - 0.5 * hr[-1].mean(0), rtol=1e-12)


def test_logistic_regression_closed_form():
    W, b = _net((3, 1), 8)
    xf, xr = _batches(3, 21, 9)
    r = disc_fwd_bwd(W, b, xf, xr)
    zf = xf @ W[0][0] + b[0][0]
    zr = xr @ W[0][0] + b[0][0]
    dW = (sigmoid(zf)[:, None] * xf).mean(0) + ((sigmoid(zr) - 1)[:, None] * xr).mean(0)
    np.testing.assert_allclose(r["dW"][0][0], dW, rtol=1e-12)
    np.testing.assert_allclose(r["db"][0][0], sigmoid(zf).mean() + (sigmoid(zr) - 1).mean(), rtol=1e-12)
    np.testing.assert_allclose(r["dLg_din"], ((sigmoid(zf) - 1) / len(zf))[:, None] * W[0][0][None, :], rtol=1e-12)


def test_bce_at_zero_and_large_logits():
    LD, LG = bce_losses(np.zeros(5), np.zeros(7))
    assert abs(LD - 2 * np.log(2)) < 1e-15 and abs(LG - np.log(2)) < 1e-15
    LD, LG = bce_losses(np.array([-800.0]), np.array([800.0]))
    assert LD < 1e-300 and abs(LG - 800.0) < 1e-12


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(10)
    a = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.005859375, 3e38, 1e-40]])
    a32 = a.astype(np.float32)
    ref = torch.tensor(a32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_bf16(a32), ref)


def test_bf16_mode_is_close_to_fp64():
    W, b = _net((2, 32, 32, 32, 1), 11)
    xf, xr = _batches(2, 64, 12)
    r = disc_fwd_bwd(W, b, xf, xr)
    q = disc_fwd_bwd(W, b, xf, xr, bf16=True)
    rel = lambda p, t: np.linalg.norm(p - t) / np.linalg.norm(t)
    assert 0 < rel(q["logits_fake"], r["logits_fake"]) < 2e-2
    assert 0 < rel(q["dW"][1], r["dW"][1]) < 5e-2


def test_bf16_mode_structure_reduces_to_fp64():
    """With the rounding map replaced by the identity, the bf16 evaluation is the float64 one."""
    from oracle.mlp import _disc_bf16
    W, b = _net((8, 16, 16, 16, 1), 13)
    xf, xr = _batches(8, 30, 14)
    r = disc_fwd_bwd(W, b, xf, xr)
    q = _disc_bf16(W, b, xf, xr, 0.2, lambda a: a)
    for k in ("logits_fake", "logits_real", "dLg_din"):
        np.testing.assert_allclose(q[k], r[k], rtol=1e-12, atol=1e-15)
    assert abs(q["loss_d"] - r["loss_d"]) < 1e-14
    for l in range(len(W)):
        np.testing.assert_allclose(q["dW"][l], r["dW"][l], rtol=1e-11, atol=1e-15)
        np.testing.assert_allclose(q["db"][l], r["db"][l], rtol=1e-11, atol=1e-15)


def test_kink_variants_without_kinks_is_the_gradient():
    """No unit near the kink: a single variant, equal to torch float64 autograd dz/dx."""
    from oracle.mlp import input_grad_kink_variants
    W, b = _net((3, 9, 7, 5, 1), 21)
    x = np.random.default_rng(22).uniform(0.05, 0.95, 3)
    v = input_grad_kink_variants(W, b, x, margin=1e-12)
    assert v.shape == (1, 3)
    xt = torch.tensor(x, requires_grad=True)
    h = xt
    for l in range(len(W)):
        h = h @ torch.tensor(W[l]).T + torch.tensor(b[l])
        if l < len(W) - 1:
            h = torch.nn.functional.leaky_relu(h, 0.2)
    h.sum().backward()
    np.testing.assert_allclose(v[0], xt.grad.numpy(), rtol=1e-13, atol=1e-15)


def test_kink_variants_are_the_one_sided_derivatives():
    """A unit placed exactly on the kink: the two variants are the directional
    derivatives of z from either side (one-sided finite differences)."""
    from oracle.mlp import input_grad_kink_variants
    W, b = _net((2, 6, 6, 1), 23)
    x = np.array([0.37, 0.61])
    o = 2
    b[0] = b[0].copy()
    b[0][o] = -W[0][o] @ x                      # pre-activation of unit o of layer 1 is 0
    v = input_grad_kink_variants(W, b, x, margin=1e-9)
    assert v.shape == (2, 2)

    def z(xx):
        h = xx
        for l in range(len(W)):
            h = W[l] @ h + b[l]
            if l < len(W) - 1:
                h = np.where(h > 0, h, 0.2 * h)
        return h[0]

    d = W[0][o] / np.linalg.norm(W[0][o])      # moves unit o's pre-activation up
    eps = 1e-7
    right = (z(x + eps * d) - z(x)) / eps       # slope 1 side
    left = (z(x) - z(x - eps * d)) / eps        # slope 0.2 side
    got = sorted([float(v[0] @ d), float(v[1] @ d)])
    want = sorted([right, left])
    assert abs(right - left) > 1e-3             # the kink is visible
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-9)


@pytest.mark.parametrize("bf16", [False, True])
def test_input_grad_condition_sums(bf16):
    """dLg_din_cond is the per-entry sum of |terms| of dL_G/d(input): it bounds
    |dLg_din| entrywise (triangle inequality), it equals |dLg_din| when every
    layer has one unit (a single term per entry), and it does not depend on
    the signs of the first layer's weights."""
    W, b = _net((3, 16, 16, 1), 21)
    xf, xr = _batches(3, 40, 22)
    r = disc_fwd_bwd(W, b, xf, xr, bf16=bf16)
    assert np.all(np.abs(r["dLg_din"]) <= r["dLg_din_cond"] * (1 + 1e-12))
    assert np.any(np.abs(r["dLg_din"]) < 0.5 * r["dLg_din_cond"])      # some entries do cancel
    W1, b1 = _net((3, 1, 1, 1), 23)
    r1 = disc_fwd_bwd(W1, b1, xf, xr, bf16=bf16)
    np.testing.assert_allclose(r1["dLg_din_cond"], np.abs(r1["dLg_din"]), rtol=1e-13, atol=0)
    Wf = [w.copy() for w in W]
    Wf[0][:, 1] *= -1.0                                                    # flip one input column's sign
    rf = disc_fwd_bwd(Wf, b, xf * np.array([1.0, -1.0, 1.0]), xr * np.array([1.0, -1.0, 1.0]), bf16=bf16)
    np.testing.assert_allclose(rf["dLg_din_cond"], r["dLg_din_cond"], rtol=1e-12)


def test_step_input_grad_condition_through_the_feature_map():
    """run_step maps the condition sums through |Jacobian| of the HD8 map, so they
    still bound |dL/dx| entrywise."""
    import oracle
    from workloads import gen, get
    from workloads.configs import scaled
    w = scaled(get("higher_dim"), 2, 64)
    inp = gen.make_inputs(w)
    # the workload's network narrowed to 16 hidden units (8-16-16-16-16-1)
    W = [m[:16, :16] if l else m[:16] for l, m in enumerate(inp["W"][:-1])] + [inp["W"][-1][:, :16]]
    b = [v[:16] for v in inp["b"][:-1]] + [inp["b"][-1]]
    real = oracle.sample(inp["theta_star"], 100, 1)
    for bf16 in (False, True):
        r = oracle.run_step(inp["theta"], 64, 0, W, b, real, features="hd8", bf16=bf16)
        assert r["dL_dx_cond"].shape == r["dL_dx"].shape
        assert np.all(np.abs(r["dL_dx"]) <= r["dL_dx_cond"] * (1 + 1e-12))


def test_weight_grad_condition_sums():
    """dW_cond / db_cond are the sums over events of |terms| of dW / db: they
    bound |dW|, |db| entrywise, some entries cancel, and with one fake event and
    the same event as the real batch the logit bias gradient has exactly two
    terms, sigmoid(z) and -sigmoid(-z), so its condition sum is their absolute sum."""
    W, b = _net((3, 12, 12, 1), 31)
    xf, xr = _batches(3, 50, 32)
    r = disc_fwd_bwd(W, b, xf, xr)
    for l in range(len(W)):
        assert np.all(np.abs(r["dW"][l]) <= r["dW_cond"][l] * (1 + 1e-12))
        assert np.all(np.abs(r["db"][l]) <= r["db_cond"][l] * (1 + 1e-12))
    assert any(np.any(np.abs(r["dW"][l]) < 0.5 * r["dW_cond"][l]) for l in range(len(W)))
    same = disc_fwd_bwd(W, b, xf[:1], xf[:1])
    z = same["logits_fake"][0]
    np.testing.assert_allclose(same["db_cond"][-1], [sigmoid(z) + sigmoid(-z)], rtol=1e-12)
    np.testing.assert_allclose(same["db"][-1], [sigmoid(z) - sigmoid(-z)], rtol=1e-12)


# --- kink_margin: the relative distance of the nearest hidden unit from the LeakyReLU kink ---

def _margin(W, b, x):
    from oracle.mlp import kink_margin
    _, pres, hs = mlp_forward(W, b, x)
    return kink_margin(W, b, hs, pres)


def test_kink_margin_hand_value_and_exact_kink():
    # 1 -> 1 -> 1 -> 1: pre_1 = 2 * 1.5 - 1 = 2 against |3| + |-1| = 4 (0.5); h_1 = 2,
    # pre_2 = -3 * 2 + 0.5 = -5.5 against 6 + 0.5 (0.846...); the margin is the smaller
    W = [np.array([[2.0]]), np.array([[-3.0]]), np.array([[1.0]])]
    b = [np.array([-1.0]), np.array([0.5]), np.array([0.0])]
    m = _margin(W, b, np.array([[1.5]]))
    assert m.shape == (1,) and m[0] == 0.5
    # the second unit decides once the first sits further from its kink
    b2 = [np.array([10.0]), np.array([0.5]), np.array([0.0])]
    h1 = 2 * 1.5 + 10.0
    assert abs(_margin(W, b2, np.array([[1.5]]))[0] - (3 * h1 - 0.5) / (3 * h1 + 0.5)) < 1e-15
    # a unit exactly on its kink: margin 0
    W3 = [np.array([[1.0, -1.0], [0.5, 0.25]]), np.array([[1.0, 1.0]])]
    b3 = [np.array([0.0, 0.1]), np.array([0.0])]
    m3 = _margin(W3, b3, np.array([[0.375, 0.375], [0.5, 0.25]]))
    assert m3[0] == 0.0 and m3[1] > 0.0


def test_kink_margin_positive_scale_invariance():
    """LeakyReLU is positively homogeneous, so scaling a layer's weights and bias by
    c > 0 scales its pre-activations and their sums of |terms| alike (and every later
    layer's input by c): the margin does not change."""
    W, b = _net((3, 9, 7, 5, 1), 21)
    x = np.random.default_rng(22).uniform(0.05, 0.95, (50, 3))
    m = _margin(W, b, x)
    c = [3.7, 0.02, 11.0, 0.5]
    Ws = [w * k for w, k in zip(W, c)]
    bs = [v * np.prod(c[:l + 1]) for l, v in enumerate(b)]
    # layer l's input is scaled by prod(c[:l]), so its bias takes the factor of its output
    np.testing.assert_allclose(_margin(Ws, bs, x), m, rtol=1e-10)


def test_kink_margin_is_the_flip_threshold():
    """For one event and the first hidden layer (input fixed), perturbing every term
    W[o][k] x_k and the bias b[o] of every unit by a relative amount eta changes a
    pre-activation by at most eta * sum|terms|: below the margin no unit changes sign,
    and the adversarial perturbation at the margin puts the nearest unit on its kink."""
    rng = np.random.default_rng(23)
    for trial in range(20):
        F, H = int(rng.integers(1, 6)), int(rng.integers(2, 30))
        W = [rng.standard_normal((H, F)), rng.standard_normal((1, H))]
        b = [rng.standard_normal(H) * 0.3, np.zeros(1)]
        x = rng.uniform(-1, 1, (1, F))
        m = _margin(W, b, x)[0]
        pre = W[0] @ x[0] + b[0]
        s = np.sign(pre)[:, None]

        def perturbed(eta):
            # every term moves toward zero of its unit's pre-activation by eta |term|
            Wp = W[0] * (1.0 - eta * s * np.sign(W[0] * x[0][None, :]))
            bp = b[0] * (1.0 - eta * np.sign(pre) * np.sign(b[0]))
            return Wp @ x[0] + bp

        assert np.all(np.sign(perturbed(m * (1 - 1e-6))) == np.sign(pre))
        o = int(np.argmin(np.abs(pre) / (np.abs(W[0]) @ np.abs(x[0]) + np.abs(b[0]))))
        assert abs(perturbed(m)[o]) <= 1e-12 * (np.abs(W[0][o]) @ np.abs(x[0]) + abs(b[0][o]))


# --- logit_cond: sum of |terms| of the logit layer ---

def test_logit_cond_bounds_the_logit_and_single_unit_case():
    from oracle.mlp import logit_cond
    W, b = _net((2, 8, 8, 1), 24)
    xf, xr = _batches(2, 30, 25)
    r = disc_fwd_bwd(W, b, xf, xr)
    assert np.all(np.abs(r["logits_fake"]) <= r["logits_fake_cond"] * (1 + 1e-15))
    assert np.all(np.abs(r["logits_real"]) <= r["logits_real_cond"] * (1 + 1e-15))
    # one unit in the last hidden layer with a zero bias: a single term, so the sum of
    # |terms| is the logit's magnitude
    W1, b1 = _net((2, 4, 1, 1), 26)
    b1[-1][:] = 0.0
    z, _, hs = mlp_forward(W1, b1, xf)
    np.testing.assert_allclose(logit_cond(W1, b1, hs), np.abs(z), rtol=1e-15)
    # flipping the sign of a logit weight leaves it unchanged
    W2 = [w.copy() for w in W]
    W2[-1][0, 3] *= -1.0
    _, _, hs0 = mlp_forward(W, b, xf)
    _, _, hs2 = mlp_forward(W2, b, xf)
    np.testing.assert_array_equal(logit_cond(W2, b, hs2), logit_cond(W, b, hs0))
