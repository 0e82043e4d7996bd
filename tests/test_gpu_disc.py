"""GPU parity of the discriminator step (fp32) against the CPU oracle,
through the C ABI: logits, losses, weight gradients, dL_G/dx and dL_G/dtheta."""
import numpy as np
import pytest

import oracle
import paper_2407_00051_amd as sg
from tests.parity import assert_condition_aware, assert_normwise, to_np
from workloads import gen, get
from workloads.configs import scaled

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
TOL = 1e-4
KINK = 1e-5   # relative pre-activation margin below which fp32 and fp64 may branch differently


def _setup(w, n_real=None):
    inp = gen.make_inputs(w)
    dev = "cuda:0"
    th = torch.tensor(inp["theta"], device=dev)
    ts = torch.tensor(inp["theta_star"], device=dev)
    W = [torch.tensor(m, device=dev) for m in inp["W"]]
    b = [torch.tensor(v, device=dev) for v in inp["b"]]
    n_real = n_real or w.n_events
    return inp, th, ts, W, b, n_real


def _oracle(inp, w, real_np):
    return oracle.run_step(inp["theta"], w.events_per_theta, w.fake_seed, inp["W"], inp["b"], real_np,
                           features=w.features)


def _check_near_kinks(gx, ref, W, b, idx, features="identity"):
    """Events within KINK of a LeakyReLU kink: the computed dL_G/dx must equal
    e_G dz/dx for one admissible choice of one-sided slopes at the near-kink
    units (several results are correct there; the oracle enumerates them).
    Returns the worst error and the oracle's dL_G/dx with those events set to
    the admissible variant the computation took."""
    eG = -oracle.mlp.sigmoid(-ref["logits_fake"]) / ref["logits_fake"].shape[0]
    worst = 0.0
    matched = ref["dL_dx"].copy()
    for i in idx:
        x = ref["x"][i:i + 1]
        if features == "identity":
            v = eG[i] * oracle.input_grad_kink_variants(W, b, x[0], margin=KINK)
        else:   # dz/dy of the two observables, taken back to the coordinates
            vy = oracle.input_grad_kink_variants(W, b, oracle.features_proxy2(x)[0], margin=KINK)
            v = eG[i] * vy @ oracle.features_proxy2_jacobian(x)[0]
        errs = np.abs(v - gx[i]).max(axis=1) / np.abs(v).max()
        k = int(np.argmin(errs))
        worst = max(worst, errs[k])
        assert errs[k] <= TOL, (i, errs[k], gx[i], v)
        matched[i] = v[k]
    return worst, matched


def _check(o, ref, n_layers, fused=True, W=None, b=None, n_theta=None, E=None, features="identity"):
    assert_normwise(to_np(o["logits_fake"]), ref["logits_fake"], TOL, "logits_fake")
    assert_normwise(to_np(o["logits_real"]), ref["logits_real"], TOL, "logits_real")
    assert abs(o["loss_d"].item() - ref["loss_d"]) <= TOL * abs(ref["loss_d"])
    assert abs(o["loss_g"].item() - ref["loss_g"]) <= TOL * abs(ref["loss_g"])
    for l in range(n_layers):
        assert_normwise(to_np(o["dW"][l]), ref["dW"][l], TOL, f"dW[{l}]")
        assert_normwise(to_np(o["db"][l]), ref["db"][l], TOL, f"db[{l}]")
    # dL_G/dx per event: events whose hidden pre-activations sit at rounding
    # level from the LeakyReLU kink take a precision-dependent branch; compare
    # the others elementwise-normwise and bound how many are set aside.
    gx = to_np(o["dLg_dx"]).astype(np.float64)
    keep = ref["kink_margin_fake"] > KINK
    err = np.abs(gx - ref["dL_dx"]).max(axis=1) / np.abs(ref["dL_dx"]).max(axis=1)
    print(f"  dLg_dx: {np.count_nonzero(~keep)} of {keep.size} events within {KINK:.0e} of a kink; "
          f"worst elementwise rel err there {err[~keep].max() if (~keep).any() else 0:.2e}, "
          f"elsewhere {err[keep].max():.2e}", flush=True)
    assert np.count_nonzero(~keep) <= max(3, 0.05 * keep.size)
    dtheta_ref = ref["dL_dtheta"]
    if (~keep).any() and W is not None:
        worst, matched = _check_near_kinks(gx, ref, W, b, np.flatnonzero(~keep), features)
        print(f"  near-kink events match an admissible slope choice: worst rel err {worst:.2e}", flush=True)
        # the per-parameter sums of the slope choices the computation took
        dtheta_ref, _ = oracle.param_grad(matched, ref["dxda"], ref["dxdb"], n_theta, E)
    assert_normwise(gx[keep], ref["dL_dx"][keep], TOL, "dLg_dx (away from kinks)")
    if fused:
        assert_normwise(to_np(o["dLg_dtheta"]), dtheta_ref, TOL, "dLg_dtheta")
        assert_condition_aware(to_np(o["dLg_dtheta"]), dtheta_ref, ref["dL_dtheta_cond"], TOL, "dLg_dtheta")


@pytest.mark.parametrize("name,n_theta,E", [
    ("pr1_tiny", None, None),      # full tiny workload
    ("small", 4, 2048),            # small-batch network on a reduced batch
    ("small", None, None),         # full small-batch workload (the benchmarked one)
])
def test_fused_source_path(gpu_ctx, name, n_theta, E):
    w = scaled(get(name), n_theta, E)
    print(f"case {name} n_theta={w.n_theta} E={w.events_per_theta}", flush=True)
    inp, th, ts, W, b, n_real = _setup(w)
    real = gpu_ctx.sample_events(ts, n_real, w.real_seed)
    o = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=w.events_per_theta,
                                                          seed=w.fake_seed))
    torch.cuda.synchronize()
    real_np = oracle.sample(inp["theta_star"], n_real, w.real_seed)
    ref = _oracle(inp, w, real_np)
    _check(o, ref, len(W), W=inp["W"], b=inp["b"], n_theta=w.n_theta, E=w.events_per_theta)


# The other compiled fp32 networks: width 64 with one to three hidden-to-hidden
# layers, width 128 with one, and d = 3 identity features at both widths; E =
# 1,000 (tiles straddling parameter rows, a partial last tile) and a ragged
# real batch.
@pytest.mark.parametrize("H,NH,d", [(64, 2, 2), (64, 3, 2), (128, 1, 2), (64, 1, 3), (64, 2, 3), (128, 2, 3)])
def test_other_fp32_networks(gpu_ctx, H, NH, d):
    from dataclasses import replace
    w = replace(get("small"), name=f"fp32_H{H}_NH{NH}_d{d}", n_theta=3, d=d, events_per_theta=1000,
                widths=(d,) + (H,) * (NH + 1) + (1,), theta_source="uniform")
    print(f"case {w.name} n_theta=3 E=1000 n_real=2500", flush=True)
    inp, th, ts, W, b, _ = _setup(w)
    real = gpu_ctx.sample_events(ts, 2500, w.real_seed)
    o = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=1000, seed=w.fake_seed))
    torch.cuda.synchronize()
    real_np = oracle.sample(inp["theta_star"], 2500, w.real_seed)
    ref = _oracle(inp, w, real_np)
    _check(o, ref, len(W), W=inp["W"], b=inp["b"], n_theta=w.n_theta, E=w.events_per_theta)


def test_three_call_path_matches_fused(gpu_ctx):
    """sample_events -> disc_fwd_bwd(fake_x) -> param_grad(BUFFER) equals the fused call."""
    w = scaled(get("small"), 4, 4096)
    inp, th, ts, W, b, n_real = _setup(w)
    real = gpu_ctx.sample_events(ts, n_real, w.real_seed)
    x = gpu_ctx.sample_events(th, w.events_per_theta, w.fake_seed)
    o3 = gpu_ctx.disc_fwd_bwd(W, b, real, fake_x=x)
    g3 = gpu_ctx.param_grad(th, w.events_per_theta, w.fake_seed, dL_dx=o3["dLg_dx"])
    of = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=w.events_per_theta,
                                                           seed=w.fake_seed))
    assert torch.equal(o3["logits_fake"], of["logits_fake"])
    assert torch.equal(o3["dLg_dx"], of["dLg_dx"])
    for l in range(len(W)):
        assert torch.equal(o3["dW"][l], of["dW"][l])
    real_np = oracle.sample(inp["theta_star"], n_real, w.real_seed)
    ref = _oracle(inp, w, real_np)
    assert_normwise(to_np(g3), ref["dL_dtheta"], TOL, "dLg_dtheta (3 calls)")


@pytest.mark.parametrize("n_theta,E,n_real", [(3, 1000, 2999), (1, 50, 64), (2, 64, 1)])
def test_ragged_sizes(gpu_ctx, n_theta, E, n_real):
    """E not a multiple of the 64-event tile (sample + buffer + reduce path) and odd real counts."""
    w = scaled(get("small"), n_theta, E)
    print(f"case ragged n_theta={n_theta} E={E} n_real={n_real}", flush=True)
    inp, th, ts, W, b, _ = _setup(w)
    real = gpu_ctx.sample_events(ts, n_real, w.real_seed)
    o = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=E, seed=w.fake_seed))
    torch.cuda.synchronize()
    real_np = oracle.sample(inp["theta_star"], n_real, w.real_seed)
    _check(o, _oracle(inp, w, real_np), len(W), W=inp["W"], b=inp["b"], n_theta=w.n_theta, E=w.events_per_theta)


def test_deterministic_repeat(gpu_ctx):
    w = scaled(get("small"), 8, 4096)
    inp, th, ts, W, b, n_real = _setup(w)
    real = gpu_ctx.sample_events(ts, n_real, w.real_seed)
    src = dict(theta=th, events_per_theta=w.events_per_theta, seed=w.fake_seed)
    o1 = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=src)
    o2 = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=src)
    for k in ("logits_fake", "logits_real", "loss_d", "loss_g", "dLg_dx", "dLg_dtheta"):
        assert torch.equal(o1[k], o2[k]), k
    for l in range(len(W)):
        assert torch.equal(o1["dW"][l], o2["dW"][l]) and torch.equal(o1["db"][l], o2["db"][l])


def test_zero_logit_layer(gpu_ctx):
    """With the logit layer zeroed: L_D = 2 ln 2, L_G = ln 2 and dL_G/dtheta = 0 exactly."""
    w = scaled(get("pr1_tiny"), 1, 4096)
    inp, th, ts, W, b, n_real = _setup(w)
    W[-1].zero_()
    b[-1].zero_()
    real = gpu_ctx.sample_events(ts, n_real, w.real_seed)
    o = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=w.events_per_theta,
                                                          seed=w.fake_seed))
    assert abs(o["loss_d"].item() - 2 * np.log(2)) < 1e-6 and abs(o["loss_g"].item() - np.log(2)) < 1e-6
    assert torch.count_nonzero(o["dLg_dtheta"]).item() == 0
    assert torch.count_nonzero(o["dLg_dx"]).item() == 0


@pytest.mark.parametrize("n_theta,E", [
    (None, None),    # the full paper shape: 1,024 x 100 events, tiles straddling parameter rows
    (7, 100),        # a partial last tile
    (3, 64),         # rows aligned with tiles
])
def test_paper_shape_proxy_pipeline(gpu_ctx, n_theta, E):
    """Six parameters -> three Kumaraswamy coordinates -> two observables ->
    2-128-128-128-128-1 discriminator, sampled inside the kernel."""
    w = scaled(get("paper"), n_theta, E)
    print(f"case paper n_theta={w.n_theta} E={w.events_per_theta}", flush=True)
    inp, th, ts, W, b, n_real = _setup(w)
    real = gpu_ctx.sample_events(ts, n_real, w.real_seed)
    o = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=w.events_per_theta,
                                                          seed=w.fake_seed), features=sg.FEAT_PROXY2)
    torch.cuda.synchronize()
    real_np = oracle.sample(inp["theta_star"], n_real, w.real_seed)
    ref = _oracle(inp, w, real_np)
    _check(o, ref, len(W), W=inp["W"], b=inp["b"], n_theta=w.n_theta, E=w.events_per_theta, features="proxy2")


def test_paper_shape_three_calls_match_fused(gpu_ctx):
    """sample_events -> disc_fwd_bwd(fake_x, PROXY2) -> param_grad(BUFFER) equals the fused call."""
    w = scaled(get("paper"), 16, 100)
    inp, th, ts, W, b, n_real = _setup(w)
    real = gpu_ctx.sample_events(ts, n_real, w.real_seed)
    x = gpu_ctx.sample_events(th, w.events_per_theta, w.fake_seed)
    o3 = gpu_ctx.disc_fwd_bwd(W, b, real, fake_x=x, features=sg.FEAT_PROXY2)
    g3 = gpu_ctx.param_grad(th, w.events_per_theta, w.fake_seed, dL_dx=o3["dLg_dx"])
    of = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=w.events_per_theta,
                                                           seed=w.fake_seed), features=sg.FEAT_PROXY2)
    assert torch.equal(o3["logits_fake"], of["logits_fake"])
    assert torch.equal(o3["dLg_dx"], of["dLg_dx"])
    for l in range(len(W)):
        assert torch.equal(o3["dW"][l], of["dW"][l])
    real_np = oracle.sample(inp["theta_star"], n_real, w.real_seed)
    ref = _oracle(inp, w, real_np)
    assert_normwise(to_np(g3), ref["dL_dtheta"], TOL, "dLg_dtheta (3 calls)")
    assert_normwise(to_np(of["dLg_dtheta"]), ref["dL_dtheta"], TOL, "dLg_dtheta (fused)")


def test_row_sharding_matches_full_run(gpu_ctx):
    """Two shards of the parameter rows, each with its own counter base, sample the
    same events as the full run; their dL_G/dtheta rows equal the full run's up to
    the 1/N of the mean (tiles straddle rows differently in each run)."""
    w = scaled(get("paper"), 10, 100)
    inp, th, ts, W, b, n_real = _setup(w)
    real = gpu_ctx.sample_events(ts, n_real, w.real_seed)
    kw = dict(features=sg.FEAT_PROXY2, want_grads=False, want_logits=False)
    full = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=100, seed=w.fake_seed), **kw)
    halves = []
    for r0, r1 in ((0, 5), (5, 10)):
        o = gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th[r0:r1].clone(), events_per_theta=100,
                                                             seed=w.fake_seed, counter_base=r0 * 100), **kw)
        halves.append(o["dLg_dtheta"] * 0.5)          # N_shard / N_full
        torch.testing.assert_close(o["dLg_dx"] * 0.5, full["dLg_dx"][r0 * 100:r1 * 100], rtol=1e-6, atol=0)
    torch.testing.assert_close(torch.cat(halves), full["dLg_dtheta"], rtol=2e-6, atol=1e-9)
