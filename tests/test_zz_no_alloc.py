"""The no-allocation discriminator step (sagips_disc_fwd_bwd_noalloc) against the
allocating one, through the C ABI: same kernels, workspace from the library's
fixed per-device scratch instead of a hipMalloc'd one.  Two calls in a row, the
second on a smaller input, must each equal the allocating call's outputs."""
import numpy as np
import pytest

from workloads import gen, get
from workloads.configs import scaled

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2407_00051_amd as sg  # noqa: E402


def _inputs(w, n_real):
    inp = gen.make_inputs(w)
    dev = "cuda:0"
    t = lambda a: torch.tensor(a, device=dev)     # noqa: E731
    return t(inp["theta"]), t(inp["theta_star"]), [t(m) for m in inp["W"]], [t(v) for v in inp["b"]]


def _outputs(W, b, n_fake, n_real, d, n_theta):
    f32 = dict(dtype=torch.float32, device="cuda:0")
    nan = float("nan")
    return {"logits_fake": torch.full((n_fake,), nan, **f32), "logits_real": torch.full((n_real,), nan, **f32),
            "loss_d": torch.full((1,), nan, **f32), "loss_g": torch.full((1,), nan, **f32),
            "dW": [torch.full_like(m, nan) for m in W], "db": [torch.full_like(v, nan) for v in b],
            "dLg_dx": torch.full((n_fake, d), nan, **f32), "dLg_dtheta": torch.full((n_theta, 2 * d), nan, **f32)}


def _step(ctx, w, th, ts, W, b, n_real, no_alloc):
    real = ctx.sample_events(ts, n_real, w.real_seed)
    prec = sg.BF16 if w.precision == "bf16" else sg.F32
    feats = {"identity": sg.FEAT_IDENTITY, "hd8": sg.FEAT_HD8, "proxy2": sg.FEAT_PROXY2}[w.features]
    outs = _outputs(W, b, w.n_events, n_real, w.d, w.n_theta)
    torch.cuda.synchronize()
    o = ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=th, events_per_theta=w.events_per_theta, seed=w.fake_seed),
                         precision=prec, features=feats, outputs=outs, no_alloc=no_alloc)
    torch.cuda.synchronize()
    return o


def _same(a, b):
    for k in ("logits_fake", "logits_real", "loss_d", "loss_g", "dLg_dx", "dLg_dtheta"):
        assert torch.equal(a[k], b[k]), k
    for l in range(len(a["dW"])):
        assert torch.equal(a["dW"][l], b["dW"][l]) and torch.equal(a["db"][l], b["db"][l]), l


@pytest.mark.parametrize("calls", [
    # fused fp32 step (the small-batch network), then a smaller batch of it
    [("small", 32, 2048, 65536), ("small", 3, 700, 1500)],
    # the paper's network on its observables, then fewer rows; then the split path
    # (E < 64: events sampled into the scratch, dL/dtheta reduced afterwards)
    [("paper", 1024, 100, 102400), ("paper", 40, 50, 1000)],
    # the small-batch network with a second call larger than the first's tiles
    [("small", 1, 64, 64), ("small", 16, 4096, 65536)],
])
def test_noalloc_matches_allocating_call(gpu_ctx, calls):
    for name, n_theta, E, n_real in calls:
        w = scaled(get(name), n_theta, E)
        print(f"case {name} n_theta={n_theta} E={E} n_real={n_real}", flush=True)
        th, ts, W, b = _inputs(w, n_real)
        ref = _step(gpu_ctx, w, th, ts, W, b, n_real, no_alloc=False)
        got = _step(gpu_ctx, w, th, ts, W, b, n_real, no_alloc=True)
        assert not torch.isnan(got["logits_fake"]).any()
        _same(got, ref)


@pytest.mark.parametrize("name,n_theta,E,n_real", [
    ("medium", 2, 300, 500),          # bf16 at width 256: the weight-gradient partials alone are 67 MB
    ("small", 8192, 8192, 65536),     # fp32 with 2^26 fake events: the per-tile partials exceed the scratch
])
def test_noalloc_rejects_a_workspace_beyond_the_scratch(gpu_ctx, name, n_theta, E, n_real):
    """A call whose workspace exceeds the scratch is rejected before launch, its
    outputs untouched."""
    lib = sg.load_library()
    assert lib.sagips_noalloc_scratch_bytes() == 64 << 20
    w = scaled(get(name), n_theta, E)
    th, ts, W, b = _inputs(scaled(get(name), 2, 64), 64)
    theta = torch.full((n_theta, 2 * w.d), 2.0, dtype=torch.float32, device="cuda:0")
    real = torch.full((n_real, w.d), 0.5, dtype=torch.float32, device="cuda:0")
    outs = _outputs(W, b, w.n_events, n_real, w.d, n_theta)
    prec = sg.BF16 if w.precision == "bf16" else sg.F32
    torch.cuda.synchronize()
    with pytest.raises(sg.SagipsError) as ei:
        gpu_ctx.disc_fwd_bwd(W, b, real, fake_source=dict(theta=theta, events_per_theta=E, seed=0),
                             precision=prec, outputs=outs, no_alloc=True)
    assert ei.value.status == sg.E_INVAL and "no-allocation" in str(ei.value)
    torch.cuda.synchronize()
    assert torch.isnan(outs["logits_fake"]).all() and torch.isnan(outs["dW"][1]).all()
    assert torch.isnan(outs["dLg_dtheta"]).all()
