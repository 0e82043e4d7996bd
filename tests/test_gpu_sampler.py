"""GPU parity of the sampler and of the per-parameter gradient reduction
against the CPU oracle, through the C ABI."""
import numpy as np
import pytest

import oracle
from oracle.sampler import uniform_from_words
from tests.parity import assert_condition_aware, assert_normwise, max_rel, to_np, words_np
from workloads import gen, get

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _theta(n, d, seed=0):
    return torch.tensor(gen.theta_uniform(n, d, seed), device="cuda:0")


@pytest.mark.parametrize("n_theta,E,d,seed,base,stream", [
    (1, 16384, 2, 0, 0, 0),                 # the tiny workload's fake events
    (3, 1000, 2, 7, 2**32 - 1500, 0),       # ragged E, counter crosses the lo/hi carry
    (2, 777, 3, 2**40 + 5, 123, 3),         # d = 3, large seed, stream != 0
])
def test_words_bit_exact_and_events(gpu_ctx, n_theta, E, d, seed, base, stream):
    print(f"case n_theta={n_theta} E={E} d={d} seed={seed} base={base}", flush=True)
    th = _theta(n_theta, d, 5)
    x, w = gpu_ctx.sample_events(th, E, seed, counter_base=base, stream=stream, want_words=True)
    torch.cuda.synchronize()
    ref = oracle.sample(th.cpu().numpy(), E, seed, base, stream, return_all=True)
    assert np.array_equal(words_np(w), ref["words"])
    # u is exact on both sides, so the words pin u; events to 1e-5 elementwise
    e = max_rel(to_np(x), ref["x"])
    print(f"  events max rel err {e:.2e}", flush=True)
    assert e <= 1e-5


def test_unit_theta_events_equal_u(gpu_ctx):
    """a = b = 1 is the identity quantile; the fp32 log/exp evaluation stays within the events bar of u."""
    th = torch.ones((2, 4), device="cuda:0")
    x, w = gpu_ctx.sample_events(th, 4096, 9, want_words=True)
    u = uniform_from_words(words_np(w)[:, :2])
    e = max_rel(to_np(x), u)
    print(f"  a=b=1 events vs u: max rel err {e:.2e}", flush=True)
    assert e <= 1e-5


def test_stress_full_size_sampled_events(gpu_ctx):
    """The bandwidth-stress workload at full size (64 x 4,194,304 events): words
    and events of 200k randomly chosen events against the oracle, one by one."""
    w = get("stress")
    th = torch.tensor(gen.make_inputs(w)["theta"], device="cuda:0")
    x, words = gpu_ctx.sample_events(th, w.events_per_theta, w.fake_seed, want_words=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    idx = np.unique(np.concatenate([rng.integers(0, w.n_events, 200_000), [0, w.n_events - 1]]))
    ti = torch.tensor(idx, device="cuda:0")
    gx = to_np(x[ti])
    gw = words_np(words[ti])
    rw = oracle.event_words(w.fake_seed, idx.astype(np.uint64))
    assert np.array_equal(gw, rw)
    thn = th.cpu().numpy().astype(np.float64)
    rows = idx // w.events_per_theta
    u = uniform_from_words(rw[:, :2])
    rx = oracle.kumaraswamy_icdf(u, thn[rows][:, 0::2], thn[rows][:, 1::2])
    e = max_rel(gx, rx)
    print(f"  sampled events max rel err {e:.2e}", flush=True)
    assert e <= 1e-5


def test_sharding_invariance(gpu_ctx):
    """Two calls over halves of the rows (counter_base offset) give the same words and events."""
    th = _theta(4, 2, 1)
    E = 5000
    x, w = gpu_ctx.sample_events(th, E, 3, want_words=True)
    x0, w0 = gpu_ctx.sample_events(th[:2].contiguous(), E, 3, want_words=True)
    x1, w1 = gpu_ctx.sample_events(th[2:].contiguous(), E, 3, counter_base=2 * E, want_words=True)
    assert torch.equal(torch.cat([w0, w1]), w) and torch.equal(torch.cat([x0, x1]), x)


@pytest.mark.parametrize("n_theta,E,d", [(8, 65536, 2), (5, 10007, 2), (3, 4099, 3), (1, 1, 2)])
def test_param_grad_quadratic(gpu_ctx, n_theta, E, d):
    print(f"case quadratic n_theta={n_theta} E={E} d={d}", flush=True)
    th = _theta(n_theta, d, 2)
    g, loss = gpu_ctx.param_grad(th, E, 4)
    ref = oracle.run_step(th.cpu().numpy(), E, 4, critic="quadratic")
    assert_normwise(to_np(g), ref["dL_dtheta"], 1e-4, "dL/dtheta")
    assert_condition_aware(to_np(g), ref["dL_dtheta"], ref["dL_dtheta_cond"], 1e-4, "dL/dtheta")
    assert abs(float(loss.item()) - ref["loss"]) <= 1e-4 * abs(ref["loss"])


def test_param_grad_buffer(gpu_ctx):
    th = _theta(6, 2, 3)
    E = 3001
    rng = np.random.default_rng(1)
    gx = rng.standard_normal((6 * E, 2)).astype(np.float32)
    g = gpu_ctx.param_grad(th, E, 11, dL_dx=torch.tensor(gx, device="cuda:0"), counter_base=99)
    s = oracle.sample(th.cpu().numpy(), E, 11, 99, return_all=True)
    ref, cond = oracle.param_grad(gx.astype(np.float64), s["dxda"], s["dxdb"], 6, E)
    assert_normwise(to_np(g), ref, 1e-4, "dL/dtheta")
    assert_condition_aware(to_np(g), ref, cond, 1e-4, "dL/dtheta")


def test_stress_full_size_param_grad_rows(gpu_ctx):
    """Full bandwidth-stress workload; rows 0 and 63 (4,194,304 events each) checked against the oracle."""
    w = get("stress")
    th = torch.tensor(gen.make_inputs(w)["theta"], device="cuda:0")
    g, loss = gpu_ctx.param_grad(th, w.events_per_theta, w.fake_seed)
    g = to_np(g)
    thn = th.cpu().numpy()
    for row in (0, w.n_theta - 1):
        ref = oracle.run_step(thn[row:row + 1], w.events_per_theta, w.fake_seed, critic="quadratic",
                              counter_base=row * w.events_per_theta)
        assert_normwise(g[row], ref["dL_dtheta"][0], 1e-4, f"row {row}")
        assert_condition_aware(g[row:row + 1], ref["dL_dtheta"], ref["dL_dtheta_cond"], 1e-4, f"row {row}")


def test_deterministic_repeat(gpu_ctx):
    th = _theta(4, 2, 4)
    a, la = gpu_ctx.param_grad(th, 100000, 5)
    b, lb = gpu_ctx.param_grad(th, 100000, 5)
    assert torch.equal(a, b) and torch.equal(la, lb)


def test_stress_full_size_loss_and_gradient_statistics(gpu_ctx):
    """The whole bandwidth-stress step (64 x 4,194,304 events): the loss over all
    2^28 events and every parameter row's dL/dtheta against their expectations
    from the Kumaraswamy moments E[X^n] = b B(1 + n/a, b) (and their derivatives
    through the digamma function), within 6 standard errors.  The loss's standard
    error comes from the fourth moment; each gradient component's from the
    per-event terms of the oracle on 16,384 events of its row.  A property of the
    full-size output that holds at any size; the oracle itself pins two rows
    exactly (test above)."""
    from scipy import special
    w = get("stress")
    thn = gen.make_inputs(w)["theta"].astype(np.float64)
    th = torch.tensor(gen.make_inputs(w)["theta"], device="cuda:0")
    g, loss = gpu_ctx.param_grad(th, w.events_per_theta, w.fake_seed)
    g, loss = to_np(g).astype(np.float64), float(loss.item())
    E = w.events_per_theta
    a, b = thn[:, 0::2], thn[:, 1::2]                       # [rows][d]

    def m(n):
        return b * special.beta(1 + n / a, b)

    def dm(n):
        r = m(n)
        da = r * (-n / a**2) * (special.digamma(1 + n / a) - special.digamma(1 + n / a + b))
        db = r * (1 / b + special.digamma(b) - special.digamma(1 + n / a + b))
        return da, db
    q2 = m(2) - m(1) + 0.25                                 # E[(X - 1/2)^2]
    q4 = m(4) - 2 * m(3) + 1.5 * m(2) - 0.5 * m(1) + 1 / 16  # E[(X - 1/2)^4]
    EL, sdL = E * q2.sum(), np.sqrt(E * (q4 - q2**2).sum())
    zL = (loss - EL) / sdL
    print(f"  loss {loss:.9e}, expectation {EL:.9e} (standard error {sdL:.3e}): {zL:+.2f} s.e.", flush=True)
    assert abs(zL) <= 6.0
    (d2a, d2b), (d1a, d1b) = dm(2), dm(1)
    Eg = np.empty_like(g)
    Eg[:, 0::2], Eg[:, 1::2] = E * (d2a - d1a), E * (d2b - d1b)   # d E[L_row] / d(a_j, b_j)
    n_sub = 16384
    sd = np.empty_like(g)
    for r in range(w.n_theta):
        s = oracle.sample(thn[r:r + 1], n_sub, w.fake_seed, counter_base=r * E, return_all=True)
        t = 2.0 * (s["x"] - 0.5)
        sd[r, 0::2] = np.std(t * s["dxda"], axis=0, ddof=1)
        sd[r, 1::2] = np.std(t * s["dxdb"], axis=0, ddof=1)
    z = (g - Eg) / (sd * np.sqrt(E))
    print(f"  dL/dtheta: {g.size} components, largest |deviation| {np.abs(z).max():.2f} s.e.", flush=True)
    assert np.abs(z).max() <= 6.0
