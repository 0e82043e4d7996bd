"""GPU parity of the generator (forward, backward) and of the ensemble response
against the oracle, through the C ABI."""
import numpy as np
import pytest

import oracle
from tests.parity import assert_normwise, to_np
from workloads import gen, get

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2407_00051_amd as sg  # noqa: E402

TOL = 1e-4
KINK = 1e-4    # relative pre-activation margin below which fp32 and fp64 may take different LeakyReLU slopes
WIDTHS = (6, 128, 128, 128, 128, 6)


def _dev(arrs):
    return [torch.tensor(a, device="cuda:0") for a in arrs]


def _member(W, b, m):
    return [w[m].astype(np.float64) for w in W], [v[m].astype(np.float64) for v in b]


def _kink_rows(W, b, n, slope=0.2):
    """Rows whose hidden pre-activations come within KINK (relative to the sum of
    absolute terms) of the LeakyReLU kink, for one member."""
    h = n.astype(np.float64)
    near = np.zeros(n.shape[0], dtype=bool)
    for l in range(len(W) - 1):
        pre = h @ W[l].T + b[l]
        scale = np.abs(h) @ np.abs(W[l]).T + np.abs(b[l])
        near |= (np.abs(pre) <= KINK * scale).any(axis=1)
        h = np.where(pre > 0, pre, slope * pre)
    return near


@pytest.mark.parametrize("M,k", [(1, 1), (3, 100), (2, 1000), (100, 1024)])
def test_gen_forward_matches_oracle(gpu_ctx, M, k):
    print(f"case gen_forward M={M} k={k}", flush=True)
    W, b = gen.generator_stack(WIDTHS, M, seed=M + k)
    n = gen.noise(k, WIDTHS[0], seed=k)
    th = gpu_ctx.gen_forward(_dev(W), _dev(b), torch.tensor(n, device="cuda:0"))
    torch.cuda.synchronize()
    got = to_np(th)
    for m in range(M):
        ref = oracle.generator_forward(*_member(W, b, m), n)
        err = np.abs(got[m] - ref).max() / np.abs(ref).max()
        assert err <= TOL, (m, err)


@pytest.mark.parametrize("M,k", [(1, 1024), (2, 333), (1, 64), (1, 1)])
def test_gen_backward_matches_oracle(gpu_ctx, M, k):
    """dW, db of sum <g, theta> for a random g; rows near a LeakyReLU kink get g = 0
    (several slopes are correct there), so both sides sum the same rows."""
    print(f"case gen_backward M={M} k={k}", flush=True)
    W, b = gen.generator_stack(WIDTHS, M, seed=7 * M + k)
    n = gen.noise(k, WIDTHS[0], seed=k + 1)
    g = np.random.default_rng(k).standard_normal((M, k, WIDTHS[-1])).astype(np.float32)
    for m in range(M):
        g[m, _kink_rows(*_member(W, b, m), n)] = 0.0
    dW, db = gpu_ctx.gen_backward(_dev(W), _dev(b), torch.tensor(n, device="cuda:0"), torch.tensor(g, device="cuda:0"))
    torch.cuda.synchronize()
    for m in range(M):
        rW, rb = oracle.generator_backward(*_member(W, b, m), n, g[m].astype(np.float64))
        for l in range(len(W)):
            assert_normwise(to_np(dW[l])[m], rW[l], TOL, f"dW[{l}] member {m}")
            assert_normwise(to_np(db[l])[m], rb[l], TOL, f"db[{l}] member {m}")


# The other compiled generator depths (one and two hidden-to-hidden layers) and
# other input/output widths (up to 8), forward and backward.
@pytest.mark.parametrize("widths,M,k", [((4, 128, 128, 2), 3, 300), ((8, 128, 128, 128, 8), 2, 1000),
                                        ((1, 128, 128, 128, 5), 1, 77)])
def test_gen_other_shapes(gpu_ctx, widths, M, k):
    print(f"case gen widths={widths} M={M} k={k}", flush=True)
    W, b = gen.generator_stack(widths, M, seed=len(widths) + k)
    n = gen.noise(k, widths[0], seed=k + 2)
    nd = torch.tensor(n, device="cuda:0")
    th = to_np(gpu_ctx.gen_forward(_dev(W), _dev(b), nd))
    g = np.random.default_rng(k).standard_normal((M, k, widths[-1])).astype(np.float32)
    for m in range(M):
        g[m, _kink_rows(*_member(W, b, m), n)] = 0.0
    dW, db = gpu_ctx.gen_backward(_dev(W), _dev(b), nd, torch.tensor(g, device="cuda:0"))
    torch.cuda.synchronize()
    for m in range(M):
        ref = oracle.generator_forward(*_member(W, b, m), n)
        assert np.abs(th[m] - ref).max() / np.abs(ref).max() <= TOL, m
        rW, rb = oracle.generator_backward(*_member(W, b, m), n, g[m].astype(np.float64))
        for l in range(len(W)):
            assert_normwise(to_np(dW[l])[m], rW[l], TOL, f"dW[{l}] member {m}")
            assert_normwise(to_np(db[l])[m], rb[l], TOL, f"db[{l}] member {m}")


def test_gen_backward_zero_signal(gpu_ctx):
    W, b = gen.generator_stack(WIDTHS, 1, seed=3)
    n = torch.tensor(gen.noise(200, 6, seed=4), device="cuda:0")
    dW, db = gpu_ctx.gen_backward(_dev(W), _dev(b), n, torch.zeros((1, 200, 6), device="cuda:0"))
    assert all(torch.count_nonzero(t).item() == 0 for t in dW + db)


@pytest.mark.parametrize("M,k", [(1, 50), (2, 77), (20, 1024), (100, 1024)])
def test_ensemble_response_matches_oracle(gpu_ctx, M, k):
    print(f"case ensemble M={M} k={k}", flush=True)
    W, b = gen.generator_stack(WIDTHS, M, seed=M)
    n = gen.noise(k, WIDTHS[0], seed=M + 1)
    p_true = np.array([2.0, 5.0, 1.5, 3.0, 3.0, 2.0], dtype=np.float32)
    o = gpu_ctx.ensemble_response(_dev(W), _dev(b), torch.tensor(n, device="cuda:0"),
                                  p_true=torch.tensor(p_true, device="cuda:0"))
    torch.cuda.synchronize()
    th = np.stack([oracle.generator_forward(*_member(W, b, m), n) for m in range(M)])
    p_hat, sigma = oracle.ensemble_response(th)
    r_hat = oracle.residual(p_true, p_hat)
    np.testing.assert_allclose(to_np(o["p_hat"]), p_hat, rtol=TOL)
    if M == 1:
        assert torch.count_nonzero(o["sigma"]).item() == 0
    else:
        np.testing.assert_allclose(to_np(o["sigma"]), sigma, rtol=TOL, atol=TOL * np.abs(p_hat).max())
    np.testing.assert_allclose(to_np(o["r_hat"]), r_hat, atol=TOL * np.abs(p_hat / p_true).max())


def test_ensemble_identical_members_have_no_spread(gpu_ctx):
    W, b = gen.generator_stack(WIDTHS, 1, seed=5)
    W7 = [np.repeat(w, 7, axis=0) for w in W]
    b7 = [np.repeat(v, 7, axis=0) for v in b]
    n = torch.tensor(gen.noise(300, 6, seed=6), device="cuda:0")
    o = gpu_ctx.ensemble_response(_dev(W7), _dev(b7), n)
    single = gpu_ctx.ensemble_response(_dev(W), _dev(b), n)
    assert (o["sigma"] <= 1e-6 * o["p_hat"]).all()
    torch.testing.assert_close(o["p_hat"], single["p_hat"], rtol=1e-6, atol=0)


def test_ensemble_workload_full_size(gpu_ctx):
    """The benchmarked ensemble: 100 members of the paper's generator, 1,024 noise vectors."""
    w = get("ensemble")
    W, b = gen.generator_stack(w.widths, w.n_members, w.weight_seed)
    n = gen.noise(w.k, w.widths[0], w.noise_seed)
    o = gpu_ctx.ensemble_response(_dev(W), _dev(b), torch.tensor(n, device="cuda:0"))
    th = np.stack([oracle.generator_forward(*_member(W, b, m), n) for m in range(w.n_members)])
    p_hat, sigma = oracle.ensemble_response(th)
    np.testing.assert_allclose(to_np(o["p_hat"]), p_hat, rtol=TOL)
    np.testing.assert_allclose(to_np(o["sigma"]), sigma, rtol=TOL)


def test_generator_rejects_bad_arguments(gpu_ctx):
    import ctypes
    W, b = gen.generator_stack((6, 96, 96, 6), 1, seed=1)     # unsupported hidden width
    n = torch.zeros((10, 6), device="cuda:0")
    with pytest.raises(sg.SagipsError):
        gpu_ctx.gen_forward(_dev(W), _dev(b), n)
    # several members need a [M][k][out] signal
    W2, b2 = gen.generator_stack(WIDTHS, 2, seed=1)
    with pytest.raises(ValueError):
        gpu_ctx.gen_backward(_dev(W2), _dev(b2), n, torch.zeros((10, 6), device="cuda:0"))
    # p_true without r_hat is refused before any launch
    W, b = _dev(gen.generator_stack(WIDTHS, 1, seed=1)[0]), _dev(gen.generator_stack(WIDTHS, 1, seed=1)[1])
    g, _ = gpu_ctx._gen(W, b, 0.2)
    pt = torch.ones(6, device="cuda:0")
    ph = torch.empty(6, device="cuda:0")
    st = gpu_ctx.lib.sagips_ensemble_response(gpu_ctx.h, ctypes.byref(g), n.data_ptr(), 10, pt.data_ptr(),
                                              ph.data_ptr(), ph.data_ptr(), None)
    assert st == sg.E_INVAL
