"""GPU parity of the bootstrap draw (sagips_bootstrap) against the oracle,
through the C ABI: drawn rows bit-exact, gathered values exact."""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2407_00051_amd as sg  # noqa: E402


@pytest.mark.parametrize("n_data,d,n_out,seed,step", [
    (1, 2, 100, 0, 0),                  # a single row
    (1000, 2, 777, 5, 3),               # ragged sizes
    (4096, 3, 10000, 7, 123456),        # d = 3, a power-of-two row count, more draws than rows
    (3_000_017, 2, 1_500_008, 2**40 + 11, 2**32 - 1),   # 64-bit seed, the largest step
])
def test_bootstrap_matches_oracle(gpu_ctx, n_data, d, n_out, seed, step):
    print(f"case bootstrap n_data={n_data} d={d} n_out={n_out}", flush=True)
    rng = np.random.default_rng(n_data)
    data_np = rng.standard_normal((n_data, d)).astype(np.float32)
    data = torch.tensor(data_np, device="cuda:0")
    out, idx = gpu_ctx.bootstrap(data, n_out, seed, step, want_idx=True)
    torch.cuda.synchronize()
    ref_idx = oracle.bootstrap_indices(n_data, n_out, seed, step)
    got = idx.cpu().numpy()
    assert np.array_equal(got, ref_idx), np.flatnonzero(got != ref_idx)[:10]
    assert np.array_equal(out.cpu().numpy(), data_np[ref_idx])


def test_bootstrap_full_size_sampled(gpu_ctx):
    """Medium-size reference data (8,388,608 events) and a 50% draw: every drawn
    row checked, at the launch configuration the benchmark times."""
    n_data, n_out = 1 << 23, 1 << 22
    data = torch.randn((n_data, 2), device="cuda:0")
    out, idx = gpu_ctx.bootstrap(data, n_out, 2024, 17, want_idx=True)
    torch.cuda.synchronize()
    ref_idx = oracle.bootstrap_indices(n_data, n_out, 2024, 17)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    assert torch.equal(out, data[torch.tensor(ref_idx, device="cuda:0")])
    # the variant without the index output (the one the benchmark times) draws the same rows
    assert torch.equal(gpu_ctx.bootstrap(data, n_out, 2024, 17), out)


def test_bootstrap_three_observable_full_size(gpu_ctx):
    """Three-observable reference data at full size (33,554,432 events, 16,777,216 draws)."""
    n_data, n_out = 1 << 25, 1 << 24
    data = torch.randn((n_data, 3), device="cuda:0")
    out = gpu_ctx.bootstrap(data, n_out, 99, 4)
    torch.cuda.synchronize()
    ref_idx = torch.tensor(oracle.bootstrap_indices(n_data, n_out, 99, 4), device="cuda:0")
    assert torch.equal(out, data[ref_idx])


def test_bootstrap_rejects_bad_arguments(gpu_ctx):
    data = torch.zeros((100, 2), device="cuda:0")
    with pytest.raises(sg.SagipsError):
        gpu_ctx.bootstrap(data, 0, 1, 1)
    with pytest.raises(ValueError):
        gpu_ctx.bootstrap(torch.zeros((100, 4), device="cuda:0"), 10, 1, 1)
    # out overlapping data is refused before any launch
    with pytest.raises(sg.SagipsError):
        gpu_ctx.bootstrap(data, 50, 1, 1, out=data[:50])


@pytest.mark.parametrize("n_data,d,n_out,seed,step", [
    (1, 2, 100, 0, 0),                  # one slab, one row drawn 100 times
    (1000, 2, 777, 5, 3),               # ragged
    (4096, 3, 10000, 7, 123456),        # more draws than rows
    (16384 * 3 + 5, 2, 70001, 11, 9),   # a partial last slab
    (3_000_017, 2, 1_500_008, 2**40 + 11, 2**32 - 1),
])
def test_bootstrap_row_order_matches_oracle(gpu_ctx, n_data, d, n_out, seed, step):
    print(f"case bootstrap rows n_data={n_data} d={d} n_out={n_out}", flush=True)
    rng = np.random.default_rng(n_data + 1)
    data_np = rng.standard_normal((n_data, d)).astype(np.float32)
    data = torch.tensor(data_np, device="cuda:0")
    out, idx = gpu_ctx.bootstrap(data, n_out, seed, step, want_idx=True, row_order=True)
    torch.cuda.synchronize()
    ref_x, ref_idx = oracle.bootstrap_row_order(data_np, n_out, seed, step)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    assert np.array_equal(out.cpu().numpy(), ref_x)


@pytest.mark.parametrize("n_data,d,n_out", [(1 << 23, 2, 1 << 22), (1 << 25, 3, 1 << 24)])
def test_bootstrap_row_order_full_size(gpu_ctx, n_data, d, n_out):
    """The benchmarked sizes: the row-order sample is the draw-order sample's
    multiset (per-row counts), in ascending order, with the rows' values."""
    data = torch.randn((n_data, d), device="cuda:0")
    out, idx = gpu_ctx.bootstrap(data, n_out, 31, 6, want_idx=True, row_order=True)
    _, draws = gpu_ctx.bootstrap(data, n_out, 31, 6, want_idx=True)
    assert torch.equal(torch.bincount(idx, minlength=n_data), torch.bincount(draws, minlength=n_data))
    assert bool((idx[1:] >= idx[:-1]).all())
    assert torch.equal(out, data[idx])
    # without the index output
    assert torch.equal(gpu_ctx.bootstrap(data, n_out, 31, 6, row_order=True), out)


def test_bootstrap_row_order_limits(gpu_ctx):
    data = torch.zeros((100, 2), device="cuda:0")
    big = torch.zeros(((1 << 27) + 1, 2), device="cuda:0")
    with pytest.raises(sg.SagipsError):
        gpu_ctx.bootstrap(big, 10, 1, 1, row_order=True)
    del big
    with pytest.raises(sg.SagipsError):
        gpu_ctx.bootstrap(data, 0, 1, 1, row_order=True)
