"""Pins tests/fullsize_reference.py (the torch float64 restatement used for the
full-size reduced outputs of the bf16 workloads) to the oracle, on the CPU:
both evaluations (the float64 network and its bf16 rounding points), several
network depths and input widths, ragged batches and chunk sizes that split
them unevenly."""
import numpy as np
import pytest

import oracle
from tests import fullsize_reference as ref
from workloads import gen

torch = pytest.importorskip("torch")


def _net(widths, seed):
    W, b = gen.xavier_mlp(widths, seed)
    return [np.asarray(w, dtype=np.float64) for w in W], [np.asarray(v, dtype=np.float64) for v in b]


@pytest.mark.parametrize("widths,nf,nr,chunk", [
    ((2, 16, 16, 16, 1), 300, 257, 64),
    ((8, 32, 32, 32, 32, 1), 200, 211, 77),
    ((3, 16, 16, 1), 50, 49, 1000),
])
@pytest.mark.parametrize("bf16", [False, True])
def test_matches_oracle(widths, nf, nr, chunk, bf16):
    W, b = _net(widths, 5)
    rng = np.random.default_rng(11)
    F = widths[0]
    fake = rng.random((nf, F))
    real = rng.random((nr, F))
    o = oracle.disc_fwd_bwd(W, b, fake, real, bf16=bf16)
    r = ref.reduced_outputs(W, b, fake, real, bf16=bf16, chunk=chunk)
    assert abs(r["loss_d"] - o["loss_d"]) <= 1e-12 * abs(o["loss_d"])
    assert abs(r["loss_g"] - o["loss_g"]) <= 1e-12 * abs(o["loss_g"])
    for l in range(len(W)):
        for got, want, what in ((r["dW"][l], o["dW"][l], "dW"), (r["db"][l], o["db"][l], "db")):
            got = got.numpy()
            scale = np.abs(want).max()
            assert np.max(np.abs(got - want)) <= 1e-11 * scale, (what, l)
        if not bf16:
            np.testing.assert_allclose(r["dW_cond"][l].numpy(), o["dW_cond"][l], rtol=1e-12)
            np.testing.assert_allclose(r["db_cond"][l].numpy(), o["db_cond"][l], rtol=1e-12)


def test_round_bf16_matches_oracle():
    x = np.random.default_rng(0).standard_normal(100_000) * np.exp(np.random.default_rng(1).uniform(-30, 30, 100_000))
    assert np.array_equal(ref.round_bf16(torch.tensor(x)).numpy(), oracle.round_bf16(x))


def test_chunking_invariance():
    """The sums do not depend on where the batch is split (up to float64 rounding)."""
    W, b = _net((2, 16, 16, 1), 3)
    rng = np.random.default_rng(4)
    fake, real = rng.random((500, 2)), rng.random((480, 2))
    a = ref.reduced_outputs(W, b, fake, real, bf16=True, chunk=500)
    c = ref.reduced_outputs(W, b, fake, real, bf16=True, chunk=37)
    for l in range(len(W)):
        np.testing.assert_allclose(a["dW"][l].numpy(), c["dW"][l].numpy(), rtol=1e-12, atol=1e-15)
