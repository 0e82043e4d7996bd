"""Pin of the oracle's bf16 discriminator mode by an independent route.

The oracle writes the bf16-operand backward out by hand.  Here the same
network runs through torch float64 autograd instead, with two
straight-through functions placing the roundings: one rounds a value in the
forward pass (activations, hidden weights) and one rounds the gradient that
flows back through a pre-activation (the unit-seed signal of every layer).
Autograd supplies the chain itself (transposes, LeakyReLU slopes, the input
gradient), so a dropped rounding point, a transposed operand or a wrong slope
in the oracle shows up as a mismatch.  The weight gradients are then the
e_D-weighted sums of the captured signals, bf16(e_D delta)^T h for the hidden
layers (the rounding of the weight-gradient operand).
"""
import numpy as np
import pytest
import torch

from oracle.mlp import disc_fwd_bwd


class _RoundValue(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        return x.to(torch.bfloat16).to(torch.float64)

    @staticmethod
    def backward(ctx, g):
        return g


class _RoundGrad(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return g.to(torch.bfloat16).to(torch.float64)


def _bf16(x):
    return x.to(torch.bfloat16).to(torch.float64)


def _autograd_disc(W, b, xf, xr, slope=0.2):
    n = len(W)
    Wt = [torch.tensor(w, dtype=torch.float64) for w in W]
    bt = [torch.tensor(v, dtype=torch.float64) for v in b]
    Wq = [_RoundValue.apply(w) if 0 < l < n - 1 else w for l, w in enumerate(Wt)]

    def run(x_np):
        x = torch.tensor(x_np, dtype=torch.float64, requires_grad=True)
        h = x
        ins, pres = [], []
        for l in range(n - 1):
            ins.append(h.detach())
            raw = h @ Wq[l].T + bt[l]
            raw.retain_grad()
            pres.append(raw)
            h = _RoundValue.apply(torch.nn.functional.leaky_relu(_RoundGrad.apply(raw), slope))
        ins.append(h.detach())
        z = (h @ Wt[-1].T + bt[-1])[:, 0]
        z.backward(torch.ones_like(z))           # unit seed per event
        deltas = [p.grad for p in pres]            # rounded unit-seed signal of each layer
        return z.detach(), ins, deltas, x.grad

    zf, ins_f, d_f, gx = run(xf)
    zr, ins_r, d_r, _ = run(xr)
    nf, nr = zf.shape[0], zr.shape[0]
    sp = torch.nn.functional.softplus
    loss_d = sp(zf).mean() + sp(-zr).mean()
    loss_g = sp(-zf).mean()
    e = torch.cat([torch.sigmoid(zf) / nf, -torch.sigmoid(-zr) / nr])
    eG = -torch.sigmoid(-zf) / nf
    ins = [torch.cat([p, q]) for p, q in zip(ins_f, ins_r)]
    dl = [torch.cat([p, q]) for p, q in zip(d_f, d_r)]
    dW, db = [None] * n, [None] * n
    dW[n - 1] = (e[:, None] * ins[n - 1]).sum(0)[None, :]
    db[n - 1] = e.sum()[None]
    for l in range(n - 1):
        s = e[:, None] * dl[l]
        dW[l] = (_bf16(s) if l > 0 else s).T @ ins[l]
        db[l] = s.sum(0)
    return {"logits_fake": zf, "logits_real": zr, "loss_d": loss_d, "loss_g": loss_g,
            "dW": dW, "db": db, "dLg_din": eG[:, None] * gx}


def _case(widths, n, seed):
    rng = np.random.default_rng(seed)
    W = [rng.uniform(-1, 1, (o, i)) * np.sqrt(6.0 / (i + o)) for i, o in zip(widths[:-1], widths[1:])]
    b = [rng.uniform(-1, 1, o) / np.sqrt(i) for i, o in zip(widths[:-1], widths[1:])]
    xf = rng.uniform(0.0, 1.0, (n, widths[0]))
    xr = rng.uniform(0.0, 1.0, (n + 5, widths[0]))
    return W, b, xf, xr


def _rel(p, t):
    p, t = np.asarray(p, np.float64), np.asarray(t, np.float64)
    return np.linalg.norm(p - t) / max(np.linalg.norm(t), 1e-300)


@pytest.mark.parametrize("widths,n,seed", [((2, 32, 32, 32, 1), 200, 1), ((8, 48, 48, 48, 48, 1), 150, 2),
                                           ((3, 16, 1), 100, 3)])
def test_bf16_mode_matches_autograd_with_rounding_points(widths, n, seed):
    W, b, xf, xr = _case(widths, n, seed)
    q = disc_fwd_bwd(W, b, xf, xr, bf16=True)
    a = {k: (v.numpy() if torch.is_tensor(v) else v) for k, v in _autograd_disc(W, b, xf, xr).items()}
    # Both sides are float64 with roundings at the same points; sums are formed
    # in different orders, so a value sitting on a bf16 rounding boundary may
    # round differently (one element moves by 2^-8 relative).  Such flips are
    # rare: the tensors agree to far below the bf16 step.
    tol = 1e-9
    for k in ("logits_fake", "logits_real", "dLg_din"):
        assert _rel(q[k], a[k]) < tol, k
    assert abs(q["loss_d"] - float(a["loss_d"])) < 1e-12
    assert abs(q["loss_g"] - float(a["loss_g"])) < 1e-12
    for l in range(len(W)):
        assert _rel(q["dW"][l], a["dW"][l].numpy()) < tol, ("dW", l)
        assert _rel(q["db"][l], a["db"][l].numpy()) < tol, ("db", l)


def test_autograd_route_detects_a_missing_rounding_point():
    """Self-check of the pin: dropping the rounding of the signal changes the result
    far beyond the tolerance used above."""
    W, b, xf, xr = _case((2, 32, 32, 32, 1), 200, 1)
    q = disc_fwd_bwd(W, b, xf, xr, bf16=True)
    orig = _RoundGrad.backward
    try:
        _RoundGrad.backward = staticmethod(lambda ctx, g: g)
        a = _autograd_disc(W, b, xf, xr)
    finally:
        _RoundGrad.backward = orig
    assert _rel(q["dLg_din"], a["dLg_din"].numpy()) > 1e-4
