"""Discriminator objective (paper Sec. II-B.2 and Sec. III-A: a binary
classifier trained to label reference events 1 and synthetic events 0; its
hidden layers use LeakyReLU, Sec. V-A) with a binary cross-entropy loss,
forward and backward, in float64.

Network: h_0 = input features; for each hidden layer l,
pre_l = h_{l-1} W_l^T + b_l and h_l = LeakyReLU_s(pre_l); the last layer
gives the logit z = h W^T + b with no activation (the class probability is
sigmoid(z)).  Weights use the torch.nn.Linear layout W_l[out][in].

Losses (means over each batch):
  L_D = mean_real softplus(-z) + mean_fake softplus(z)
  L_G = mean_fake softplus(-z)            (non-saturating generator loss)
The backward pass returns dL_D/dW_l, dL_D/db_l and dL_G/d(input) of the fake
events, the gradient that flows back through the sampler to theta.

bf16 mode mirrors where a bf16-operand / fp32-accumulate implementation
rounds: hidden-layer weights, the activations h_1 .. h_{n-1} (after bias and
LeakyReLU) and the hidden-layer backward signals are rounded to bf16
(round-to-nearest-even); everything else stays float64.
"""
from __future__ import annotations

import numpy as np


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even), returned as float64."""
    f = np.asarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = np.nan
    return out


def _leaky(t, s):
    return np.where(t > 0, t, s * t)


def _leaky_grad(t, s):
    return np.where(t > 0, 1.0, s)


def softplus(t):
    return np.maximum(t, 0.0) + np.log1p(np.exp(-np.abs(t)))


def sigmoid(t):
    return 0.5 * (1.0 + np.tanh(0.5 * t))


def _hidden(l, n_layers):
    """Layer l (0-based) is a hidden-to-hidden GEMM layer (not the first, not the logit)."""
    return 0 < l < n_layers - 1


def kink_margin(W, b, hs, pres):
    """Per event, the smallest relative distance of any hidden pre-activation
    from the LeakyReLU kink: min over units of |pre| / (sum_k |W h_k| + |b|).

    LeakyReLU (Sec. V-A) has a jump in its derivative at 0, so the backward
    signal of an event whose margin is at rounding level depends on which side
    of 0 a given precision lands; such events are not comparable elementwise
    between an fp32 and a float64 evaluation."""
    n = len(W)
    m = np.full(hs[0].shape[0], np.inf)
    for l in range(n - 1):
        scale = np.abs(hs[l]) @ np.abs(np.asarray(W[l], dtype=np.float64)).T + np.abs(np.asarray(b[l], dtype=np.float64))
        m = np.minimum(m, (np.abs(pres[l]) / np.maximum(scale, 1e-300)).min(axis=1))
    return m


def mlp_forward(W, b, h0, slope=0.2, bf16=False):
    """Returns (z[N], pres, hs) where hs[0] is the input and hs[l+1] = act(pres[l])."""
    n = len(W)
    W = [np.asarray(w, dtype=np.float64) for w in W]
    b = [np.asarray(v, dtype=np.float64) for v in b]
    if bf16:
        W = [round_bf16(w) if _hidden(l, n) else w for l, w in enumerate(W)]
    hs = [np.asarray(h0, dtype=np.float64)]
    pres = []
    for l in range(n):
        pre = hs[-1] @ W[l].T + b[l]
        pres.append(pre)
        if l < n - 1:
            h = _leaky(pre, slope)
            if bf16:
                h = round_bf16(h)
            hs.append(h)
    return pres[-1][:, 0], pres, hs


def bce_losses(z_fake, z_real):
    """(L_D, L_G) for the logits of the fake and the real batch."""
    L_D = softplus(-z_real).mean() + softplus(z_fake).mean()
    L_G = softplus(-z_fake).mean()
    return L_D, L_G


def _backward(W, pres, hs, g_z, slope, bf16, want_input_grad):
    """Backprop a per-event logit gradient g_z through the network."""
    n = len(W)
    W = [np.asarray(w, dtype=np.float64) for w in W]
    if bf16:
        W = [round_bf16(w) if _hidden(l, n) else w for l, w in enumerate(W)]
    dW = [None] * n
    db = [None] * n
    g = g_z[:, None]                       # dL/dpre of the logit layer
    g_in = None
    for l in range(n - 1, -1, -1):
        if bf16 and _hidden(l, n):
            g = round_bf16(g)
        dW[l] = g.T @ hs[l]
        db[l] = g.sum(axis=0)
        if l > 0:
            g = (g @ W[l]) * _leaky_grad(pres[l - 1], slope)
        elif want_input_grad:
            g_in = g @ W[0]
    return dW, db, g_in


def disc_fwd_bwd(W, b, fake_in, real_in, slope=0.2, bf16=False):
    """One discriminator forward + backward over a fake and a real batch.

    Returns a dict with logits_fake, logits_real, loss_d, loss_g, dW, db (of
    L_D) and dLg_din (dL_G / d fake input, [N][F]).
    """
    z_f, pres_f, hs_f = mlp_forward(W, b, fake_in, slope, bf16)
    z_r, pres_r, hs_r = mlp_forward(W, b, real_in, slope, bf16)
    nf, nr = z_f.shape[0], z_r.shape[0]
    L_D, L_G = bce_losses(z_f, z_r)
    # d softplus(t)/dt = sigmoid(t)
    gD_f = sigmoid(z_f) / nf
    gD_r = -sigmoid(-z_r) / nr
    gG_f = -sigmoid(-z_f) / nf
    dW_f, db_f, _ = _backward(W, pres_f, hs_f, gD_f, slope, bf16, False)
    dW_r, db_r, _ = _backward(W, pres_r, hs_r, gD_r, slope, bf16, False)
    _, _, g_in = _backward(W, pres_f, hs_f, gG_f, slope, bf16, True)
    return {
        "kink_margin_fake": kink_margin(W, b, hs_f, pres_f),
        "logits_fake": z_f, "logits_real": z_r, "loss_d": L_D, "loss_g": L_G,
        "dW": [p + q for p, q in zip(dW_f, dW_r)], "db": [p + q for p, q in zip(db_f, db_r)],
        "dLg_din": g_in,
    }
