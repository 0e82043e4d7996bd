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

bf16 mode states where a bf16-operand / fp32-accumulate evaluation rounds
to bfloat16 (round to nearest even); everything else stays float64:
  * hidden-to-hidden weights, once;
  * the activations h_1 .. h_{n-1}, after bias and LeakyReLU;
  * the backward signals of the hidden layers, which carry a unit seed per
    event (backprop is linear in the seed): delta_{n-1} = w_o * leaky'(pre),
    then delta_{l-1} = (delta_l W_l) * leaky'(pre_{l-1});
  * the weight-gradient operand e_D * delta_l, rounded again after scaling.
The first layer and the logit layer keep float64 weights; dL/dx scales the
first-layer signal by e_G.
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


def logit_cond(W, b, hs):
    """Per event, the sum of |terms| of the logit: sum_o |W_L[0][o] h[o]| + |b_L|.

    The logit is a dot product over the last hidden layer; this is the scale
    against which a perturbation of its terms (for example by rounding the
    activations) is measured, as for the other condition sums."""
    wo = np.abs(np.asarray(W[-1], dtype=np.float64))[0]
    return np.abs(hs[-1]) @ wo + abs(float(np.asarray(b[-1], dtype=np.float64)[0]))


def input_grad_kink_variants(W, b, x, slope=0.2, margin=1e-5, max_units=6):
    """dz/dx of one event for every admissible choice of LeakyReLU slopes.

    Units whose pre-activation lies within `margin` of the kink (relative, as in
    kink_margin) may take either one-sided derivative, 1 or `slope`, in a
    computation with rounding errors; all other units follow the sign of their
    float64 pre-activation.  Returns an array [2^k][F] for the k (at most
    max_units, the closest ones) near-kink units: a computed input gradient of
    this event is correct if it matches one of the rows.  With k = 0 the single
    row is the plain float64 gradient."""
    n = len(W)
    W = [np.asarray(w, dtype=np.float64) for w in W]
    b = [np.asarray(v, dtype=np.float64) for v in b]
    h = np.asarray(x, dtype=np.float64)
    pres, rel = [], []
    for l in range(n - 1):
        pre = W[l] @ h + b[l]
        scale = np.abs(W[l]) @ np.abs(h) + np.abs(b[l])
        pres.append(pre)
        rel.append(np.abs(pre) / np.maximum(scale, 1e-300))
        h = _leaky(pre, slope)
    near = [(rel[l][o], l, o) for l in range(n - 1) for o in np.flatnonzero(rel[l] <= margin)]
    near = [(l, o) for _, l, o in sorted(near)[:max_units]]
    out = []
    for choice in range(1 << len(near)):
        grads = [_leaky_grad(p, slope) for p in pres]
        for bit, (l, o) in enumerate(near):
            grads[l][o] = 1.0 if (choice >> bit) & 1 else slope
        d = W[n - 1][0].copy()                    # dz/dh_{n-1}
        for l in range(n - 2, -1, -1):
            d = (d * grads[l]) @ W[l]             # dz/dh_l (h_0 = x)
        out.append(d)
    return np.array(out)


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


def _backward(W, pres, hs, g_z, slope, want_input_grad, cond=False):
    """Backprop a per-event logit gradient g_z through the network (float64).
    With cond, also the sums over events of |terms| of every dW and db entry,
    and (with want_input_grad) the per-entry sums of |terms| of the input
    gradient, sum_o |dL/dpre_0[o]| |W_1[o][j]|."""
    n = len(W)
    W = [np.asarray(w, dtype=np.float64) for w in W]
    dW = [None] * n
    db = [None] * n
    cW = [None] * n
    cb = [None] * n
    g = g_z[:, None]                       # dL/dpre of the logit layer
    g_in = None
    for l in range(n - 1, -1, -1):
        dW[l] = g.T @ hs[l]
        db[l] = g.sum(axis=0)
        if cond:
            cW[l] = np.abs(g).T @ np.abs(hs[l])
            cb[l] = np.abs(g).sum(axis=0)
        if l > 0:
            g = (g @ W[l]) * _leaky_grad(pres[l - 1], slope)
        elif want_input_grad:
            g_in = g @ W[0]
            if cond:
                c_in = np.abs(g) @ np.abs(W[0])
    if cond:
        return dW, db, g_in, cW, cb, (c_in if want_input_grad else None)
    return dW, db, g_in


def _disc_bf16(W, b, fake_in, real_in, slope, rnd, rnd_a=None, rnd_d=None, rnd_e=None):
    """disc_fwd_bwd with the bf16 rounding points of the module docstring.  `rnd`
    is the rounding map of the hidden weights (round_bf16, or the identity to
    check the structure); rnd_a, rnd_d and rnd_e, those of the activations, of
    the unit-seed signals and of the scaled weight-gradient operand (default:
    the same map), so that each point's share of the deviation from the float64
    network can be measured on its own."""
    n = len(W)
    rnd_a = rnd if rnd_a is None else rnd_a
    rnd_d = rnd if rnd_d is None else rnd_d
    rnd_e = rnd if rnd_e is None else rnd_e
    W = [np.asarray(w, dtype=np.float64) for w in W]
    b = [np.asarray(v, dtype=np.float64) for v in b]
    Wq = [rnd(w) if _hidden(l, n) else w for l, w in enumerate(W)]

    def fwd(h0):
        hs = [np.asarray(h0, dtype=np.float64)]
        for l in range(n - 1):
            hs.append(rnd_a(_leaky(hs[-1] @ Wq[l].T + b[l], slope)))
        return (hs[-1] @ W[-1].T + b[-1])[:, 0], hs

    z_f, hs_f = fwd(fake_in)
    z_r, hs_r = fwd(real_in)
    nf, nr = z_f.shape[0], z_r.shape[0]
    L_D, L_G = bce_losses(z_f, z_r)
    e = np.concatenate([sigmoid(z_f) / nf, -sigmoid(-z_r) / nr])
    eG = -sigmoid(-z_f) / nf
    hs = [np.concatenate([p, q]) for p, q in zip(hs_f, hs_r)]
    dW = [None] * n
    db = [None] * n
    dW[n - 1] = (e[:, None] * hs[n - 1]).sum(axis=0)[None, :]
    db[n - 1] = np.array([e.sum()])
    d = rnd_d(W[n - 1][0][None, :] * _leaky_grad(hs[n - 1], slope))     # unit-seed signal of layer n-2
    for l in range(n - 2, 0, -1):                                       # hidden-to-hidden layers
        dW[l] = rnd_e(e[:, None] * d).T @ hs[l]
        db[l] = (e[:, None] * d).sum(axis=0)
        d = rnd_d((d @ Wq[l]) * _leaky_grad(hs[l], slope))
    dW[0] = (e[:, None] * d).T @ hs[0]
    db[0] = (e[:, None] * d).sum(axis=0)
    g_in = eG[:, None] * (d[:nf] @ W[0])
    c_in = np.abs(eG)[:, None] * (np.abs(d[:nf]) @ np.abs(W[0]))
    return {
        "kink_margin_fake": np.full(nf, np.inf),
        "logits_fake": z_f, "logits_real": z_r, "loss_d": L_D, "loss_g": L_G,
        "dW": dW, "db": db, "dLg_din": g_in, "dLg_din_cond": c_in,
    }


def disc_fwd_bwd(W, b, fake_in, real_in, slope=0.2, bf16=False):
    """One discriminator forward + backward over a fake and a real batch.

    Returns a dict with logits_fake, logits_real, loss_d, loss_g, dW, db (of
    L_D) and dLg_din (dL_G / d fake input, [N][F]).
    """
    if bf16:
        return _disc_bf16(W, b, fake_in, real_in, slope, round_bf16)
    z_f, pres_f, hs_f = mlp_forward(W, b, fake_in, slope)
    z_r, pres_r, hs_r = mlp_forward(W, b, real_in, slope)
    nf, nr = z_f.shape[0], z_r.shape[0]
    L_D, L_G = bce_losses(z_f, z_r)
    # d softplus(t)/dt = sigmoid(t)
    gD_f = sigmoid(z_f) / nf
    gD_r = -sigmoid(-z_r) / nr
    gG_f = -sigmoid(-z_f) / nf
    dW_f, db_f, _, cW_f, cb_f, _ = _backward(W, pres_f, hs_f, gD_f, slope, False, cond=True)
    dW_r, db_r, _, cW_r, cb_r, _ = _backward(W, pres_r, hs_r, gD_r, slope, False, cond=True)
    _, _, g_in, _, _, c_in = _backward(W, pres_f, hs_f, gG_f, slope, True, cond=True)
    return {
        "kink_margin_fake": kink_margin(W, b, hs_f, pres_f),
        "logits_fake": z_f, "logits_real": z_r, "loss_d": L_D, "loss_g": L_G,
        "logits_fake_cond": logit_cond(W, b, hs_f), "logits_real_cond": logit_cond(W, b, hs_r),
        "dW": [p + q for p, q in zip(dW_f, dW_r)], "db": [p + q for p, q in zip(db_f, db_r)],
        "dW_cond": [p + q for p, q in zip(cW_f, cW_r)], "db_cond": [p + q for p, q in zip(cb_f, cb_r)],
        "dLg_din": g_in, "dLg_din_cond": c_in,
    }
