"""GAN generator as the optimiser, and the ensemble response (test infrastructure).

Generator (Sec. III: the optimiser is a GAN generator that maps random noise
to parameters; Sec. V-A: LeakyReLU hidden layers, 51,206 trainable
parameters).  The widths follow from that count: 6 -> 128 -> 128 -> 128 ->
128 -> 6 gives (6*128+128) + 3*(128*128+128) + (128*6+6) = 51,206.  Readings
(the paper is silent on them): noise n ~ N(0, 1)^6, LeakyReLU slope 0.2, and
the output passed through 1 + softplus so that every Kumaraswamy shape
parameter is above 1.

  h_0 = n;  h_l = LeakyReLU(h_{l-1} W_l^T + b_l) for the hidden layers;
  o = h W_out^T + b_out;  theta = 1 + softplus(o).

Ensemble response (Sec. VI-A, eqs. def_ens_mean and def_ens_std): for one
noise vector n and M generators G_i,
  p_hat = (1/M) sum_i G_i(n),   sigma = sqrt((1/M) sum_i (G_i(n) - p_hat)^2),
and for a batch of k noise vectors both are averaged over the batch.  The
normalised residual of eq. def_param_res is r_i = (p_i - p_hat_i) / p_i.

Pins (tests/test_oracle_generator.py): forward against torch float64
modules, backward against torch autograd and finite differences, the
ensemble against its M = 1, identical-member and M = 2 closed forms and
numpy's population standard deviation.
"""
from __future__ import annotations

import numpy as np

from .mlp import softplus, sigmoid

G_WIDTHS = (6, 128, 128, 128, 128, 6)


def _leaky(t, s):
    return np.where(t > 0, t, s * t)


def generator_forward(W, b, noise, slope=0.2, return_all=False):
    """theta[k][P] = 1 + softplus(G(noise)); with return_all also the
    pre-activations and activations of every layer (float64)."""
    h = np.asarray(noise, dtype=np.float64)
    hs, pres = [h], []
    L = len(W)
    for l in range(L):
        pre = h @ np.asarray(W[l], dtype=np.float64).T + np.asarray(b[l], dtype=np.float64)
        pres.append(pre)
        h = _leaky(pre, slope) if l < L - 1 else pre
        hs.append(h)
    theta = 1.0 + softplus(h)
    if not return_all:
        return theta
    return {"theta": theta, "pres": pres, "hs": hs}


def generator_backward(W, b, noise, dL_dtheta, slope=0.2):
    """dL/dW_l and dL/db_l for a given dL/dtheta[k][P] (chain rule through
    1 + softplus, whose derivative is sigmoid, and the LeakyReLU layers)."""
    f = generator_forward(W, b, noise, slope, return_all=True)
    L = len(W)
    g = np.asarray(dL_dtheta, dtype=np.float64) * sigmoid(f["pres"][-1])
    dW, db = [None] * L, [None] * L
    for l in range(L - 1, -1, -1):
        dW[l] = g.T @ f["hs"][l]
        db[l] = g.sum(axis=0)
        if l > 0:
            g = (g @ np.asarray(W[l], dtype=np.float64)) * np.where(f["pres"][l - 1] > 0, 1.0, slope)
    return dW, db


def ensemble_response(thetas):
    """thetas[M][k][P] (member i's prediction for noise vector n): returns
    (p_hat[P], sigma[P]), each averaged over the k noise vectors."""
    t = np.asarray(thetas, dtype=np.float64)
    M = t.shape[0]
    p_hat = t.sum(axis=0) / M                          # [k][P]
    sigma = np.sqrt(((t - p_hat) ** 2).sum(axis=0) / M)
    return p_hat.mean(axis=0), sigma.mean(axis=0)


def residual(p_true, p_hat):
    """Normalised residual r_i = (p_i - p_hat_i) / p_i."""
    p = np.asarray(p_true, dtype=np.float64)
    return (p - np.asarray(p_hat, dtype=np.float64)) / p
