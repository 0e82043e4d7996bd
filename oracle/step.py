"""The step end to end: theta -> events -> [features] -> discriminator ->
BCE -> backward -> dL/dtheta (paper Sec. II: parameters p pass through the
pipeline to an objective whose gradient reaches p by backpropagation through
every differentiable module).

The per-parameter reduction is the chain rule through the sampler:
  dL/da_j(i) = sum over events k of sample i of dL/dx_{k,j} * dx_{k,j}/da_j
and likewise for b_j.  For the quadratic critic L = sum (x - 1/2)^2 over all
events and coordinates, dL/dx = 2 (x - 1/2).
"""
from __future__ import annotations

import numpy as np

from .mlp import disc_fwd_bwd
from .sampler import features_hd8, features_hd8_jacobian, features_proxy2, features_proxy2_jacobian, sample

FEATURES = {"hd8": (features_hd8, features_hd8_jacobian),
            "proxy2": (features_proxy2, features_proxy2_jacobian)}


def param_grad(dL_dx: np.ndarray, dxda: np.ndarray, dxdb: np.ndarray, n_theta: int, E: int):
    """dL/dtheta[n_theta][2d] and the condition sums sum|terms| of each entry."""
    N, d = dL_dx.shape
    ta = (dL_dx * dxda).reshape(n_theta, E, d)
    tb = (dL_dx * dxdb).reshape(n_theta, E, d)
    g = np.empty((n_theta, 2 * d))
    c = np.empty((n_theta, 2 * d))
    g[:, 0::2], g[:, 1::2] = ta.sum(axis=1), tb.sum(axis=1)
    c[:, 0::2], c[:, 1::2] = np.abs(ta).sum(axis=1), np.abs(tb).sum(axis=1)
    return g, c


def quadratic_critic(x: np.ndarray):
    """L = sum (x - 1/2)^2 and dL/dx."""
    return float(((x - 0.5) ** 2).sum()), 2.0 * (x - 0.5)


def run_step(theta, E, fake_seed, W=None, b=None, real_x=None, features="identity",
             bf16=False, slope=0.2, counter_base=0, critic=None):
    """Whole step.  With critic="quadratic" the discriminator is replaced by the
    quadratic critic.  Returns a dict of every intermediate the GPU path exposes."""
    theta = np.asarray(theta, dtype=np.float64)
    n_theta = theta.shape[0]
    s = sample(theta, E, fake_seed, counter_base, return_all=True)
    out = dict(s)
    if critic == "quadratic":
        loss, g = quadratic_critic(s["x"])
        out["loss"] = loss
        out["dL_dx"] = g
    else:
        if features == "identity":
            fin, rin = s["x"], real_x
        else:
            fmap = FEATURES[features][0]
            fin, rin = fmap(s["x"]), fmap(real_x)
        r = disc_fwd_bwd(W, b, fin, rin, slope, bf16)
        out.update(r)
        if features == "identity":
            g, gc = r["dLg_din"], r["dLg_din_cond"]
        else:
            J = FEATURES[features][1](s["x"])
            g = np.einsum("nf,nfd->nd", r["dLg_din"], J)
            gc = np.einsum("nf,nfd->nd", r["dLg_din_cond"], np.abs(J))
        out["dL_dx"] = g
        out["dL_dx_cond"] = gc       # per entry: sum of |terms| (through |Jacobian| for mapped features)
    out["dL_dtheta"], out["dL_dtheta_cond"] = param_grad(out["dL_dx"], s["dxda"], s["dxdb"], n_theta, E)
    return out
