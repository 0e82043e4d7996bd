"""Differentiable inverse-CDF event sampler (paper Sec. V-A: the proxy
pipeline samples events with the inverse CDF of a differentiable
one-dimensional distribution) for the Kumaraswamy(a, b) family.

  CDF       F(x; a, b) = 1 - (1 - x^a)^b,            0 < x < 1
  quantile  x(u; a, b) = (1 - (1 - u)^(1/b))^(1/a)

Each observable j of an event uses its own pair (a_j, b_j) = (theta[2j],
theta[2j+1]) and its own uniform u_j, taken from Philox word j.
"""
from __future__ import annotations

import numpy as np

from .philox import event_words


def uniform_from_words(w: np.ndarray) -> np.ndarray:
    """u = ((w >> 9) + 1/2) * 2^-23: the centre of one of 2^23 equal cells of
    (0, 1).  Exact in float32 (2m+1 < 2^24), never 0 or 1, and 1-u is exact."""
    m = (np.asarray(w, dtype=np.uint64) >> np.uint64(9)).astype(np.float64)
    return (m + 0.5) * 2.0 ** -23


def kumaraswamy_cdf(x, a, b):
    return 1.0 - (1.0 - x ** a) ** b


def kumaraswamy_icdf(u, a, b):
    """The quantile function, evaluated literally in float64."""
    return (1.0 - (1.0 - u) ** (1.0 / b)) ** (1.0 / a)


def pathwise(x, a, b):
    """Reparameterisation derivatives dx/da and dx/db at fixed u.

    Implicit-function form: F(x(u; a, b); a, b) = u gives
    dx/dtheta = -(dF/dtheta) / (dF/dx), i.e.
      dx/da = -x ln(x) / a
      dx/db = (1 - x^a) ln(1 - x^a) / (a b x^(a-1)).
    """
    xa = x ** a
    dxda = -x * np.log(x) / a
    dxdb = (1.0 - xa) * np.log1p(-xa) / (a * b * x ** (a - 1.0))
    return dxda, dxdb


def _ids(n_theta, E, counter_base):
    return np.uint64(counter_base) + np.arange(n_theta * E, dtype=np.uint64)


def sample(theta: np.ndarray, E: int, seed: int, counter_base: int = 0, stream: int = 0,
           return_all: bool = False):
    """Events x[n_theta*E][d] for theta[n_theta][2d], event id = base + i*E + k.

    Returns x (float64), and with return_all also the words, u and the pathwise
    derivatives dx/da, dx/db (each [N][d]).
    """
    theta = np.asarray(theta, dtype=np.float64)
    n_theta, P = theta.shape
    d = P // 2
    words = event_words(seed, _ids(n_theta, E, counter_base), stream)
    u = uniform_from_words(words[:, :d])
    a = np.repeat(theta[:, 0::2], E, axis=0)
    b = np.repeat(theta[:, 1::2], E, axis=0)
    x = kumaraswamy_icdf(u, a, b)
    if not return_all:
        return x
    dxda, dxdb = pathwise(x, a, b)
    return {"words": words, "u": u, "x": x, "dxda": dxda, "dxdb": dxdb, "a": a, "b": b}


def features_hd8(x: np.ndarray) -> np.ndarray:
    """Eight observables from a 3D event: [x1, x2, x3, x1x2, x2x3, x1x3,
    ln x1, ln(1 - x3)]."""
    x1, x2, x3 = x[:, 0], x[:, 1], x[:, 2]
    return np.stack([x1, x2, x3, x1 * x2, x2 * x3, x1 * x3, np.log(x1), np.log1p(-x3)], axis=1)


def features_hd8_jacobian(x: np.ndarray) -> np.ndarray:
    """d features / d x, [N][8][3]."""
    x1, x2, x3 = x[:, 0], x[:, 1], x[:, 2]
    J = np.zeros((x.shape[0], 8, 3))
    J[:, 0, 0] = 1
    J[:, 1, 1] = 1
    J[:, 2, 2] = 1
    J[:, 3, 0], J[:, 3, 1] = x2, x1
    J[:, 4, 1], J[:, 4, 2] = x3, x2
    J[:, 5, 0], J[:, 5, 2] = x3, x1
    J[:, 6, 0] = 1.0 / x1
    J[:, 7, 2] = -1.0 / (1.0 - x3)
    return J


def features_proxy2(x: np.ndarray) -> np.ndarray:
    """The two observables of the paper-shape pipeline (Sec. V: six parameters
    in, two observables out; the mapping itself is not given).  Reading: three
    independent Kumaraswamy draws, one per parameter pair, share the third
    draw:  y0 = x1 + x3,  y1 = x2 + x3.  By Kotlarski's lemma the joint law of
    (y0, y1) identifies the laws of x1, x2 and x3 up to a common shift, which
    their common support (0, 1) removes, so the six parameters stay
    recoverable."""
    return np.stack([x[:, 0] + x[:, 2], x[:, 1] + x[:, 2]], axis=1)


def features_proxy2_jacobian(x: np.ndarray) -> np.ndarray:
    """d(y0, y1) / d(x1, x2, x3), [N][2][3]."""
    J = np.zeros((x.shape[0], 2, 3))
    J[:, 0, 0] = 1.0
    J[:, 0, 2] = 1.0
    J[:, 1, 1] = 1.0
    J[:, 1, 2] = 1.0
    return J
