"""Optimiser step for the generator and the discriminator (test infrastructure).

Sec. V-A gives the learning rates (generator 1e-5, discriminator 1e-4) but not
the optimiser.  Reading: Adam (Kingma and Ba, ICLR 2015, Algorithm 1) with
beta1 = 0.9, beta2 = 0.999, eps = 1e-8 and no weight decay, the defaults of
the PyTorch the paper ran on.  For step t = 1, 2, ... and gradient g:

  m <- beta1 m + (1 - beta1) g
  v <- beta2 v + (1 - beta2) g^2
  p <- p - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)

Pins (tests/test_oracle_optim.py): torch.optim.Adam in float64 over several
steps, and the first step's closed form lr * g / (|g| + eps).
"""
from __future__ import annotations

import numpy as np

BETA1, BETA2, EPS = 0.9, 0.999, 1e-8


def adam_step(p, g, m, v, t: int, lr: float, beta1: float = BETA1, beta2: float = BETA2, eps: float = EPS):
    """One Adam step on arrays of any shape; returns (p, m, v) as new float64 arrays."""
    p = np.asarray(p, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    return p - lr * m_hat / (np.sqrt(v_hat) + eps), m, v
