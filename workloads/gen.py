"""Seeded input draws (numpy PCG64), shared by the oracle tests and the HIP path.

Nothing here is part of the step being measured: theta is the step's input,
the discriminator weights are its parameters.  All draws are float64 and are
rounded once to float32, the storage type of the step's inputs.
"""
from __future__ import annotations

import numpy as np

from .configs import Workload


def theta_uniform(n_theta: int, d: int, seed: int = 0) -> np.ndarray:
    """theta[n_theta][2d] ~ U(1, 6), ordered (a1, b1, a2, b2[, a3, b3])."""
    rng = np.random.default_rng(seed)
    return (1.0 + 5.0 * rng.random((n_theta, 2 * d))).astype(np.float32)


def _leaky(t, slope=0.2):
    return np.where(t > 0, t, slope * t)


def theta_from_generator(n_theta: int, d: int, seed: int = 3) -> np.ndarray:
    """theta from a 16->64->64->2d generator MLP fed N(0,1) noise.

    The generator is the optimiser of the paper's GAN (Sec. III): LeakyReLU
    hidden layers, Kaiming-normal weights, zero biases; the output goes
    through 1 + softplus so every shape parameter is >= 1.  Computed in
    float64 and rounded once to float32.
    """
    rng = np.random.default_rng(seed)
    noise = rng.standard_normal((n_theta, 16))
    widths = (16, 64, 64, 2 * d)
    gain = np.sqrt(2.0 / (1.0 + 0.2 ** 2))
    h = noise
    for li, (fi, fo) in enumerate(zip(widths[:-1], widths[1:])):
        w = rng.standard_normal((fo, fi)) * (gain / np.sqrt(fi))
        h = h @ w.T
        if li < len(widths) - 2:
            h = _leaky(h)
    out = np.logaddexp(0.0, h)
    return (1.0 + out).astype(np.float32)


def xavier_mlp(widths, seed: int = 2):
    """Discriminator weights in torch.nn.Linear layout.

    W[l] is [widths[l+1]][widths[l]] ~ Xavier-uniform (gain 1); b[l] ~
    U(-1/sqrt(fan_in), 1/sqrt(fan_in)) so that every bias path carries a
    non-zero value.  Drawn layer by layer, weight then bias, float32.
    """
    rng = np.random.default_rng(seed)
    Ws, bs = [], []
    for fi, fo in zip(widths[:-1], widths[1:]):
        bound = np.sqrt(6.0 / (fi + fo))
        Ws.append(rng.uniform(-bound, bound, (fo, fi)).astype(np.float32))
        bb = 1.0 / np.sqrt(fi)
        bs.append(rng.uniform(-bb, bb, (fo,)).astype(np.float32))
    return Ws, bs


def generator_stack(widths, n_members: int, seed: int = 21, slope: float = 0.2):
    """Parameters of n_members generators, stacked member-major: W[l] is
    [M][out][in] ~ Kaiming-normal for LeakyReLU(slope) (the paper's init,
    Sec. V-A), b[l] is [M][out] ~ U(-1/sqrt(fan_in), 1/sqrt(fan_in)).  float32."""
    rng = np.random.default_rng(seed)
    gain = np.sqrt(2.0 / (1.0 + slope ** 2))
    Ws, bs = [], []
    for fi, fo in zip(widths[:-1], widths[1:]):
        Ws.append((rng.standard_normal((n_members, fo, fi)) * (gain / np.sqrt(fi))).astype(np.float32))
        bs.append(rng.uniform(-1.0 / np.sqrt(fi), 1.0 / np.sqrt(fi), (n_members, fo)).astype(np.float32))
    return Ws, bs


def noise(k: int, dim: int, seed: int = 22) -> np.ndarray:
    """Generator input noise [k][dim] ~ N(0, 1), float32."""
    return np.random.default_rng(seed).standard_normal((k, dim)).astype(np.float32)


def make_inputs(w: Workload) -> dict:
    """All seeded inputs of one workload: theta, theta*, weights and seeds."""
    if w.theta_source == "generator":
        theta = theta_from_generator(w.n_theta, w.d, w.generator_seed)
    else:
        theta = theta_uniform(w.n_theta, w.d, w.theta_seed)
    out = {
        "theta": theta,
        "theta_star": np.asarray(w.theta_star, dtype=np.float32).reshape(1, -1),
        "fake_seed": w.fake_seed,
        "real_seed": w.real_seed,
        "events_per_theta": w.events_per_theta,
    }
    if w.widths is not None:
        out["W"], out["b"] = xavier_mlp(w.widths, w.weight_seed)
    return out
