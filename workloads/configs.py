"""The five synthetic workloads of the single-rank step.

Shapes follow the paper's step (Sec. V-A, Tab. gen_settings: a batch of
parameter samples, a fixed number of events per sample, an equal-sized real
batch) scaled to MI355X sizes.  Each workload is a frozen description; the
arrays are drawn by :mod:`workloads.gen`.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    n_theta: int                 # parameter samples per step
    d: int                       # observables per event (2 or 3); theta has 2d entries
    events_per_theta: int        # E
    widths: Optional[Tuple[int, ...]]   # discriminator widths incl. input and the 1-wide logit; None = quadratic critic
    precision: str               # "f32" or "bf16" (hidden-layer GEMM operands)
    features: str                # "identity" or "hd8"
    theta_source: str            # "uniform" (U(1,6)) or "generator" (16->64->64->4 MLP)
    theta_seed: int = 0
    fake_seed: int = 0           # Philox key of the fake events
    real_seed: int = 1           # Philox key of the real events
    weight_seed: int = 2
    generator_seed: int = 3

    @property
    def n_events(self) -> int:
        return self.n_theta * self.events_per_theta

    @property
    def n_params(self) -> int:
        return 2 * self.d

    @property
    def theta_star(self) -> Tuple[float, ...]:
        # (a1,b1,a2,b2) as the workload states; the third pair for d=3 is a
        # chosen value (the paper names no distribution at all).
        return (2.0, 5.0, 1.5, 3.0) if self.d == 2 else (2.0, 5.0, 1.5, 3.0, 3.0, 2.0)

    def mlp_macs(self) -> int:
        """Multiply-accumulates per sample through the discriminator."""
        if self.widths is None:
            return 0
        return sum(a * b for a, b in zip(self.widths[:-1], self.widths[1:]))


CONFIGS = {
    "pr1_tiny": Workload("pr1_tiny", 1, 2, 16384, (2, 64, 64, 1), "f32", "identity", "uniform"),
    "small": Workload("small", 32, 2, 8192, (2, 128, 128, 128, 1), "f32", "identity", "generator"),
    "medium": Workload("medium", 256, 2, 16384, (2, 256, 256, 256, 256, 1), "bf16", "identity", "uniform"),
    "higher_dim": Workload("higher_dim", 1024, 3, 16384, (8, 512, 512, 512, 512, 1), "bf16", "hd8", "uniform"),
    "stress": Workload("stress", 64, 2, 4194304, None, "f32", "identity", "uniform"),
    # the paper's own step shape (Sec. V-A, Tab. gen_settings): 1,024 parameter samples of six
    # parameters x 100 events, the 2-128-128-128-128-1 discriminator on two observables
    "paper": Workload("paper", 1024, 3, 100, (2, 128, 128, 128, 128, 1), "f32", "proxy2", "uniform"),
}


@dataclass(frozen=True)
class BootstrapWorkload:
    """One step's bootstrap draw of the real batch from a rank's data (Sec. IV-B).

    The pool holds twice the step's real batch and each step draws half of
    it, with replacement; the pool's events are Kumaraswamy draws at
    theta_star, resident in HBM before the step."""
    name: str
    n_data: int                  # events in the rank's pool
    d: int
    n_out: int                   # draws per step
    seed: int = 5                # Philox key of the draws
    pool_seed: int = 1           # Philox key of the pool's events
    row_order: bool = False      # the same multiset in ascending row order

    @property
    def theta_star(self) -> Tuple[float, ...]:
        return (2.0, 5.0, 1.5, 3.0) if self.d == 2 else (2.0, 5.0, 1.5, 3.0, 3.0, 2.0)


BOOTSTRAP_CONFIGS = {
    # the real batch of the 256 x 16,384-event step, drawn from a pool of twice its size
    "bootstrap": BootstrapWorkload("bootstrap", 2 * 4194304, 2, 4194304),
    # the real batch of the 1,024 x 16,384-event three-observable step
    "bootstrap_d3": BootstrapWorkload("bootstrap_d3", 2 * 16777216, 3, 16777216),
    # the same draws listed in ascending row order (a counting sort by pool slab)
    "bootstrap_rows": BootstrapWorkload("bootstrap_rows", 2 * 4194304, 2, 4194304, row_order=True),
    "bootstrap_rows_d3": BootstrapWorkload("bootstrap_rows_d3", 2 * 16777216, 3, 16777216, row_order=True),
}


@dataclass(frozen=True)
class EnsembleWorkload:
    """Ensemble response of M generators on a batch of k noise vectors (Sec. VI-A).

    The paper's generator is 6-128-128-128-128-6 (51,206 parameters); its
    ensembles hold 20 members, one of them 100, and each generator predicts
    1,024 parameter samples per step."""
    name: str
    n_members: int
    k: int
    widths: Tuple[int, ...] = (6, 128, 128, 128, 128, 6)
    weight_seed: int = 21
    noise_seed: int = 22

    @property
    def theta_star(self) -> Tuple[float, ...]:
        return (2.0, 5.0, 1.5, 3.0, 3.0, 2.0)


ENSEMBLE_CONFIGS = {
    "ensemble": EnsembleWorkload("ensemble", 100, 1024),
}


@dataclass(frozen=True)
class TrainWorkload:
    """One GAN training step of the loop-closure test at the paper's shape
    (Sec. V-A, Tab. gen_settings): the generator predicts k = 1,024 parameter
    samples, each yields E = 100 events, the discriminator sees the two
    observables of those and of an equal reference batch, bootstrapped each
    step from a pool of twice its size (Sec. IV-B, Sec. VI-C)."""
    name: str
    k: int = 1024
    events_per_theta: int = 100
    g_widths: Tuple[int, ...] = (6, 128, 128, 128, 128, 6)
    d_widths: Tuple[int, ...] = (2, 128, 128, 128, 128, 1)
    seed: int = 0

    @property
    def n_events(self) -> int:
        return self.k * self.events_per_theta

    @property
    def theta_star(self) -> Tuple[float, ...]:
        return (2.0, 5.0, 1.5, 3.0, 3.0, 2.0)


TRAIN_CONFIGS = {"train": TrainWorkload("train")}


def get(name: str):
    for table in (CONFIGS, BOOTSTRAP_CONFIGS, ENSEMBLE_CONFIGS, TRAIN_CONFIGS):
        if name in table:
            return table[name]
    raise KeyError(name)


def scaled(w: Workload, n_theta: Optional[int] = None, events_per_theta: Optional[int] = None) -> Workload:
    """Same workload with fewer parameter samples or events (parity-size cases)."""
    from dataclasses import replace
    return replace(w, n_theta=n_theta or w.n_theta, events_per_theta=events_per_theta or w.events_per_theta)
