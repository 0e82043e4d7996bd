"""Bootstrapped sub-sampling of a rank's reference data (test infrastructure).

Sec. IV-B: every rank draws its training sub-samples from its data by
bootstrapping, i.e. uniformly with replacement, and feeds them through the
GAN.  Reading of the draw (the paper names no generator): draw i of a step
takes row

    idx_i = floor(w0 * n_data / 2^32)

where w0 is the first word of Philox4x32-10 under key (seed lo, seed hi) and
counter (i lo, i hi, stream, step).  Each step thus draws a fresh sub-sample
that depends only on (seed, step, i).  bootstrap_row_order lists the same
multiset in ascending row order.  floor(w0 * n / 2^32) maps the 2^32
equally likely words onto n rows, each row receiving floor or ceil of 2^32/n
words (exactly equal when n divides 2^32).
"""
from __future__ import annotations

import numpy as np

from .philox import philox4x32_10

STREAM_BOOTSTRAP = 4


def bootstrap_indices(n_data: int, n_out: int, seed: int, step: int, stream: int = STREAM_BOOTSTRAP) -> np.ndarray:
    """Row index of each of n_out draws (int64), exact integer arithmetic."""
    if not (1 <= n_data <= (1 << 32)):
        raise ValueError("n_data must be in [1, 2^32]")
    i = np.arange(n_out, dtype=np.uint64)
    ctr = np.empty((n_out, 4), dtype=np.uint64)
    ctr[:, 0] = i & np.uint64(0xFFFFFFFF)
    ctr[:, 1] = i >> np.uint64(32)
    ctr[:, 2] = np.uint64(stream & 0xFFFFFFFF)
    ctr[:, 3] = np.uint64(step & 0xFFFFFFFF)
    w0 = philox4x32_10(ctr, (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))[:, 0].astype(np.uint64)
    # w0 < 2^32 and n_data <= 2^32: the product is below 2^64, exact in uint64
    return ((w0 * np.uint64(n_data)) >> np.uint64(32)).astype(np.int64)


def bootstrap(data: np.ndarray, n_out: int, seed: int, step: int):
    """(data[idx], idx): the step's sub-sample of the rows of `data`."""
    idx = bootstrap_indices(data.shape[0], n_out, seed, step)
    return data[idx], idx


def bootstrap_row_order(data: np.ndarray, n_out: int, seed: int, step: int):
    """The same sub-sample as a multiset listed in ascending row order: row r
    appears as often as it was drawn.  A batch used as a whole (a mean loss,
    summed gradients) does not depend on the order of its rows."""
    idx = np.sort(bootstrap_indices(data.shape[0], n_out, seed, step), kind="stable")
    return data[idx], idx
