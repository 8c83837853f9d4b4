"""fp64 oracle of the batch-SOM update that follows the search (test
infrastructure).

What it computes (paper, Section 3: after the best-matching unit of every
document is found, that unit and its neighbours are updated; Section 6.1,
Table 4, splits the update into a scatter into accumulators, a neighbourhood
blur, a write-back of the codebook and a norms refresh).  The paper defers the
neighbourhood function and its schedule to its companion paper, so this module
states a reading, the textbook batch map:

  * accumulate, over every searched document d with best unit b_d and feature
    set S_d:  acc[f, b_d] += 1 for f in S_d,  count[b_d] += 1;
  * neighbourhood on the rows x cols grid (neuron j at row j // cols, column
    j % cols), a Gaussian of width sigma truncated to |dr| <= R and |dc| <= R
    with R = ceil(3 sigma):  h(i, j) = exp(-(dr^2 + dc^2) / (2 sigma^2)), and
    h = identity for sigma == 0;
  * write-back: W[f, j] = sum_i h(i, j) acc[f, i] / sum_i h(i, j) count[i]
    wherever that denominator is positive; a neuron whose neighbourhood
    caught no document keeps its weights.

Everything is a direct evaluation in fp64: update_finish with a dense [N, N]
neighbourhood matrix (small maps only), update_finish_at with the window sums
of the definition at listed units (any map size).  Pins (tests/test_oracle_update.py): sigma = 0
gives each unit the mean of its documents; one document moves every unit of
its neighbourhood exactly onto itself; the dense matrix equals the product of
two one-dimensional Gaussians (separability) and is symmetric; the update is
linear in the accumulators (two batches accumulated = one batch of both);
document order does not matter; update_finish_at equals update_finish on
small maps, and on a 512 x 512 map reproduces the one-document and sigma = 0
closed forms.
"""

from __future__ import annotations

import math
from typing import Optional

import numpy as np


def update_accumulate(indptr: np.ndarray, indices: np.ndarray, bmu: np.ndarray, F: int, N: int,
                      acc: Optional[np.ndarray] = None, count: Optional[np.ndarray] = None):
    """Add one batch into the accumulators: acc [F, N] and count [N] (int64)."""
    if acc is None:
        acc = np.zeros((F, N), np.int64)
    if count is None:
        count = np.zeros(N, np.int64)
    for d in range(len(indptr) - 1):
        b = int(bmu[d])
        feats = np.asarray(indices[int(indptr[d]):int(indptr[d + 1])], np.int64)
        acc[feats, b] += 1
        count[b] += 1
    return acc, count


def neighbourhood_radius(sigma: float) -> int:
    """R = ceil(3 sigma): taps with |offset| <= R along each grid axis."""
    return int(math.ceil(3.0 * float(sigma))) if sigma > 0 else 0


def neighbourhood(rows: int, cols: int, sigma: float) -> np.ndarray:
    """Dense h(i, j) over the N = rows * cols neurons (fp64)."""
    N = rows * cols
    r = np.arange(N) // cols
    c = np.arange(N) % cols
    dr = r[:, None] - r[None, :]
    dc = c[:, None] - c[None, :]
    if sigma <= 0:
        return np.eye(N)
    R = neighbourhood_radius(sigma)
    h = np.exp(-(dr.astype(np.float64) ** 2 + dc.astype(np.float64) ** 2) / (2.0 * sigma * sigma))
    h[(np.abs(dr) > R) | (np.abs(dc) > R)] = 0.0
    return h


def update_finish(W: np.ndarray, acc: np.ndarray, count: np.ndarray, rows: int, cols: int,
                  sigma: float) -> np.ndarray:
    """New codebook [F, N] (fp64) from the accumulators; W is the old one."""
    H = neighbourhood(rows, cols, sigma)
    num = acc.astype(np.float64) @ H            # [F, N]: sum_i acc[f, i] h(i, j)
    den = count.astype(np.float64) @ H          # [N]
    new = np.array(W[:, :rows * cols], dtype=np.float64)
    moved = den > 0
    new[:, moved] = num[:, moved] / den[moved]
    return new


def update_finish_at(W_at: np.ndarray, acc: np.ndarray, count: np.ndarray, rows: int, cols: int,
                     sigma: float, units) -> np.ndarray:
    """New weights at the listed units only, for maps too large for the dense matrix.

    W_at [F', len(units)] holds the old weights there, acc [F', N] the
    accumulators of the same F' features, count [N] the unit counts.  For unit
    j the window sums of the definition are evaluated term by term:
    num = sum over units i with |dr| <= R and |dc| <= R of h(i, j) acc[:, i],
    den likewise over count; the unit moves to num / den when den > 0.
    """
    R = neighbourhood_radius(sigma)
    out = np.array(W_at, dtype=np.float64)
    for k, j in enumerate(units):
        r, c = divmod(int(j), cols)
        num = np.zeros(acc.shape[0], np.float64)
        den = 0.0
        for rr in range(max(0, r - R), min(rows, r + R + 1)):
            for cc in range(max(0, c - R), min(cols, c + R + 1)):
                i = rr * cols + cc
                h = 1.0 if sigma <= 0 else math.exp(-((rr - r) ** 2 + (cc - c) ** 2) / (2.0 * sigma * sigma))
                num += h * acc[:, i].astype(np.float64)
                den += h * float(count[i])
        if den > 0:
            out[:, k] = num / den
    return out
