"""Oracle: routing-affinity-weighted calibration Grams, one per expert.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's calibration Gram of an expert weights the activations routed to
that expert by their routing affinities (App. B.2, Eq. app_affinity_gram):
H = X Diag(g) X^T = sum_t g_t x_t x_t^T over the tokens routed to the
expert.  Reading fixed here: the same 1/n as the shared Gram (n = all
calibration rows), so that with weights normalized per token the experts'
Grams add up to the shared one,

    H_e = (1/n) sum_{i in expert e} w_i x_{row_i} x_{row_i}^T,

and the activation-aware loss of a unit of expert e is delta H_e delta^T
(Eq. app_down_exact_metric with H_e).
"""
from __future__ import annotations

import numpy as np

from .quant import score_rows


def gram_routed(X, offsets, rows, weights, n: int | None = None) -> np.ndarray:
    """H_e = (1/n) sum_i w_i x_{rows_i} x_{rows_i}^T for i in [offsets[e], offsets[e+1]),
    fp64 [E][d][d]; n defaults to the number of rows of X."""
    X = np.asarray(X, dtype=np.float64)
    n = X.shape[0] if n is None else n
    offsets = np.asarray(offsets, dtype=np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    w = np.asarray(weights, dtype=np.float64)
    E = offsets.shape[0] - 1
    out = np.zeros((E, X.shape[1], X.shape[1]))
    for e in range(E):
        i0, i1 = offsets[e], offsets[e + 1]
        Xe = X[rows[i0:i1]]
        out[e] = (Xe * w[i0:i1, None]).T @ Xe / n
    return out


def score_routed(C, Hs, units_per_h: int, bits, G: int) -> np.ndarray:
    """L[u][j] = delta H_{u // units_per_h} delta^T with the group rule of quant.py."""
    C = np.asarray(C)
    out = np.empty((C.shape[0], len(bits)))
    for e in range(C.shape[0] // units_per_h):
        sl = slice(e * units_per_h, (e + 1) * units_per_h)
        out[sl] = score_rows(C[sl], np.asarray(Hs[e], dtype=np.float64), bits, G)
    return out
