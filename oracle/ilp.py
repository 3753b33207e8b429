"""Oracle: exact bit allocation (the per-projection integer linear program).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper assigns one width per spectral unit by the ILP of Sec. 3.3
(Eq. ilp_piecewise_projection; App. B.4, Eq. ilp_piecewise_eps):

    minimize   sum_u C[u, b_u]
    subject to sum_u b_u <= B,   exactly one width per unit,

solved independently per projection type, with the bit cost of a width being
the width itself.  The paper hands this to a commercial MILP solver and says
nothing about ties or tolerances.  Readings fixed here:

* Costs are integerized before solving so that sums are exact:
  K = 62 - ceil(log2(units + 1)), scale = 2^K / max|C| (one fp64 division),
  C_int = rint(C * scale) as int64 (all zero if max|C| = 0).
* Among all optima the lexicographically smallest vector of widths, in unit
  order, is returned.
* B < min(width) * units is infeasible.
* The budget is floor(avg_bits * units) (average bits per unit), not the
  paper's FP16-basis-adjusted b_eq (App. B.5).
"""
from __future__ import annotations

import itertools
import math

import numpy as np


class Infeasible(ValueError):
    pass


def integerize(L) -> np.ndarray:
    """Exact int64 costs: rint(L * 2^K / max|L|), K = 62 - ceil(log2(units+1))."""
    L = np.asarray(L, dtype=np.float64)
    if not np.all(np.isfinite(L)):
        raise ValueError("integerize: non-finite cost")
    units = L.shape[0]
    K = 62 - int(units).bit_length()          # bit_length(u) == ceil(log2(u + 1))
    m = float(np.max(np.abs(L))) if L.size else 0.0
    if m == 0.0:
        return np.zeros(L.shape, dtype=np.int64)
    scale = math.ldexp(1.0, K) / m
    return np.rint(L * scale).astype(np.int64)


def objective(L, bits, bits_u) -> float:
    """sum_u L[u, j_u] where bits[j_u] == bits_u[u]."""
    L = np.asarray(L, dtype=np.float64)
    idx = np.searchsorted(np.asarray(bits), np.asarray(bits_u))
    return float(np.sum(L[np.arange(L.shape[0]), idx]))


def _setup(L, bits, budget):
    bits = [int(b) for b in bits]
    if any(b2 <= b1 for b1, b2 in zip(bits, bits[1:])):
        raise ValueError("bits must be strictly ascending")
    Li = integerize(L)
    U = Li.shape[0]
    ex = [b - bits[0] for b in bits]
    cap = int(budget) - U * bits[0]
    if cap < 0:
        raise Infeasible("budget below min(bits) * units")
    cap = min(cap, U * ex[-1])
    return bits, Li, U, ex, cap


def _backward_step(g_next: np.ndarray, row: np.ndarray, ex, cap: int,
                   out: np.ndarray = None, tmp: np.ndarray = None) -> np.ndarray:
    """g_i(c) = min_j row[j] + g_{i+1}(c - ex_j) over widths with ex_j <= c.

    ``out`` and ``tmp`` (cap + 1 entries each, neither aliasing g_next) are
    optional preallocated buffers; the result is written to ``out``."""
    if out is None:
        out = np.empty_like(g_next)
    if tmp is None:
        tmp = np.empty_like(g_next)
    np.add(g_next, row[0], out=out)
    for j in range(1, len(ex)):
        e = ex[j]
        if e > cap:
            continue
        cand = tmp[: cap + 1 - e]
        np.add(g_next[: cap + 1 - e], row[j], out=cand)
        np.minimum(out[e:], cand, out=out[e:])
    return out


def allocate_dp(L, bits, budget: int, block: int = 256, full_limit: int = 1 << 26):
    """Exact optimum by dynamic programming over the remaining extra bits.

    g_i(c) is the least integerized cost of units i..U-1 using at most c bits
    above min(bits) each; g_U = 0.  The forward pass picks, at each unit, the
    smallest width that still attains the optimum, which yields the
    lexicographically smallest optimal vector.  Large instances keep every
    ``block``-th table and recompute the rest block by block.

    Returns (bits_u uint8 [units], optimum as an int in integerized units).
    """
    bits, Li, U, ex, cap = _setup(L, bits, budget)
    out = np.zeros(U, dtype=np.uint8)
    if U == 0:
        return out, 0
    zero = np.zeros(cap + 1, dtype=np.int64)

    def forward(i0, i1, tables, c):
        # tables[t] = g_{i0 + t} for t = 0 .. i1 - i0
        for i in range(i0, i1):
            gi, gn = tables[i - i0], tables[i - i0 + 1]
            for j in range(len(ex)):
                if ex[j] <= c and Li[i, j] + gn[c - ex[j]] == gi[c]:
                    out[i] = bits[j]
                    c -= ex[j]
                    break
            else:  # pragma: no cover - the optimum is always attained
                raise AssertionError("dp reconstruction failed")
        return c

    if U * (cap + 1) <= full_limit:
        tables = [None] * (U + 1)
        tables[U] = zero
        for i in range(U - 1, -1, -1):
            tables[i] = _backward_step(tables[i + 1], Li[i], ex, cap)
        forward(0, U, tables, cap)
        return out, int(tables[0][cap])

    ckpt = {U: zero}
    g = zero
    bufs = [np.empty(cap + 1, dtype=np.int64) for _ in range(2)]
    tmp = np.empty(cap + 1, dtype=np.int64)
    for i in range(U - 1, -1, -1):
        g = _backward_step(g, Li[i], ex, cap, out=bufs[i % 2], tmp=tmp)
        if i % block == 0:
            ckpt[i] = g.copy()
    best = int(ckpt[0][cap])
    c = cap
    blk = [np.empty(cap + 1, dtype=np.int64) for _ in range(block)]  # reused per block
    for i0 in range(0, U, block):
        i1 = min(i0 + block, U)
        tables = [None] * (i1 - i0 + 1)
        tables[-1] = ckpt[i1] if i1 in ckpt else None
        if tables[-1] is None:  # i1 == U is always checkpointed; others are block multiples
            raise AssertionError("missing checkpoint")
        for t in range(i1 - i0 - 1, 0, -1):
            tables[t] = _backward_step(tables[t + 1], Li[i0 + t], ex, cap,
                                       out=blk[t] if t < len(blk) else None, tmp=tmp)
        tables[0] = ckpt[i0]
        c = forward(i0, i1, tables, c)
    return out, best


def allocate_exhaustive(L, bits, budget: int):
    """Brute force over every assignment (<= 8 units), lexicographic order.

    Assignments are enumerated in lexicographic order of their width
    vectors and the incumbent is replaced only on strict improvement, so the
    first optimum found is the lexicographically smallest.
    """
    bits, Li, U, ex, cap = _setup(L, bits, budget)
    if U > 8:
        raise ValueError("exhaustive search is for tiny instances")
    best = None
    best_idx = None
    for idx in itertools.product(range(len(bits)), repeat=U):
        w = sum(bits[j] for j in idx)
        if w > budget:
            continue
        cost = int(sum(int(Li[u, j]) for u, j in enumerate(idx)))
        if best is None or cost < best:
            best, best_idx = cost, idx
    return np.array([bits[j] for j in best_idx], dtype=np.uint8), best
