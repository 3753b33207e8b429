"""Pins for the oracle's exact bit allocation."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle.ilp import Infeasible

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _cases():
    with open(os.path.join(GOLDEN, "ilp_examples.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_ilp_hand_solved(case):
    L = np.array(case["L"], dtype=np.float64)
    for solver in (oracle.allocate_dp, oracle.allocate_exhaustive):
        bits_u, _ = solver(L, case["bits"], case["budget"])
        assert bits_u.tolist() == case["bits_u"]
        assert oracle.objective(L, case["bits"], bits_u) == case["objective"]


def _random_L(g, U, nb, ties=False):
    L = g.gamma(2.0, 1.0, size=(U, nb)) * np.logspace(0, -3, nb)[None, :]
    if ties:
        L = np.round(L * 4) / 4
        L[g.integers(0, U)] = L[g.integers(0, U)]   # duplicate unit
        L[g.integers(0, U)] = 0.0                   # zero unit
    return L.astype(np.float32)


@pytest.mark.parametrize("seed", range(12))
def test_dp_matches_exhaustive(seed):
    g = np.random.default_rng(100 + seed)
    U = int(g.integers(1, 8))
    bits = [1, 2, 3, 4] if seed % 3 else [1, 2, 3, 4, 8]
    L = _random_L(g, U, len(bits), ties=seed % 2 == 0)
    for budget in range(U * bits[0], U * bits[-1] + 2):
        a, va = oracle.allocate_dp(L, bits, budget)
        b, vb = oracle.allocate_exhaustive(L, bits, budget)
        assert va == vb
        assert a.tolist() == b.tolist()
        assert int(a.astype(int).sum()) <= budget


def test_checkpointed_dp_equals_full_dp():
    g = np.random.default_rng(7)
    L = _random_L(g, 700, 5, ties=True)
    bits = [1, 2, 3, 4, 8]
    budget = 2 * 700 + 17
    a, va = oracle.allocate_dp(L, bits, budget)
    b, vb = oracle.allocate_dp(L, bits, budget, block=64, full_limit=0)
    assert va == vb and np.array_equal(a, b)


def test_extreme_budgets():
    g = np.random.default_rng(8)
    L = _random_L(g, 50, 4)
    bits = [1, 2, 3, 4]
    a, _ = oracle.allocate_dp(L, bits, 50)
    assert np.all(a == 1)
    a, _ = oracle.allocate_dp(L, bits, 4 * 50)
    Li = oracle.integerize(L)
    assert np.array_equal(a, np.array(bits)[np.argmin(Li, axis=1)])
    with pytest.raises(Infeasible):
        oracle.allocate_dp(L, bits, 49)


def test_optimum_monotone_and_bounded():
    g = np.random.default_rng(9)
    U = 120
    L = _random_L(g, U, 4)
    bits = [1, 2, 3, 4]
    Li = oracle.integerize(L).astype(np.float64)
    prev = None
    for budget in range(U, 4 * U + 1, 37):
        a, v = oracle.allocate_dp(L, bits, budget)
        if prev is not None:
            assert v <= prev
        prev = v
        # Lagrangian lower bound: sum_u min_b (C + lam b) - lam B <= OPT
        for lam in (0.0, 1e16, 1e17, 1e18):
            lb = np.sum(np.min(Li + lam * np.array(bits)[None, :], axis=1)) - lam * budget
            assert lb <= v * (1 + 1e-12) + 1
    # never worse than a uniform 2-bit assignment at the same budget
    a, v = oracle.allocate_dp(L, bits, 2 * U)
    assert v <= int(np.sum(oracle.integerize(L)[:, 1]))


def test_integerize_exact_scale():
    L = np.array([[0.0, 1.5], [3.0, -0.75]])
    Li = oracle.integerize(L)
    K = 62 - (2).bit_length()
    assert Li[1, 0] == 2 ** K
    assert Li[0, 1] == 2 ** (K - 1)
    assert Li[1, 1] == -(2 ** (K - 2))
    assert not oracle.integerize(np.zeros((3, 2))).any()
