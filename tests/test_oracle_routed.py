"""Pins of the oracle's routed per-expert calibration Grams (App. B.2, Eq.
app_affinity_gram) and their loss table, and of the synthetic router."""
import numpy as np
import pytest

import oracle
import synth
from oracle import routed


def _tiny():
    cfg = synth.CONFIGS["tiny"]
    X = synth.calibration_input(cfg, "gate")
    return cfg, X, synth.routing(cfg, X)


def test_router_is_top_k_with_normalized_weights():
    cfg, X, (off, tok, w) = _tiny()
    n, k = X.shape[0], synth.TOP_K["tiny"]
    assert off[0] == 0 and off[-1] == n * k
    assert np.all(np.diff(off) >= 0)
    # every token appears k times (once per chosen expert) and its weights sum to 1
    assert np.array_equal(np.bincount(tok, minlength=n), np.full(n, k))
    sums = np.bincount(tok, weights=w.astype(np.float64), minlength=n)
    np.testing.assert_allclose(sums, 1.0, rtol=1e-6)
    assert np.all(w > 0)
    for e in range(cfg.E):
        assert np.all(np.diff(tok[off[e]:off[e + 1]]) > 0)


def test_expert_grams_add_up_to_the_shared_gram():
    """With per-token weights summing to 1, sum_e H_e = X^T X / n (the shared H)."""
    cfg, X, (off, tok, w) = _tiny()
    X64 = synth.as_f64(X, cfg.dtype)
    Hs = routed.gram_routed(X64, off, tok, w)
    H = oracle.gram(X64)
    # the fp32 weights of a token sum to 1 within ~1e-7
    assert np.linalg.norm(Hs.sum(axis=0) - H) <= 1e-6 * np.linalg.norm(H)
    for H in Hs:
        assert np.allclose(H, H.T)
        assert np.min(np.linalg.eigvalsh(H)) > -1e-9 * np.max(np.abs(H))


def test_expert_gram_by_explicit_loops():
    g = np.random.default_rng(1)
    X = g.standard_normal((9, 5))
    off = np.array([0, 3, 3, 7])
    tok = np.array([0, 4, 8, 1, 2, 5, 6])
    w = g.random(7)
    Hs = routed.gram_routed(X, off, tok, w)
    for e in range(3):
        ref = np.zeros((5, 5))
        for i in range(off[e], off[e + 1]):
            for a in range(5):
                for b in range(5):
                    ref[a, b] += w[i] * X[tok[i], a] * X[tok[i], b]
        np.testing.assert_allclose(Hs[e], ref / 9, rtol=1e-12, atol=1e-15)
    assert np.all(Hs[1] == 0)


def test_routed_loss_is_the_affinity_weighted_output_error():
    """L[u, b] = (1/n) sum_t g_t (delta . x_t)^2 over expert e's tokens."""
    g = np.random.default_rng(2)
    n, d, E, upe, G = 64, 64, 3, 4, 32
    X = g.standard_normal((n, d))
    off = np.array([0, 20, 50, 70])
    tok = np.concatenate([np.sort(g.choice(n, 20, replace=False)),
                          np.sort(g.choice(n, 30, replace=False)),
                          np.sort(g.choice(n, 20, replace=False))])
    w = g.random(70)
    Hs = routed.gram_routed(X, off, tok, w)
    C = (g.standard_normal((E * upe, d)) * 0.1).astype(np.float32)
    L = routed.score_routed(C, Hs, upe, (1, 3), G)
    for u in range(E * upe):
        e = u // upe
        for j, b in enumerate((1, 3)):
            delta = C[u].astype(np.float64) - oracle.fake_quant(C[u], b, G)[0]
            i0, i1 = off[e], off[e + 1]
            brute = np.sum(w[i0:i1] * (X[tok[i0:i1]] @ delta) ** 2) / n
            assert abs(L[u, j] - brute) <= 1e-10 * brute
