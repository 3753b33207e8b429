"""Pins for the oracle's Gram, cross-expert Gram, shared basis and factors.

Each check ties the oracle to something other than its own formula: closed
forms, an independent SVD, trace identities, reconstruction, and a planted
low-rank structure.
"""
import numpy as np
import pytest

import oracle
import synth


def _rng(seed):
    return np.random.default_rng(seed)


# --------------------------------------------------------------------------- H
def test_gram_scaled_identity():
    # X = [sqrt(n) I_d ; 0] (n > d rows): H = X^T X / n = I exactly.
    n, d = 10, 4
    X = np.zeros((n, d))
    X[:d] = np.sqrt(n) * np.eye(d)
    H = oracle.gram(X)
    assert H.shape == (d, d)
    np.testing.assert_allclose(H, np.eye(d), atol=1e-15)


def test_gram_is_a_mean_not_a_sum():
    # Stacking the calibration set twice must not change the mean Gram.
    X = _rng(1).standard_normal((37, 12))
    H = oracle.gram(X)
    np.testing.assert_allclose(oracle.gram(np.vstack([X, X])), H, rtol=0, atol=1e-14 * np.abs(H).max())


def test_gram_two_tokens_closed_form():
    # rows (a, 0) and (0, b): H = diag(a^2, b^2) / 2
    H = oracle.gram(np.array([[3.0, 0.0], [0.0, 5.0]]))
    np.testing.assert_allclose(H, np.diag([4.5, 12.5]), atol=1e-15)


def test_gram_psd_and_trace():
    X = _rng(2).standard_normal((64, 20)) * np.linspace(0.1, 5, 20)
    H = oracle.gram(X)
    np.testing.assert_allclose(H, H.T, atol=0)
    assert np.linalg.eigvalsh(H).min() > -1e-12 * np.abs(H).max()
    assert np.isclose(np.trace(H), np.sum(X * X) / X.shape[0], rtol=1e-13)


# --------------------------------------------------------------------------- M
def test_gram_experts_trace_and_concat():
    W = _rng(3).standard_normal((5, 7, 11))
    M = oracle.gram_experts(W)
    assert np.isclose(np.trace(M), sum(np.sum(w * w) for w in W), rtol=1e-13)
    Wcat = np.hstack(list(W))                      # [d_out][E * d_in]
    sv = np.linalg.svd(Wcat, compute_uv=False)
    ev = np.sort(np.linalg.eigvalsh(M))[::-1]
    np.testing.assert_allclose(ev, sv ** 2, rtol=1e-10, atol=1e-10 * sv[0] ** 2)


# --------------------------------------------------------------------------- U
def test_shared_basis_matches_independent_svd():
    W = _rng(4).standard_normal((3, 16, 40))
    M = oracle.gram_experts(W)
    Ut, lam = oracle.shared_basis(M, 6)
    Wcat = np.hstack(list(W))
    Us, sv, _ = np.linalg.svd(Wcat, full_matrices=False)
    np.testing.assert_allclose(lam, sv[:6] ** 2, rtol=1e-11)
    # eigenvectors agree with left singular vectors up to sign (distinct spectrum)
    for k in range(6):
        cos = abs(float(Ut[k] @ Us[:, k]))
        assert cos > 1 - 1e-10
    assert np.all(np.diff(lam) <= 0)


def test_shared_basis_residual_orthonormal_sign():
    W = _rng(5).standard_normal((4, 24, 30))
    M = oracle.gram_experts(W)
    Ut, lam = oracle.shared_basis(M, 10)
    U = Ut.T
    assert np.linalg.norm(M @ U - U * lam) <= 1e-12 * np.linalg.norm(M)
    np.testing.assert_allclose(Ut @ U, np.eye(10), atol=1e-13)
    for k in range(10):
        i = int(np.argmax(np.abs(Ut[k])))
        assert Ut[k, i] > 0


def test_full_rank_basis_reconstructs_experts():
    # r = d_out: U C_e = U U^T W_e = W_e to round-off.
    W = _rng(6).standard_normal((3, 12, 20))
    M = oracle.gram_experts(W)
    Ut, _ = oracle.shared_basis(M, 12)
    C = oracle.project(Ut, W)
    for e in range(3):
        np.testing.assert_allclose(Ut.T @ C[e * 12:(e + 1) * 12], W[e], atol=1e-12)


def test_planted_shared_subspace_is_recovered():
    # Noise-free synthetic experts: W_e = U0 A_e, so rank(M) = k0 and the top-k0
    # eigenvectors span span(U0) (principal angles ~ 0).
    cfg = synth.CONFIGS["tiny"]
    U0 = np.linalg.qr(synth.shared_component(cfg, "gate").astype(np.float64))[0]
    g = _rng(7)
    W = [U0 @ g.standard_normal((cfg.k0, 256)) for _ in range(4)]
    M = oracle.gram_experts(W)
    Ut, lam = oracle.shared_basis(M, 40)
    k0 = cfg.k0
    s = np.linalg.svd(Ut[:k0] @ U0, compute_uv=False)
    assert s.min() > 1 - 1e-10
    assert lam[k0:].max() < 1e-9 * lam[0]


# --------------------------------------------------------------------------- C
def test_factor_energy_identities():
    W = _rng(8).standard_normal((2, 10, 18))
    M = oracle.gram_experts(W)
    for r in (4, 10):
        Ut, _ = oracle.shared_basis(M, r)
        C = oracle.project(Ut, W)
        alpha = oracle.unit_energy(C)
        for e in range(2):
            Ce = C[e * r:(e + 1) * r]
            assert np.isclose(np.sum(alpha[e * r:(e + 1) * r] ** 2), np.sum(Ce * Ce), rtol=1e-13)
            if r < 10:
                assert np.sum(Ce * Ce) < np.sum(W[e] * W[e])
            else:
                assert np.isclose(np.sum(Ce * Ce), np.sum(W[e] * W[e]), rtol=1e-12)


def test_project_layout_unit_index():
    # unit u = e*r + k is basis vector k applied to expert e
    W = _rng(9).standard_normal((3, 6, 5))
    Ut = np.linalg.qr(_rng(10).standard_normal((6, 6)))[0][:, :4].T
    C = oracle.project(Ut, W)
    assert C.shape == (12, 5)
    for e in range(3):
        for k in range(4):
            np.testing.assert_allclose(C[e * 4 + k], Ut[k] @ W[e], rtol=1e-14)
