"""Pins of the oracle's input-space basis (gate/up projections, Sec. 3.2) and
its diagonal-approximation loss.

The loss pin is brute force: when H is diagonal in the basis Phi the
cross-unit terms phi_k^T H phi_l vanish, so the measured output error
||(W_e - W^_e) X^T||^2 / n must equal the summed table plus the truncation
loss exactly; for a generic H it must not.
"""
import numpy as np
import pytest

import oracle
from oracle import inspace


def _weights(E, d_out, d_in, seed, k0=None):
    g = np.random.default_rng(seed)
    if k0 is None:
        return g.standard_normal((E, d_out, d_in)) * 0.1
    V0 = np.linalg.qr(g.standard_normal((d_in, k0)))[0]
    return np.stack([g.standard_normal((d_out, k0)) @ V0.T for _ in range(E)]), V0


def test_gram_in_trace_and_spectrum():
    """trace(M_in) = sum_e ||W_e||_F^2, and the eigenvalues of M_in are the
    squared singular values of the stacked W_cat (independent SVD)."""
    W = _weights(4, 24, 40, seed=1)
    M = inspace.gram_experts_in(W)
    assert np.allclose(M, M.T)
    assert abs(np.trace(M) - np.sum(W * W)) < 1e-10 * np.trace(M)
    s = np.linalg.svd(W.reshape(-1, 40), compute_uv=False)
    ev = np.sort(np.linalg.eigvalsh(M))[::-1]
    np.testing.assert_allclose(ev, s ** 2, rtol=1e-10, atol=1e-10 * s[0] ** 2)


def test_full_rank_basis_reconstructs_every_expert():
    """r = d_in: W_e = C_e^T Phi^T with C_e = Phi^T W_e^T (Eq. shared_basis_input_proj)."""
    W = _weights(3, 16, 48, seed=2)
    Vt, _ = oracle.shared_basis(inspace.gram_experts_in(W), 48)
    C = inspace.project_in(Vt, W)
    for e in range(3):
        np.testing.assert_allclose(C[e * 48:(e + 1) * 48].T @ Vt, W[e], atol=1e-12)


def test_planted_input_space_recovered():
    """Experts sharing a k0-dimensional input subspace give rank(M_in) = k0 and
    a top-k0 basis spanning it."""
    W, V0 = _weights(5, 20, 64, seed=3, k0=6)
    M = inspace.gram_experts_in(W)
    ev = np.sort(np.linalg.eigvalsh(M))[::-1]
    assert ev[6] < 1e-10 * ev[0]
    Vt, _ = oracle.shared_basis(M, 6)
    cosines = np.linalg.svd(Vt @ V0, compute_uv=False)
    assert np.all(cosines > 1 - 1e-10)


def test_basis_importance_is_the_activation_energy():
    """beta_k = ||X phi_k||^2 / n from the calibration rows."""
    g = np.random.default_rng(4)
    X = g.standard_normal((300, 32))
    X[:, 3] *= 7
    Vt = np.linalg.qr(g.standard_normal((32, 10)))[0].T
    b = inspace.basis_importance(Vt, oracle.gram(X))
    brute = np.array([np.sum((X @ v) ** 2) / 300 for v in Vt])
    np.testing.assert_allclose(b, brute, rtol=1e-11)


def _loss_setup(seed, diagonal_in_basis):
    g = np.random.default_rng(seed)
    E, d_out, d_in, r, G = 3, 64, 64, 40, 32
    W = _weights(E, d_out, d_in, seed=seed)
    Vfull, _ = oracle.shared_basis(inspace.gram_experts_in(W), d_in)
    n = 4 * d_in
    if diagonal_in_basis:
        lam = np.exp(g.standard_normal(d_in))
        # X^T X / n = Phi diag(lam) Phi^T: rows sqrt(n lam_k / 4) phi_k^T, four times
        X = np.tile(np.sqrt(n * lam / 4)[:, None] * Vfull, (4, 1))
    else:
        X = g.standard_normal((n, d_in))
        X[:, ::7] *= 5
    H = oracle.gram(X)
    Vt = Vfull[:r]
    C = inspace.project_in(Vt, W).astype(np.float32)
    beta = inspace.basis_importance(Vt, H)
    bits = (1, 2, 3, 4)
    L = inspace.score_diag(C, beta, r, bits, G)
    choice = g.integers(0, len(bits), size=E * r)
    Chat = np.stack([oracle.fake_quant(C[u], bits[choice[u]], G)[0] for u in range(E * r)])
    brute = trunc = 0.0
    for e in range(E):
        What = Chat[e * r:(e + 1) * r].T @ Vt
        brute += np.sum(((W[e] - What) @ X.T) ** 2) / n
        trunc += np.sum(((W[e] - W[e] @ Vt.T @ Vt) @ X.T) ** 2) / n
    table = float(np.sum(L[np.arange(E * r), choice]))
    # the reference for the table uses the fp32 rows the table quantizes
    Cf = C.astype(np.float64)
    extra = 0.0
    for e in range(E):
        dW = (W[e] - Cf[e * r:(e + 1) * r].T @ Vt) - (W[e] - W[e] @ Vt.T @ Vt)
        extra += np.sum((dW @ X.T) ** 2) / n   # fp32 rounding of C, ~1e-14
    return brute, table + trunc, extra


@pytest.mark.parametrize("seed", range(3))
def test_diagonal_loss_is_exact_when_h_is_diagonal_in_the_basis(seed):
    brute, model, extra = _loss_setup(seed, diagonal_in_basis=True)
    assert abs(brute - model) <= 1e-6 * brute + 10 * extra + 1e-12


def test_diagonal_loss_is_an_approximation_for_generic_h():
    brute, model, _ = _loss_setup(7, diagonal_in_basis=False)
    assert abs(brute - model) > 1e-4 * brute


def test_identity_h_gives_rtn_error_norms():
    g = np.random.default_rng(9)
    C = (g.standard_normal((12, 128)) * 0.05).astype(np.float32)
    L = inspace.score_diag(C, np.ones(4), 4, (2, 3), 64)
    for u in range(12):
        for j, b in enumerate((2, 3)):
            d = C[u].astype(np.float64) - oracle.fake_quant(C[u], b, 64)[0]
            assert abs(L[u, j] - np.sum(d * d)) <= 1e-12 * max(1.0, L[u, j])
