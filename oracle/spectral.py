"""Oracle: calibration Gram, cross-expert Gram, shared basis, spectral factors.

TEST INFRASTRUCTURE ONLY (see the package docstring).  All arithmetic fp64.
"""
from __future__ import annotations

import numpy as np


def gram(X: np.ndarray) -> np.ndarray:
    """H = (1/n) sum_t x_t x_t^T for calibration rows X [n][d].

    The paper weights each calibration token by its routing affinity,
    H = X Diag(g) X^T = sum_t g_t x_t x_t^T, which is PSD because g_t >= 0
    (App. B.2, Eq. app_affinity_gram; Lemma spectrum_wise_error_decomp).
    Reading: one activation matrix per layer shared by all experts, with the
    uniform weight g_t = 1/n, so that H is the mean outer product.  Here the
    tokens are the rows of X, hence H = X^T X / n.
    """
    X = np.asarray(X, dtype=np.float64)
    n = X.shape[0]
    if n == 0:
        raise ValueError("gram: no calibration rows")
    return (X.T @ X) / float(n)


def gram_experts(W) -> np.ndarray:
    """M = sum_e W_e W_e^T for expert weights W [E][d_out][d_in].

    App. B.1 concatenates the experts along the input channel,
    W_cat = [W_1 ... W_E] (Eq. app_down_w_cat), and takes its SVD
    W_cat = Phi Sigma V_cat^T (Eq. app_down_cat_svd_absorbed).  The left
    singular vectors Phi are the eigenvectors of W_cat W_cat^T, and that
    product is the sum of the per-expert Grams.  Experts are accumulated one
    at a time so that W_cat is never formed.
    """
    M = None
    for We in W:
        We = np.asarray(We, dtype=np.float64)
        P = We @ We.T
        M = P if M is None else M + P
    if M is None:
        raise ValueError("gram_experts: no experts")
    return M


def shared_basis(M: np.ndarray, r: int):
    """Top-r eigenpairs of the symmetric PSD M.

    Returns (Ut, lam): Ut [r][d_out] holds the eigenvectors as rows, lam [r]
    the eigenvalues, in descending order.  The paper keeps the left singular
    vectors Phi of W_cat as the unquantized shared basis (App. B.1,
    Eq. app_down_cat_svd_absorbed); lam_k = sigma_k(W_cat)^2.

    Readings (the paper fixes no conventions for the SVD): order by
    eigenvalue, descending; the sign of each eigenvector is chosen so that its
    entry of largest magnitude is positive, ties going to the lowest index.
    Truncation to r columns is the configuration's shared rank.
    """
    M = np.asarray(M, dtype=np.float64)
    d = M.shape[0]
    if not (1 <= r <= d):
        raise ValueError("shared_basis: need 1 <= r <= d_out")
    w, V = np.linalg.eigh(M)
    order = np.argsort(-w, kind="stable")[:r]
    lam = w[order]
    U = V[:, order]
    for k in range(r):
        i = int(np.argmax(np.abs(U[:, k])))
        if U[i, k] < 0:
            U[:, k] = -U[:, k]
    return np.ascontiguousarray(U.T), lam


def project(Ut: np.ndarray, W) -> np.ndarray:
    """Spectral factors C_e = U^T W_e, stacked as [E*r][d_in].

    With W_e = Phi P~_e^T (Eq. app_down_p_tilde_partition) and Phi
    orthonormal, P~_e^T = Phi^T W_e.  Truncated to the first r basis vectors
    this is U^T W_e.  Row k of C_e is the spectral component of expert e along
    basis vector k: unit u = e*r + k.
    """
    Ut = np.asarray(Ut, dtype=np.float64)
    out = [Ut @ np.asarray(We, dtype=np.float64) for We in W]
    return np.concatenate(out, axis=0)


def unit_energy(C: np.ndarray) -> np.ndarray:
    """Spectral energy alpha_u = ||c_u||_2 of each unit (Def. spectral_energy_matrix)."""
    C = np.asarray(C, dtype=np.float64)
    return np.sqrt(np.sum(C * C, axis=1))


def truncation_loss(Ut: np.ndarray, We: np.ndarray, X: np.ndarray) -> float:
    """||(I - U U^T) W_e X^T||_F^2 / n: the loss of dropping the basis tail.

    This part of the reconstruction error does not depend on the bit
    assignment (the ILP only sees the kept r components).
    """
    Ut = np.asarray(Ut, dtype=np.float64)
    We = np.asarray(We, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    R = We - Ut.T @ (Ut @ We)
    Y = R @ X.T
    return float(np.sum(Y * Y) / X.shape[0])
