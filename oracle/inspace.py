"""Oracle: the input-space shared basis of the paper's gate/up projections.

TEST INFRASTRUCTURE ONLY (see the package docstring).

For a gate or up projection the experts share their input space (Sec. 3.2):
the expert weights are stacked along the output channels,

    W_cat = [W_1; ...; W_E]  ((E d_out) x d_in)  =  P~_cat Phi^T,

with Phi the right singular vectors of W_cat (Eq. shared_basis_input_proj),
i.e. the eigenvectors of M_in = W_cat^T W_cat = sum_e W_e^T W_e.  Expert e is
W_e = P~_e Phi^T with P~_e = W_e Phi; its spectral unit k is the column
p~_{e,k} = W_e phi_k (length d_out), of energy alpha = ||p~_{e,k}||
(Definitions spectral_energy_matrix, spectral_matrix).  Rows of
C_e = Phi_r^T W_e^T are those columns.

Quantizing the units perturbs W_e by Delta = sum_k delta_k phi_k^T, and the
activation-aware loss tr(Delta H Delta^T) couples units through
phi_k^T H phi_l (Lemma spectrum_wise_error_decomp).  The paper drops the
cross terms (the diagonal approximation before Corollary
additive_spectrum_wise_loss), leaving

    L[e, k, b] = beta_k ||c - Q_b(c)||^2,   beta_k = phi_k^T H phi_k  (Eq. beta_def),

with c = p~_{e,k} quantized by the group rule of ``quant.py`` and beta_k
shared by all experts.  It is exact when H is diagonal in the basis Phi.
"""
from __future__ import annotations

import numpy as np

from .quant import fake_quant


def gram_experts_in(W) -> np.ndarray:
    """M_in = sum_e W_e^T W_e = W_cat^T W_cat, fp64 [d_in][d_in]."""
    W = np.asarray(W, dtype=np.float64)
    E, d_out, d_in = W.shape
    M = np.zeros((d_in, d_in))
    for e in range(E):
        M += W[e].T @ W[e]
    return M


def project_in(Vt, W) -> np.ndarray:
    """C_e = Phi_r^T W_e^T for every expert, stacked [E*r][d_out]; unit u = e*r + k
    is the column W_e phi_k."""
    Vt = np.asarray(Vt, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    return np.concatenate([Vt @ W[e].T for e in range(W.shape[0])], axis=0)


def basis_importance(Vt, H) -> np.ndarray:
    """beta_k = phi_k^T H phi_k for the rows phi_k^T of Vt (Eq. beta_def)."""
    Vt = np.asarray(Vt, dtype=np.float64)
    return np.sum((Vt @ np.asarray(H, dtype=np.float64)) * Vt, axis=1)


def score_diag(C, beta, r: int, bits, G: int) -> np.ndarray:
    """L[u][j] = beta[u % r] * ||c_u - Q_{bits[j]}(c_u)||^2, the fp32 rows C
    quantized by the group rule and the error taken in fp64."""
    C32 = np.ascontiguousarray(np.asarray(C), dtype=np.float32)
    beta = np.asarray(beta, dtype=np.float64)
    units = C32.shape[0]
    w = beta[np.arange(units) % r]
    out = np.empty((units, len(bits)))
    c64 = C32.astype(np.float64)
    for j, b in enumerate(bits):
        d = c64 - fake_quant(C32, int(b), G)
        out[:, j] = w * np.sum(d * d, axis=1)
    return out
