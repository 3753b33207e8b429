"""Oracle: the paper's piecewise surrogate cost and equivalent-bit budget.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The ILP of the paper (Sec. 3.3, Eq. ilp_piecewise_projection; App. B.4,
Theorem app_spectrum_loss) does not consume measured losses: it prices width
b for spectral unit k at

    L_k(b) = alpha_k^2 * beta_k^gamma * E_k(b),

with alpha_k the spectral energy (norm) of the unit, beta_k its
activation-aware importance and E_k(b) the normalized distortion of its unit
direction p_k (Eq. piecewise_error_surrogate / piecewise_expected_eps) over
the candidate widths {0, 1, 2, 3, 4, 6, 8, 16}:

    E_k(b) = (d rho_k^2 / 3) exp(-2 ln2 b),  rho_k = ||p_k||_inf   b in {6, 8, 16}
             kappa_b  (one shared constant per width)              b in {2, 3, 4}
             sin^2 theta_k, cos theta_k = ||p_k||_1 / sqrt(d)       b = 1
             1                                                     b = 0 (eviction)

Readings fixed here (the hot path builds every basis in the output space,
so every unit is a row c of C_e = U^T W_e, as for the paper's down
projection):

* alpha_k = ||c_k||_2 and p_k = c_k / alpha_k (Sec. 3.2; App. B.1);
* beta_k = p_k^T H p_k, the down-projection form of Eq. app_down_beta_approx
  / app_unified_beta_def, with H the calibration Gram of the projection;
* a unit with alpha_k = 0 costs 0 at every width;
* kappa_b are the values printed in Table kappa_values;
* exp(-2 ln2 b) = 4^-b exactly.

The budget (App. B.5, Eqs. app_projection_bit_budget and
app_projection_normalized_budget): an E-expert projection of m x n weights
quantized to an equivalent b_eq bits per weight spends E m n b_eq bits; the
shared basis is kept in fp16; what is left, divided by the length of a
spectral vector, is the ILP budget in units of "bits per vector element".
In the paper the basis is the full n x n one; for a rank-r basis of an
output space of size n_out the reserved storage is 16 n_out r bits (the two
agree at r = n_out).
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

# Candidate widths (Sec. 3.3, "piecewise reconstruction-error surrogate").
WIDTHS = (0, 1, 2, 3, 4, 6, 8, 16)
# Low-bit distortion coefficients printed in Table kappa_values.
KAPPA_PRINTED = {2: 0.14949200, 3: 0.04067890, 4: 0.01184786}


def unit_stats(C):
    """Per-row (alpha^2, rho, cos theta) of the spectral rows C [units][d].

    alpha^2 = ||c||^2, p = c / alpha, rho = ||p||_inf, cos theta =
    ||p||_1 / sqrt(d) (Lemma one_bit_sign_distortion).  Rows with alpha = 0
    get rho = cos = 0.
    """
    C = np.asarray(C, dtype=np.float64)
    if C.ndim == 1:
        C = C[None, :]
    d = C.shape[1]
    a2 = np.einsum("ij,ij->i", C, C)
    alpha = np.sqrt(a2)
    safe = np.where(alpha > 0, alpha, 1.0)
    rho = np.where(alpha > 0, np.max(np.abs(C), axis=1) / safe, 0.0)
    cos = np.where(alpha > 0, np.sum(np.abs(C), axis=1) / (safe * math.sqrt(d)), 0.0)
    # ||p||_1 <= sqrt(d) ||p||_2 (Cauchy-Schwarz): cos theta <= 1, attained by
    # rows of equal magnitudes, where rounding may land just above 1
    return a2, rho, np.minimum(cos, 1.0)


def beta(C, H):
    """beta_k = p_k^T H p_k with p_k = c_k / ||c_k|| (0 for a zero row)."""
    C = np.asarray(C, dtype=np.float64)
    if C.ndim == 1:
        C = C[None, :]
    H = np.asarray(H, dtype=np.float64)
    q = np.sum((C @ H) * C, axis=1)               # c H c^T per row
    a2 = np.sum(C * C, axis=1)
    return np.where(a2 > 0, q / np.where(a2 > 0, a2, 1.0), 0.0)


def distortion(b: int, d: int, rho, cos, kappa=KAPPA_PRINTED):
    """E(b) of the piecewise surrogate for unit directions with the given
    rho = ||p||_inf and cos theta = ||p||_1 / sqrt(d)."""
    rho = np.asarray(rho, dtype=np.float64)
    cos = np.asarray(cos, dtype=np.float64)
    if b == 0:
        return np.ones_like(rho)
    if b == 1:
        return 1.0 - cos * cos
    if b in (2, 3, 4):
        return np.full_like(rho, float(kappa[b]))
    if b in (6, 8, 16):
        eta = d * rho * rho / 3.0                 # Lemma high_bit_distortion
        return eta * math.ldexp(1.0, -2 * b)      # exp(-2 ln2 b) = 4^-b
    raise ValueError(f"width {b} is not a candidate of the surrogate")


def surrogate_table(C, H, gamma: float, kappa=KAPPA_PRINTED, widths=WIDTHS):
    """L[u][j] = alpha_u^2 beta_u^gamma E_u(widths[j]) in fp64."""
    C = np.asarray(C, dtype=np.float64)
    d = C.shape[1]
    a2, rho, cos = unit_stats(C)
    bt = beta(C, H)
    w = np.power(np.maximum(bt, 0.0), float(gamma))
    w = np.where(a2 > 0, w, 0.0)
    cols = [a2 * w * distortion(b, d, rho, cos, kappa) for b in widths]
    return np.stack(cols, axis=1)


def budget_equivalent(E: int, n_out: int, m: int, b_eq: float, r: int | None = None) -> int:
    """ILP budget of one projection (App. B.5): floor((E n_out m b_eq -
    16 n_out r) / m), in bits per vector element; r defaults to n_out (the
    paper's full basis)."""
    r = n_out if r is None else r
    total = Fraction(E) * n_out * m * Fraction(b_eq)   # exact (b_eq is a binary fraction)
    return math.floor((total - 16 * n_out * r) / m)


# --- the quantizers the surrogate is derived from (App. B.3) ---------------

def quant_symmetric(p, b: int, s: float):
    """Symmetric uniform quantizer, Eq. app_scalar_quantization_uk:
    s * clamp(round(p / s), -2^(b-1), 2^(b-1) - 1), halves rounded to even."""
    p = np.asarray(p, dtype=np.float64)
    lo, hi = -(1 << (b - 1)), (1 << (b - 1)) - 1
    return s * np.clip(np.rint(p / s), lo, hi)


def quant_sign(p):
    """One-bit sign quantizer, Eq. app_one_bit_quantization:
    mean|p| * sign(p), with sign(0) = +1."""
    p = np.asarray(p, dtype=np.float64)
    s = np.mean(np.abs(p))
    return s * np.where(p >= 0, 1.0, -1.0)
