"""Oracle: stage-3 inference from the packed factors (one projection of an MoE layer).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper serves the quantized experts from their packed spectral factors,
dequantized inside the expert kernels (Sec. 4.4).  For the output-space
basis an expert is W_e ~ U C^_e (App. B.1, W_e = Phi P~_e^T), so a token x
routed to experts e_1..e_k with weights g_1..g_k gives

    y = sum_j g_j W_{e_j} x  ~  U z,   z = sum_j g_j C^_{e_j} x,

with C^_e the dequantized rows of expert e (exactly what ``quant.unpack``
returns) and the shared basis applied once per token.  ``moe_decode_in`` is
the input-space form of the gate/up projections, where the basis is applied
first (z = Phi^T x) and each routed expert's units are combined with z.
"""
from __future__ import annotations

import numpy as np

from .quant import unpack


def dequantized_factors(codes, params, bits_u, d: int, G: int) -> np.ndarray:
    """C^ [units][d] in fp64 (the decoder's view of the packed units)."""
    return unpack(codes, params, bits_u, d, G)


def moe_decode(Chat, r: int, Ut, X, offsets, tokens, weights) -> np.ndarray:
    """y[b] = Ut^T z_b, z_b = sum over the routing entries i of token b of
    weights[i] C^_e X[b] (e the expert whose range [offsets[e], offsets[e+1])
    holds i), fp64 [B][d_out].

    Chat: [E*r][d_in] dequantized units (unit e*r + k is row k of C^_e);
    Ut: [r][d_out]; X: [B][d_in]; the routing in the grouped-by-expert form
    of ``synth.routing`` (offsets [E+1], tokens, weights).
    """
    Chat = np.asarray(Chat, dtype=np.float64)
    Ut = np.asarray(Ut, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    B = X.shape[0]
    Z = np.zeros((B, r))
    for e in range(len(offsets) - 1):
        Ce = Chat[e * r:(e + 1) * r]
        for i in range(int(offsets[e]), int(offsets[e + 1])):
            b = int(tokens[i])
            Z[b] += float(weights[i]) * (Ce @ X[b])
    return Z @ Ut


def moe_dense(W, X, offsets, tokens, weights) -> np.ndarray:
    """The unquantized layer: y[b] = sum over token b's entries of weights[i] W_e X[b]."""
    W = np.asarray(W, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    Y = np.zeros((X.shape[0], W.shape[1]))
    for e in range(len(offsets) - 1):
        for i in range(int(offsets[e]), int(offsets[e + 1])):
            b = int(tokens[i])
            Y[b] += float(weights[i]) * (W[e] @ X[b])
    return Y


def moe_decode_in(Chat, r: int, Vt, X, offsets, tokens, weights) -> np.ndarray:
    """The input-space form (the paper's gate/up projections, Sec. 3.2 and
    Sec. 4.4): expert e is W_e ~ C^_e^T Phi_r^T with the units of C^_e the
    columns W_e phi_k (length d_out), so the basis is applied first, once per
    token, z_b = Phi_r^T x_b, and
        y_b = sum over token b's routing entries i of weights[i] C^_e^T z_b,
    fp64 [B][d_out].

    Chat: [E*r][d_out] dequantized units (unit e*r + k is row k of C^_e);
    Vt: [r][d_in] (rows phi_k^T); X: [B][d_in]; routing as ``moe_decode``.
    """
    Chat = np.asarray(Chat, dtype=np.float64)
    Vt = np.asarray(Vt, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    Z = X @ Vt.T
    Y = np.zeros((X.shape[0], Chat.shape[1]))
    for e in range(len(offsets) - 1):
        Ce = Chat[e * r:(e + 1) * r]
        for i in range(int(offsets[e]), int(offsets[e + 1])):
            b = int(tokens[i])
            Y[b] += float(weights[i]) * (Z[b] @ Ce)
    return Y
