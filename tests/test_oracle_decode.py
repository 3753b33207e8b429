"""Pins of the oracle's stage-3 decode (serving the layer from packed factors).

The decode is tied to the original weights: with the full basis (r = d_out)
and every unit stored in fp16 (width 16), U C^ x reproduces the dense MoE
output sum_j g_j W_e x up to fp16 rounding of the factors; narrower codes
approximate it less well, in order.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import decode


def _layer(seed=0):
    cfg = synth.CONFIGS["tiny"]
    W = synth.expert_weights(cfg, "gate").astype(np.float64)   # E=4, 128 x 256
    X = synth.calibration_input(cfg, "gate")[:24].astype(np.float64)
    off, tok, w = synth.routing(cfg, X.astype(np.float32))
    return cfg, W, X, off, tok, w


def _decode_at(W, X, off, tok, w, r, width, G=64):
    E, d_out, d_in = W.shape
    Ut, _ = oracle.shared_basis(oracle.gram_experts(W), r)
    C = oracle.project(Ut, W).astype(np.float32)
    bits_u = np.full(E * r, width, dtype=np.uint8)
    codes, params, _ = oracle.pack(C, bits_u, G)
    Chat = decode.dequantized_factors(codes, params, bits_u, d_in, G)
    return decode.moe_decode(Chat, r, Ut, X, off, tok, w)


def test_full_basis_fp16_factors_reproduce_the_dense_layer():
    cfg, W, X, off, tok, w = _layer()
    Y = _decode_at(W, X, off, tok, w, r=W.shape[1], width=16)
    Yd = decode.moe_dense(W, X, off, tok, w)
    err = np.linalg.norm(Y - Yd) / np.linalg.norm(Yd)
    assert err < 2 ** -11, err


def test_error_shrinks_with_the_width():
    cfg, W, X, off, tok, w = _layer()
    Yd = decode.moe_dense(W, X, off, tok, w)
    errs = [np.linalg.norm(_decode_at(W, X, off, tok, w, 128, b) - Yd) for b in (2, 3, 4, 8, 16)]
    assert all(a > b for a, b in zip(errs, errs[1:])), errs


def test_evicted_units_and_unrouted_tokens():
    """Width 0 units contribute nothing; a token with no routing entry gets y = 0."""
    cfg, W, X, off, tok, w = _layer()
    E, d_out, d_in = W.shape
    r = 64
    Ut, _ = oracle.shared_basis(oracle.gram_experts(W), r)
    C = oracle.project(Ut, W).astype(np.float32)
    bits_u = np.full(E * r, 4, dtype=np.uint8)
    bits_u[r:2 * r] = 0                       # expert 1 evicted entirely
    codes, params, _ = oracle.pack(C, bits_u, 64)
    Chat = decode.dequantized_factors(codes, params, bits_u, d_in, 64)
    keep = tok != 5                           # drop token 5's entries
    offs = np.r_[0, np.cumsum([np.sum(keep[off[e]:off[e + 1]]) for e in range(E)])]
    Y = decode.moe_decode(Chat, r, Ut, X, offs, tok[keep], w[keep])
    assert np.all(Y[5] == 0)
    # expert 1's entries change nothing
    e1 = np.zeros_like(keep)
    e1[off[1]:off[2]] = True
    m = keep & ~e1
    offs2 = np.r_[0, np.cumsum([np.sum(m[off[e]:off[e + 1]]) for e in range(E)])]
    np.testing.assert_allclose(decode.moe_decode(Chat, r, Ut, X, offs2, tok[m], w[m]), Y, rtol=1e-12,
                               atol=1e-14)


# ---- input-space form (gate/up): y = sum_j g_j C^_e^T (Phi^T x) ----

def _decode_in_at(W, X, off, tok, w, r, width, G=64, Vt=None):
    from oracle import inspace
    E, d_out, d_in = W.shape
    if Vt is None:
        Vt, _ = oracle.shared_basis(inspace.gram_experts_in(W), r)
    C = inspace.project_in(Vt, W).astype(np.float32)   # [E*r][d_out]
    bits_u = np.full(E * r, width, dtype=np.uint8)
    codes, params, _ = oracle.pack(C, bits_u, G)
    Chat = decode.dequantized_factors(codes, params, bits_u, d_out, G)
    return decode.moe_decode_in(Chat, r, Vt, X, off, tok, w)


def test_input_space_full_basis_fp16_units_reproduce_the_dense_layer():
    cfg, W, X, off, tok, w = _layer()
    Y = _decode_in_at(W, X, off, tok, w, r=W.shape[2], width=16)
    Yd = decode.moe_dense(W, X, off, tok, w)
    err = np.linalg.norm(Y - Yd) / np.linalg.norm(Yd)
    assert err < 2 ** -11, err


def test_input_space_identity_basis_is_a_dequantized_gemv():
    """Phi = I (r = d_in): units are the columns of W_e, so the decode is the
    routed GEMV with the dequantized transposed weights, by explicit loops."""
    cfg, W, X, off, tok, w = _layer()
    E, d_out, d_in = W.shape
    Vt = np.eye(d_in)
    C = np.concatenate([W[e].T for e in range(E)]).astype(np.float32)   # [E*d_in][d_out]
    bits_u = np.full(E * d_in, 3, dtype=np.uint8)
    codes, params, _ = oracle.pack(C, bits_u, 64)
    Chat = decode.dequantized_factors(codes, params, bits_u, d_out, 64)
    Y = decode.moe_decode_in(Chat, d_in, Vt, X, off, tok, w)
    ref = np.zeros((X.shape[0], d_out))
    for e in range(E):
        We = Chat[e * d_in:(e + 1) * d_in].T                # dequantized W_e
        for i in range(off[e], off[e + 1]):
            for o in range(d_out):
                ref[tok[i], o] += w[i] * sum(We[o, j] * X[tok[i], j] for j in range(0, d_in, 1))
    np.testing.assert_allclose(Y, ref, rtol=1e-10, atol=1e-12)


def test_input_space_error_shrinks_with_the_width():
    cfg, W, X, off, tok, w = _layer()
    Yd = decode.moe_dense(W, X, off, tok, w)
    errs = [np.linalg.norm(_decode_in_at(W, X, off, tok, w, 128, b) - Yd) for b in (2, 3, 4, 8, 16)]
    assert all(a > b for a, b in zip(errs, errs[1:])), errs


def test_input_space_evicted_units_and_unrouted_tokens():
    from oracle import inspace
    cfg, W, X, off, tok, w = _layer()
    E, d_out, d_in = W.shape
    r = 64
    Vt, _ = oracle.shared_basis(inspace.gram_experts_in(W), r)
    C = inspace.project_in(Vt, W).astype(np.float32)
    bits_u = np.full(E * r, 4, dtype=np.uint8)
    bits_u[2 * r:3 * r] = 0                   # expert 2 evicted entirely
    codes, params, _ = oracle.pack(C, bits_u, 64)
    Chat = decode.dequantized_factors(codes, params, bits_u, d_out, 64)
    keep = tok != 7
    offs = np.r_[0, np.cumsum([np.sum(keep[off[e]:off[e + 1]]) for e in range(E)])]
    Y = decode.moe_decode_in(Chat, r, Vt, X, offs, tok[keep], w[keep])
    assert np.all(Y[7] == 0)
    m = keep.copy()
    m[off[2]:off[3]] = False
    offs2 = np.r_[0, np.cumsum([np.sum(m[off[e]:off[e + 1]]) for e in range(E)])]
    np.testing.assert_allclose(decode.moe_decode_in(Chat, r, Vt, X, offs2, tok[m], w[m]), Y,
                               rtol=1e-12, atol=1e-14)
