"""Pins for the oracle's quantizer, loss table and packing."""
import json
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ------------------------------------------------------------------ quantizer
@pytest.mark.parametrize("case", _load("quant_examples.json")["cases"], ids=lambda c: c["name"])
def test_quantizer_hand_examples(case):
    c = np.array(case["c"], dtype=np.float32)
    G = c.shape[0]
    q, s16, m16 = oracle.quant_group(c, case["b"], G)
    assert q[0].tolist() == case["q"]
    assert float(s16[0, 0]) == case["s16"]
    assert float(m16[0, 0]) == case["m16"]
    assert oracle.fake_quant(c, case["b"], G)[0].tolist() == case["x_hat"]


def test_quantizer_matches_nearest_level_search():
    # Brute force: the nearest of the 2^b levels m16 + q*s16 (ties excluded).
    g = np.random.default_rng(11)
    c = (g.standard_normal((40, 256)) * 0.03).astype(np.float32)
    G = 64
    for b in (1, 2, 3, 4, 8):
        q, s16, m16 = oracle.quant_group(c, b, G)
        levels_q = np.arange(2 ** b, dtype=np.float64)
        for r in range(c.shape[0]):
            for grp in range(256 // G):
                s = float(s16[r, grp]); m = float(m16[r, grp])
                x = c[r, grp * G:(grp + 1) * G].astype(np.float64)
                dist = np.abs(x[:, None] - (m + levels_q[None, :] * s))
                best = np.argmin(dist, axis=1)
                srt = np.sort(dist, axis=1)
                clear = srt[:, 1] - srt[:, 0] > 1e-12 * max(s, 1e-30)
                assert np.array_equal(q[r, grp * G:(grp + 1) * G][clear], best[clear])


def test_quantizer_bounds_and_error():
    g = np.random.default_rng(12)
    c = (g.standard_t(3, size=(30, 512)) * 0.02).astype(np.float32)
    G = 128
    for b in (1, 2, 3, 4, 8):
        q, s16, m16 = oracle.quant_group(c, b, G)
        assert q.min() >= 0 and q.max() <= 2 ** b - 1
        xh = oracle.fake_quant(c, b, G)
        s = np.repeat(s16.astype(np.float64), G, axis=1)
        m = np.repeat(m16.astype(np.float64), G, axis=1)
        # inside the clamped range the error is at most half a step
        inner = (q > 0) & (q < 2 ** b - 1)
        err = np.abs(c.astype(np.float64) - xh)
        assert np.all(err[inner] <= 0.5 * s[inner] * (1 + 1e-12))
        # at the ends the error is bounded by the fp16 rounding of m and s
        slack = np.abs(m - np.repeat(c.reshape(30, -1, G).min(axis=2), G, axis=1)) \
            + (2 ** b - 1) * 2.0 ** -11 * s + 0.5 * s
        assert np.all(err <= slack * (1 + 1e-9) + 1e-30)


def test_two_level_group_is_exact_at_one_bit():
    # A group holding two fp16-representable values is reproduced exactly.
    c = np.array([[0.25, -0.5, 0.25, -0.5, -0.5, 0.25, 0.25, 0.25]], dtype=np.float32)
    assert np.array_equal(oracle.fake_quant(c, 1, 8)[0], c[0].astype(np.float64))


def test_degenerate_group_codes_zero():
    c = np.full((1, 64), 0.123, dtype=np.float32)
    q, s16, m16 = oracle.quant_group(c, 4, 64)
    assert not q.any() and float(s16[0, 0]) == 0.0


# ---------------------------------------------------------------------- score
def _tiny_problem(seed=0):
    cfg = synth.CONFIGS["tiny"]
    W = synth.expert_weights(cfg, "gate", seed=seed).astype(np.float64)
    X = synth.calibration_input(cfg, "gate", seed=seed).astype(np.float64)
    return cfg, W, X


def test_loss_equals_brute_force_output_error():
    # L = ||X delta^T||^2 / n, from the activations rather than from H.
    cfg, W, X = _tiny_problem()
    H = oracle.gram(X)
    Ut, _ = oracle.shared_basis(oracle.gram_experts(W), 64)
    C = oracle.project(Ut, W)[:48].astype(np.float32)
    L = oracle.score(C, H, cfg.bits, cfg.group)
    assert L.min() >= 0
    n = X.shape[0]
    for j, b in enumerate(cfg.bits):
        delta = C.astype(np.float64) - oracle.fake_quant(C, b, cfg.group)
        brute = np.array([np.sum((X @ dlt) ** 2) / n for dlt in delta])
        np.testing.assert_allclose(L[:, j], brute, rtol=1e-10)


def test_loss_with_identity_h_is_rtn_mse():
    c = synth.random_rows(20, 256, seed=3)
    L = oracle.score(c, np.eye(256), [1, 2, 3, 4], 64)
    for j, b in enumerate([1, 2, 3, 4]):
        delta = c.astype(np.float64) - oracle.fake_quant(c, b, 64)
        np.testing.assert_allclose(L[:, j], np.sum(delta * delta, axis=1), rtol=1e-13)


def test_loss_is_additive_pythagorean_identity():
    # For any width assignment, the output error of the reconstructed expert
    # splits exactly into the per-unit losses plus the basis-truncation loss:
    # ||(W_e - U C_hat_e) X^T||^2/n = sum_k L[e*r+k, b_k] + ||(I-UU^T) W_e X^T||^2/n.
    cfg, W, X = _tiny_problem(seed=1)
    r, G = 64, cfg.group
    H = oracle.gram(X)
    Ut, _ = oracle.shared_basis(oracle.gram_experts(W), r)
    C = oracle.project(Ut, W)                         # fp64 factors
    L = oracle.score(C, H, cfg.bits, G)               # delta = C - Q(fp32 C)
    g = np.random.default_rng(5)
    n = X.shape[0]
    for e in range(W.shape[0]):
        js = g.integers(0, len(cfg.bits), size=r)
        Ce = C[e * r:(e + 1) * r]
        Chat = np.stack([oracle.fake_quant(Ce[k].astype(np.float32), cfg.bits[js[k]], G)[0]
                         for k in range(r)])
        Y = (W[e] - Ut.T @ Chat) @ X.T
        lhs = np.sum(Y * Y) / n
        rhs = sum(L[e * r + k, js[k]] for k in range(r)) + oracle.truncation_loss(Ut, W[e], X)
        assert np.isclose(lhs, rhs, rtol=1e-9)


def test_loss_of_evicted_unit_is_energy_times_beta():
    # With delta = c (the zero-bit case of App. B.3) the loss is alpha^2 p^T H p,
    # the paper's down_proj beta surrogate, exact only under eviction
    # (App. B.2, Eq. app_down_beta_approx).  Our score with a quantizer output
    # of zero is reproduced by scoring rows whose groups are degenerate at 0.
    g = np.random.default_rng(6)
    X = g.standard_normal((100, 128))
    H = oracle.gram(X)
    c = g.standard_normal(128)
    alpha = np.linalg.norm(c)
    p = c / alpha
    delta = c - 0.0
    assert np.isclose(delta @ H @ delta, alpha ** 2 * (p @ H @ p), rtol=1e-13)
    # and the oracle's loss of a row that quantizes exactly equals zero
    z = np.zeros((1, 128), dtype=np.float32)
    assert np.all(oracle.score(z, H, [1, 2], 64) == 0)


# ---------------------------------------------------------------------- pack
def test_bitplanes_closed_form():
    gold = _load("bitplanes.json")
    words = oracle.bit_planes(np.arange(64), gold["b"])
    assert [format(int(w[0]), "016x") for w in words] == gold["planes_hex"]


def test_pack_roundtrip_and_size():
    g = np.random.default_rng(13)
    units, d, G = 37, 256, 64
    c = (g.standard_normal((units, d)) * 0.05).astype(np.float32)
    bits_u = g.choice([1, 2, 3, 4, 8], size=units).astype(np.uint8)
    codes, params, off = oracle.pack(c, bits_u, G)
    assert codes.nbytes == int(np.sum(bits_u.astype(np.int64) * d // 8))
    assert params.nbytes == units * (d // G) * 4
    xh = oracle.unpack(codes, params, bits_u, d, G)
    for u in range(units):
        assert np.array_equal(xh[u], oracle.fake_quant(c[u], int(bits_u[u]), G)[0])
    # codes decoded from planes equal the quantizer's codes
    for u in range(units):
        b = int(bits_u[u])
        q, _, _ = oracle.quant_group(c[u], b, G)
        planes = codes[off[u]:off[u + 1]].reshape(b, d // 64)
        assert np.array_equal(planes, oracle.bit_planes(q[0], b))


def test_pack_eviction_and_fp16_widths():
    """Widths 0 (evicted) and 16 (fp16 row) of the surrogate's candidate set:
    sizes b d / 8 bytes, fp16 entries four to a little-endian word (hand-made
    words: 1.0 = 0x3C00, -2.0 = 0xC000, 0.5 = 0x3800, 65504 = 0x7BFF)."""
    d, G = 64, 32
    c = np.zeros((3, d), dtype=np.float32)
    c[:, :4] = [1.0, -2.0, 0.5, 65504.0]
    c[:, 4:] = np.linspace(-1, 1, d - 4, dtype=np.float32)
    bits_u = np.array([16, 0, 2], dtype=np.uint8)
    codes, params, off = oracle.pack(c, bits_u, G)
    assert list(off) == [0, 16, 16, 18]
    assert int(codes[0]) == 0x7BFF3800C0003C00
    assert np.all(params[:2] == 0)
    xh = oracle.unpack(codes, params, bits_u, d, G)
    assert np.array_equal(xh[0], c[0].astype(np.float16).astype(np.float64))
    assert np.all(xh[1] == 0.0)
    assert np.array_equal(xh[2], oracle.fake_quant(c[2], 2, G)[0])
