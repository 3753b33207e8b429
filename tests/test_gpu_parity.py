"""GPU parity: every step of the HIP path against the fp64 oracle.

Stage-wise: each device step is fed the same inputs as the oracle step it is
compared with (the device's own upstream outputs, copied to the host), so
errors do not compound and near-degenerate eigenvectors cannot make two
correct results look different.

Bars (written in each test): H, M, C and U within 1e-3 relative Frobenius;
L within 1e-3 relative per entry; ILP widths, codes and scale/min parameters
bit-exact.
"""
import math
import sys

import numpy as np
import pytest

import oracle
import synth
from conftest import gpu_available, oracle_score_threaded

pytestmark = pytest.mark.gpu

if not gpu_available():  # pragma: no cover - collected on CPU but skipped
    pytest.skip("no GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2606_00079_amd as bm  # noqa: E402
from paper_2606_00079_amd import pipeline  # noqa: E402

DEV = "cuda:0"
REL = 1e-3


def say(*a):
    print("[gpu-parity]", *a, flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray, dtype: str):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def f64(a: np.ndarray, dtype: str) -> np.ndarray:
    return synth.as_f64(a, dtype)


def relfro(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def l_rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.maximum(np.abs(ref), 1e-30)
    return float(np.max(np.abs(got - ref) / den))


# ------------------------------------------------------------------------- H
@pytest.mark.parametrize("case", ["tiny_f32", "ragged_bf16", "ragged_f32", "qwen_bf16"])
def test_gram(case):
    say("gram", case)
    if case == "tiny_f32":
        X = synth.calibration_input(synth.CONFIGS["tiny"], "gate")
        dt = "f32"
    elif case == "ragged_bf16":
        X = synth.f32_to_bf16_bits(synth.random_rows(1001, 320, seed=1, scale=1.0, heavy=True))
        dt = "bf16"
    elif case == "ragged_f32":
        X = synth.random_rows(77, 192, seed=2, scale=3.0)
        dt = "f32"
    else:
        X = synth.calibration_input(synth.CONFIGS["qwen_gate"], "gate")
        dt = "bf16"
    H = bm.gram(dev(X, dt)).cpu().numpy()
    ref = oracle.gram(f64(X, dt))
    err = relfro(H, ref)
    say("gram", case, "rel fro", err)
    assert err <= REL
    assert np.array_equal(H, H.T)
    # per-entry: diagonal to fp32 accuracy
    assert l_rel(np.diag(H), np.diag(ref)) < 1e-5


# ------------------------------------------------------------------------- M
@pytest.mark.parametrize("case", ["tiny_f32", "ragged_bf16", "qwen_gate_bf16"])
def test_gram_experts(case):
    say("gram_experts", case)
    if case == "tiny_f32":
        W = synth.expert_weights(synth.CONFIGS["tiny"], "gate")
        dt = "f32"
    elif case == "ragged_bf16":
        W = synth.f32_to_bf16_bits(synth.random_rows(3 * 192, 320, seed=3).reshape(3, 192, 320))
        dt = "bf16"
    else:
        W = synth.expert_weights(synth.CONFIGS["qwen_gate"], "gate")
        dt = "bf16"
    M = bm.gram_experts(dev(W, dt)).cpu().numpy()
    ref = oracle.gram_experts(f64(W, dt))
    err = relfro(M, ref)
    say("gram_experts", case, "rel fro", err)
    assert err <= REL
    assert np.array_equal(M, M.T)
    assert abs(np.trace(M) - np.trace(ref)) <= 1e-5 * np.trace(ref)


def test_gram_experts_deterministic():
    say("gram_experts determinism")
    W = dev(synth.expert_weights(synth.CONFIGS["qwen_gate"], "gate", experts=range(16)), "bf16")
    a = bm.gram_experts(W).cpu().numpy()
    b = bm.gram_experts(W).cpu().numpy()
    assert np.array_equal(a, b)


# ------------------------------------------------------------------------- U
@pytest.mark.parametrize("case", ["planted", "tiny", "qwen_gate"])
def test_shared_basis(case):
    say("shared_basis", case)
    if case == "planted":
        g = np.random.default_rng(4)
        Q = np.linalg.qr(g.standard_normal((128, 128)))[0]
        lam = np.linspace(100.0, 1.0, 128)
        M = (Q * lam) @ Q.T
        r = 20
    elif case == "tiny":
        W = synth.expert_weights(synth.CONFIGS["tiny"], "gate").astype(np.float64)
        M = oracle.gram_experts(W)
        r = 64
    else:
        Wb = synth.expert_weights(synth.CONFIGS["qwen_gate"], "gate", experts=range(32))
        M = oracle.gram_experts(f64(Wb, "bf16"))
        r = 384
    Md = torch.from_numpy(M).to(DEV)
    Ut, ev, ms = bm.shared_basis(Md, r)
    Ut = Ut.cpu().numpy().astype(np.float64)
    Uo, evo = oracle.shared_basis(M, r)
    say("shared_basis", case, "host ms", ms)
    assert np.allclose(ev, evo, rtol=1e-9, atol=1e-12 * evo[0])
    U = Ut.T
    res = np.linalg.norm(M @ U - U * ev) / np.linalg.norm(M)
    orth = np.abs(Ut @ U - np.eye(r)).max()
    say("shared_basis", case, "residual", res, "orth", orth)
    assert res <= 1e-6
    assert orth <= 1e-6
    for k in range(r):
        i = int(np.argmax(np.abs(Ut[k])))
        assert Ut[k, i] > 0
    # eigenvectors with a clear gap must agree with the oracle's
    gaps = np.minimum(np.abs(np.diff(np.r_[np.inf, evo])), np.abs(np.diff(np.r_[evo, -np.inf])))
    clear = gaps > 1e-6 * evo[0]
    if case != "qwen_gate":
        assert clear.sum() > 0
    for k in np.nonzero(clear)[0]:
        assert np.abs(Ut[k] - Uo[k]).max() < 1e-5


# ------------------------------------------------------------------------- C
@pytest.mark.parametrize("case", ["tiny_f32", "ragged_bf16", "qwen_gate_bf16"])
def test_project(case):
    say("project", case)
    g = np.random.default_rng(5)
    if case == "tiny_f32":
        W = synth.expert_weights(synth.CONFIGS["tiny"], "gate")
        dt, r = "f32", 64
    elif case == "ragged_bf16":
        W = synth.f32_to_bf16_bits(synth.random_rows(3 * 192, 320, seed=6).reshape(3, 192, 320))
        dt, r = "bf16", 100
    else:
        W = synth.expert_weights(synth.CONFIGS["qwen_gate"], "gate")
        dt, r = "bf16", 384
    d_out = W.shape[1]
    Ut = np.linalg.qr(g.standard_normal((d_out, r)))[0].T.astype(np.float32)
    C = bm.project(dev(Ut, "f32"), dev(W, dt)).cpu().numpy()
    ref = oracle.project(Ut.astype(np.float64), f64(W, dt))
    err = relfro(C, ref)
    say("project", case, "rel fro", err)
    assert err <= REL
    # per row as well: every unit's factor row within the bar
    rows = np.linalg.norm(C - ref, axis=1) / np.linalg.norm(ref, axis=1)
    assert rows.max() <= REL


@pytest.mark.parametrize("case", ["beyond_fp16", "non_finite", "tiny_and_subnormal",
                                  "tiny_expert"])
@pytest.mark.parametrize("shape", ["ragged", "whole_tiles", "persistent"])
def test_project_bf16_outside_fp16_range(case, shape):
    """bf16 W is multiplied in one fp16 pass; entries beyond fp16's range
    (|W| > 65504) make that pass non-finite, and the library then recomputes
    C exactly in the two-pass bf16 form: C is finite and within the bar.  A
    non-finite W stays non-finite.  Entries far below fp16's normal range
    lose only absolute precision (at most 2^-25 each), far below the bar
    next to normal entries; a tile of factors that are all small (an expert
    of tiny weights) is recomputed exactly."""
    say("project outside fp16 range", case, shape)
    g = np.random.default_rng(8)
    # ragged: partial row and column tiles (bounds-tested stores);
    # whole_tiles: r = 128 rows and d_in = 512 columns fill the tiles exactly;
    # persistent: the same tiles over 160 experts, more tiles (320) than
    # compute units, so one persistent workgroup per CU walks several
    E, d_out, d_in, r = {"ragged": (3, 192, 320, 100), "whole_tiles": (3, 192, 512, 128),
                         "persistent": (160, 192, 512, 128)}[shape]
    Wf = synth.random_rows(E * d_out, d_in, seed=9).reshape(E, d_out, d_in)
    if case == "beyond_fp16":
        Wf[1, 7, 11] = 1.5e5
        Wf[2, 100, 300] = -7.0e4
    elif case == "non_finite":
        Wf[0, 3, 5] = np.inf
    elif case == "tiny_expert":
        Wf[0] *= 2.0 ** -30          # a whole expert below fp16's range (~1e-11)
        Wf[2, :, 128:] *= 2.0 ** -20
    else:
        m = np.random.default_rng(10).random(Wf.shape) < 0.1   # a tenth of the entries tiny
        Wf[m] *= 2.0 ** -20          # ~1e-8: fp16 subnormal or zero
        Wf[1, :, :64] *= 2.0 ** -12
    W = synth.f32_to_bf16_bits(Wf)
    Ut = np.linalg.qr(g.standard_normal((d_out, r)))[0].T.astype(np.float32)
    C = bm.project(dev(Ut, "f32"), dev(W, "bf16")).cpu().numpy().reshape(E, r, d_in)
    W64 = f64(W, "bf16")
    if case == "non_finite":
        assert not np.all(np.isfinite(C))
        return
    assert np.all(np.isfinite(C))
    for e in range(E):
        ref = oracle.project(Ut.astype(np.float64), W64[e:e + 1])
        err = relfro(C[e], ref)
        say("expert", e, "rel fro", err)
        assert err <= REL


# ------------------------------------------------------------------------- L
SCORE_CASES = [
    # (name, units, d, group, bits, heavy)
    ("tiny", None, None, None, None, None),
    ("ragged_units", 257, 256, 64, (1, 2, 3, 4), False),
    ("ragged_tile_d", 130, 192, 64, (1, 2, 3, 4), True),
    ("group32_bits8", 70, 256, 32, (1, 2, 3, 4, 8), False),
    ("group256", 40, 512, 256, (2, 4), True),
    ("one_width", 33, 128, 128, (3,), False),
    # paired-triangle schedule: odd and even row-tile counts, partial last K
    # block, an odd number of column tiles (the last unit is half empty)
    ("odd_row_tiles", 130, 704, 64, (1, 2, 3, 4), True),
    ("five_row_tiles", 70, 1280, 128, (2, 3, 4), False),
    ("four_row_tiles_ragged", 64, 960, 64, (1, 2, 3, 4), False),
    # rows ending in a 256-entry chunk of 4 entries per lane (d % 512 == 256):
    # groups of 32 lanes (lane ^ 16 by swizzle) and of 64 (lane ^ 32 too)
    ("tail_chunk_768", 90, 768, 128, (1, 2, 3, 4), False),
    ("tail_chunk_group256", 40, 768, 256, (2, 4), True),
]


def _score_inputs(case):
    name, units, d, group, bits, heavy = case
    if name == "tiny":
        cfg = synth.CONFIGS["tiny"]
        W = synth.expert_weights(cfg, "gate").astype(np.float64)
        X = synth.calibration_input(cfg, "gate")
        Ut, _ = oracle.shared_basis(oracle.gram_experts(W), 64)
        C = oracle.project(Ut, W).astype(np.float32)
        H = oracle.gram(X.astype(np.float64)).astype(np.float32)
        return C, H, cfg.group, cfg.bits
    C = synth.random_rows(units, d, seed=units + d, scale=0.05, heavy=heavy)
    X = synth.random_rows(2 * d, d, seed=d, scale=1.0, heavy=heavy)
    X[:, ::17] *= 10.0
    H = oracle.gram(X.astype(np.float64)).astype(np.float32)
    return C, H, group, bits


@pytest.mark.parametrize("case", SCORE_CASES, ids=lambda c: c[0])
def test_score(case):
    say("score", case[0])
    C, H, group, bits = _score_inputs(case)
    L = bm.score(dev(C, "f32"), dev(H, "f32"), bits, group).cpu().numpy()
    ref = oracle.score(C, H.astype(np.float64), bits, group)
    err = l_rel(L, ref)
    say("score", case[0], "max rel", err)
    assert np.all(L >= 0)
    assert err <= REL


def test_score_deterministic_and_degenerate_rows():
    say("score degenerate")
    C = synth.random_rows(64, 256, seed=9)
    C[0] = 0.0                      # all-zero unit: L = 0 at every width
    C[1] = 0.125                    # constant unit, fp16-exact: L = 0
    C[2, ::2] = 0.9375              # two-level unit whose range / (2^b - 1) is
    C[2, 1::2] = 0.0                # fp16-exact at b = 1, 2, 4: reproduced exactly
    g = np.random.default_rng(1)
    X = g.standard_normal((300, 256)).astype(np.float32)
    H = oracle.gram(X.astype(np.float64)).astype(np.float32)
    Cd, Hd = dev(C, "f32"), dev(H, "f32")
    a = bm.score(Cd, Hd, [1, 2, 4], 64).cpu().numpy()
    b = bm.score(Cd, Hd, [1, 2, 4], 64).cpu().numpy()
    assert np.array_equal(a, b)
    assert np.all(a[:3] == 0)
    ref = oracle.score(C, H.astype(np.float64), [1, 2, 4], 64)
    assert l_rel(a[3:], ref[3:]) <= REL


# ---------------------------------------------------------------------- pack
@pytest.mark.parametrize("group,d,units", [(64, 256, 300), (128, 2048, 97), (32, 192, 65),
                                           (256, 768, 40), (128, 768, 90), (32, 1280, 33)])
def test_pack_bit_exact(group, d, units):
    say("pack", group, d, units)
    g = np.random.default_rng(group + d)
    C = synth.random_rows(units, d, seed=units, scale=0.04, heavy=True)
    C[0] = 0.0
    C[1] = 0.3
    bits_u = g.choice([1, 2, 3, 4, 8], size=units).astype(np.uint8)
    off = bm.pack_layout(bits_u, d)
    bd = torch.from_numpy(bits_u).to(DEV)
    od = torch.from_numpy(off).to(DEV)
    codes, params = bm.pack(dev(C, "f32"), bd, od, group, int(off[-1]))
    rc, rp, roff = oracle.pack(C, bits_u, group)
    assert np.array_equal(off, roff)
    assert np.array_equal(codes.cpu().numpy().view(np.uint64), rc)
    assert np.array_equal(params.cpu().numpy().view(np.uint16), rp)
    xh = bm.unpack(codes, params, bd, od, units, d, group, int(off[-1])).cpu().numpy()
    ref = oracle.unpack(rc, rp, bits_u, d, group)
    assert np.array_equal(xh.astype(np.float64), ref)


@pytest.mark.parametrize("group,d", [(128, 2048), (64, 192)])
def test_pack_surrogate_widths_bit_exact(group, d):
    """Widths of the surrogate's candidate set, eviction (0) and fp16 rows
    (16) included, packed and unpacked bit for bit as the oracle does."""
    say("pack surrogate widths", group, d)
    units = 211
    g = np.random.default_rng(group + d + 1)
    C = synth.random_rows(units, d, seed=units + d, scale=0.04, heavy=True)
    C[0] = 0.0
    bits_u = g.choice([0, 1, 2, 3, 4, 6, 8, 16], size=units).astype(np.uint8)
    bits_u[:3] = [16, 0, 16]
    off = bm.pack_layout(bits_u, d)
    bd = torch.from_numpy(bits_u).to(DEV)
    od = torch.from_numpy(off).to(DEV)
    codes, params = bm.pack(dev(C, "f32"), bd, od, group, int(off[-1]))
    rc, rp, roff = oracle.pack(C, bits_u, group)
    assert np.array_equal(off, roff)
    assert np.array_equal(codes.cpu().numpy().view(np.uint64)[: len(rc)], rc)
    assert np.array_equal(params.cpu().numpy().view(np.uint16), rp)
    xh = bm.unpack(codes, params, bd, od, units, d, group, int(off[-1])).cpu().numpy()
    assert np.array_equal(xh.astype(np.float64), oracle.unpack(rc, rp, bits_u, d, group))


# -------------------------------------------------------------- end to end
def _stagewise(proj, check_ilp=True):
    """Run the pipeline and check each stage on the device's own inputs:
    every row of L, the ILP's widths and every unit's codes and parameters."""
    W, X = proj.W, proj.X
    Wd, Xd = dev(W, proj.dtype), dev(X, proj.dtype)
    res = pipeline.quantize_projection(Wd, Xd, proj.r, proj.bits, proj.group, proj.budget_bits)
    say("pipeline times", res.times)
    W64, X64 = f64(W, proj.dtype), f64(X, proj.dtype)
    # H and M against the oracle from the inputs
    assert relfro(res.H.cpu().numpy(), oracle.gram(X64)) <= REL
    M = res.M.cpu().numpy()
    assert relfro(M, oracle.gram_experts(W64)) <= REL
    # U: invariants on the device's own M
    Ut = res.Ut.cpu().numpy().astype(np.float64)
    U = Ut.T
    assert np.linalg.norm(M @ U - U * res.eigvals) / np.linalg.norm(M) <= 1e-6
    # C from the device's U
    C = res.C.cpu().numpy()
    Cref = oracle.project(res.Ut.cpu().numpy().astype(np.float64), W64)
    assert relfro(C, Cref) <= REL
    del Cref
    # L from the device's C and H, every row
    H = res.H.cpu().numpy().astype(np.float64)
    L = res.L.cpu().numpy()
    Lref = oracle_score_threaded(C, H, proj.bits, proj.group)
    err = l_rel(L, Lref)
    say("L max rel over all", L.shape[0], "units", err)
    assert err <= REL
    # ILP from the device's L: bit-exact
    if check_ilp:
        bref, _ = oracle.allocate_dp(L, proj.bits, proj.budget_bits)
        assert np.array_equal(res.bits_u, bref)
        say("ILP widths equal the oracle DP")
    # codes and params of every unit from the device's C and widths: bit-exact
    rc, rp, ro = oracle.pack(C, res.bits_u, proj.group)
    assert np.array_equal(res.offsets, ro)
    codes = res.codes.cpu().numpy().view(np.uint64)
    params = res.params.cpu().numpy().view(np.uint16)
    assert np.array_equal(codes[: len(rc)], rc)
    assert np.array_equal(params, rp)
    say("codes and params of all units bit-exact")
    assert int(res.bits_u.astype(np.int64).sum()) <= proj.budget_bits
    return res


def test_end_to_end_tiny():
    say("end-to-end tiny")
    proj = synth.make_projection("tiny")
    a = _stagewise(proj)
    # determinism of the whole path
    b = pipeline.quantize_projection(dev(proj.W, "f32"), dev(proj.X, "f32"), proj.r, proj.bits,
                                     proj.group, proj.budget_bits)
    assert np.array_equal(a.L.cpu().numpy(), b.L.cpu().numpy())
    assert np.array_equal(a.bits_u, b.bits_u)
    assert np.array_equal(a.codes.cpu().numpy(), b.codes.cpu().numpy())


def test_end_to_end_qwen_gate_full_size():
    say("end-to-end qwen gate (E=128, 768x2048, r=384)")
    proj = synth.make_projection("qwen_gate")
    _stagewise(proj, check_ilp=True)
