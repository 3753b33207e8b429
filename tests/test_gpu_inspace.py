"""GPU parity of the input-space construction of gate/up projections (Sec. 3.2)
against the fp64 oracle (oracle.inspace), through the C ABI.

Stage-wise as in test_gpu_parity.py.  Bars: M_in and C within 1e-3 relative
Frobenius; beta and the loss table within 1e-3 relative per entry; ILP
widths, codes and parameters bit-exact.
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from conftest import gpu_available
from oracle import inspace

pytestmark = pytest.mark.gpu

if not gpu_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2606_00079_amd as bm  # noqa: E402
from paper_2606_00079_amd import pipeline  # noqa: E402

DEV = "cuda:0"
REL = 1e-3


def say(*a):
    print("[gpu-inspace]", *a, flush=True)
    sys.stdout.flush()


def dev(a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def relfro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def l_rel(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-30)))


def _weights(case):
    if case == "tiny_f32":
        return synth.expert_weights(synth.CONFIGS["tiny"], "gate"), "f32"
    if case == "ragged_bf16":
        W = synth.random_rows(3 * 192, 320, seed=31).reshape(3, 192, 320)
        return synth.f32_to_bf16_bits(W), "bf16"
    return synth.expert_weights(synth.CONFIGS["qwen_gate"], "gate"), "bf16"


@pytest.mark.parametrize("case", ["tiny_f32", "ragged_bf16", "qwen_gate_bf16"])
def test_gram_experts_in(case):
    say("gram_experts_in", case)
    W, dt = _weights(case)
    M = bm.gram_experts_in(dev(W, dt)).cpu().numpy()
    ref = inspace.gram_experts_in(synth.as_f64(W, dt))
    err = relfro(M, ref)
    say("rel fro", err)
    assert err <= REL
    assert np.array_equal(M, M.T)


@pytest.mark.parametrize("case,r", [("tiny_f32", 64), ("ragged_bf16", 100), ("qwen_gate_bf16", 384)])
def test_project_in(case, r):
    say("project_in", case, r)
    W, dt = _weights(case)
    d_in = W.shape[2]
    g = np.random.default_rng(7)
    Vt = np.linalg.qr(g.standard_normal((d_in, r)))[0].T.astype(np.float32)
    C = bm.project_in(dev(Vt, "f32"), dev(W, dt)).cpu().numpy()
    ref = inspace.project_in(Vt.astype(np.float64), synth.as_f64(W, dt))
    err = relfro(C, ref)
    say("rel fro", err)
    assert err <= REL


@pytest.mark.parametrize("r,d", [(64, 256), (100, 320), (384, 2048)])
def test_basis_importance(r, d):
    say("basis_importance", r, d)
    g = np.random.default_rng(r + d)
    Vt = np.linalg.qr(g.standard_normal((d, r)))[0].T.astype(np.float32)
    X = synth.random_rows(2 * d, d, seed=d, scale=1.0, heavy=True)
    X[:, ::11] *= 9.0
    H = oracle.gram(X.astype(np.float64)).astype(np.float32)
    b = bm.basis_importance(dev(Vt, "f32"), dev(H, "f32")).cpu().numpy()
    ref = inspace.basis_importance(Vt.astype(np.float64), H.astype(np.float64))
    err = l_rel(b, ref)
    say("max rel", err)
    assert err <= REL


@pytest.mark.parametrize("units,d,r,group,bits", [
    (300, 256, 60, 64, (1, 2, 3, 4)),
    (130, 192, 13, 64, (1, 2, 3, 4, 8)),
    (77, 768, 7, 128, (2, 4)),
    (65, 512, 65, 256, (3,)),
])
def test_score_diag(units, d, r, group, bits):
    say("score_diag", units, d, r, group, bits)
    C = synth.random_rows(units, d, seed=units, scale=0.05, heavy=True)
    C[0] = 0.0
    C[1] = 0.25
    beta = np.exp(np.random.default_rng(d).standard_normal(r)).astype(np.float32)
    L = bm.score_diag(dev(C, "f32"), dev(beta, "f32"), bits, group).cpu().numpy()
    ref = inspace.score_diag(C, beta.astype(np.float64), r, bits, group)
    assert np.all(L[:2] == 0.0)
    err = l_rel(L[2:], ref[2:])
    say("max rel", err)
    assert err <= REL


def _stagewise_in(proj, r, sample_rows=None):
    Wd, Xd = dev(proj.W, proj.dtype), dev(proj.X, proj.dtype)
    res = pipeline.quantize_projection_in(Wd, Xd, r, proj.bits, proj.group, proj.E * r * 2)
    say("pipeline times", res.times)
    W64 = synth.as_f64(proj.W, proj.dtype)
    M = res.M.cpu().numpy()
    assert relfro(M, inspace.gram_experts_in(W64)) <= REL
    Vt = res.Ut.cpu().numpy().astype(np.float64)
    U = Vt.T
    assert np.linalg.norm(M @ U - U * res.eigvals) / np.linalg.norm(M) <= 1e-6
    C = res.C.cpu().numpy()
    assert relfro(C, inspace.project_in(Vt, W64)) <= REL
    H = res.H.cpu().numpy().astype(np.float64)
    beta = res.beta.cpu().numpy()
    bref = inspace.basis_importance(Vt, H)
    assert l_rel(beta, bref) <= REL
    L = res.L.cpu().numpy()
    rows = np.arange(C.shape[0]) if sample_rows is None else sample_rows
    # per-row weights beta[u % r]: with period len(rows) row i gets weight i
    Lref = inspace.score_diag(C[rows], beta.astype(np.float64)[rows % r], len(rows), proj.bits,
                              proj.group)
    assert l_rel(L[rows], Lref) <= REL
    # ILP on the device's own table, then pack, bit for bit
    bref_u, _ = oracle.allocate_dp(L, proj.bits, proj.E * r * 2)
    assert np.array_equal(res.bits_u, bref_u)
    rc, rp, roff = oracle.pack(C, res.bits_u, proj.group)
    assert np.array_equal(res.offsets, roff)
    assert np.array_equal(res.codes.cpu().numpy().view(np.uint64)[: len(rc)], rc)
    assert np.array_equal(res.params.cpu().numpy().view(np.uint16), rp)


def test_end_to_end_inspace_tiny():
    say("end-to-end input-space tiny")
    _stagewise_in(synth.make_projection("tiny"), r=64)


def test_end_to_end_inspace_qwen_gate_full_size():
    say("end-to-end input-space qwen gate (E=128, 768x2048, r=384)")
    proj = synth.make_projection("qwen_gate")
    rows = np.sort(np.random.default_rng(0).choice(proj.E * 384, size=384, replace=False))
    _stagewise_in(proj, r=384, sample_rows=rows)
