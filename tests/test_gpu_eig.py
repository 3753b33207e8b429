"""GPU parity of the device eigensolver (bitsmoe_shared_basis_gpu) against
the oracle's shared basis (numpy eigh in fp64) and the host LAPACK path.

Bars: eigenvalues within 1e-11 of lambda_max; with well separated
eigenvalues the fp32 eigenvectors (sign rule applied) within 2e-6 of the
oracle's; inside clusters, where eigenvectors are not unique, the residual
||M U - U Lambda|| / ||M|| and orthonormality within fp32 rounding and the
subspace of the separated leading eigenvalues within 1e-6 (projector norm).
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from conftest import gpu_available

pytestmark = pytest.mark.gpu

if not gpu_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2606_00079_amd as bm  # noqa: E402

DEV = "cuda:0"


def say(*a):
    print("[gpu-eig]", *a, flush=True)
    sys.stdout.flush()


def _separated(n, seed):
    """M = Q diag(1..n) Q^T (gaps of 1) with a random orthogonal Q."""
    g = np.random.default_rng(seed)
    Q = np.linalg.qr(g.standard_normal((n, n)))[0]
    lam = np.arange(1, n + 1, dtype=np.float64)[g.permutation(n)]
    return (Q * lam) @ Q.T


def _check_invariants(M, Ut, ev, r):
    M = np.asarray(M, np.float64)
    U = np.asarray(Ut, np.float64).T
    ref = np.sort(np.linalg.eigvalsh(M))[::-1][:r]
    lmax = max(abs(ref[0]), 1e-300)
    assert np.max(np.abs(ev - ref)) <= 1e-11 * lmax
    assert np.linalg.norm(M @ U - U * ev) <= 2e-6 * np.linalg.norm(M) * max(1.0, np.sqrt(r) / 8)
    assert np.linalg.norm(U.T @ U - np.eye(r)) <= 2e-6 * max(1.0, np.sqrt(r))


@pytest.mark.parametrize("n,r", [(1, 1), (2, 1), (2, 2), (3, 2), (33, 33), (33, 7), (64, 32),
                                 (65, 65), (100, 37), (257, 128), (300, 1)])
def test_separated_spectrum_matches_oracle(n, r):
    say("separated", n, r)
    M = _separated(n, seed=n + r)
    Ut, ev, _ = bm.shared_basis_gpu(torch.from_numpy(M).to(DEV), r)
    Ut = Ut.cpu().numpy()
    Uref, lref = oracle.shared_basis(M, r)
    assert np.max(np.abs(ev - lref)) <= 1e-11 * n
    assert np.max(np.abs(Ut - Uref)) <= 2e-6
    _check_invariants(M, Ut, ev, r)


@pytest.mark.parametrize("n,r", [(4133, 200)])
def test_large_separated_spectrum_matches_oracle(n, r):
    """A larger, ragged size (4133: no panel or tile boundary lines up with
    the end of the matrix) against numpy eigh, element by element."""
    say("separated, large", n, r)
    M = _separated(n, seed=11)
    Ut, ev, ms = bm.shared_basis_gpu(torch.from_numpy(M).to(DEV), r)
    say("gpu eigensolve ms", round(ms, 1))
    Ut = Ut.cpu().numpy()
    Uref, lref = oracle.shared_basis(M, r)
    assert np.max(np.abs(ev - lref)) <= 1e-11 * n
    assert np.max(np.abs(Ut - Uref)) <= 2e-6
    U = Ut.astype(np.float64).T
    assert np.linalg.norm(M @ U - U * ev) <= 2e-6 * np.linalg.norm(M) * max(1.0, np.sqrt(r) / 8)
    assert np.linalg.norm(U.T @ U - np.eye(r)) <= 2e-6 * max(1.0, np.sqrt(r))


def test_rank_deficient_and_repeated():
    """A rank-5 M of size 96 (the zero eigenvalue repeated 91 times) and a
    doubly repeated leading eigenvalue: invariants only."""
    g = np.random.default_rng(3)
    B = g.standard_normal((96, 5))
    M = B @ B.T
    Ut, ev, _ = bm.shared_basis_gpu(torch.from_numpy(M).to(DEV), 20)
    _check_invariants(M, Ut.cpu().numpy(), ev, 20)
    Q = np.linalg.qr(g.standard_normal((40, 40)))[0]
    lam = np.r_[9.0, 9.0, np.linspace(1, 5, 38)]
    M2 = (Q * lam) @ Q.T
    Ut2, ev2, _ = bm.shared_basis_gpu(torch.from_numpy(M2).to(DEV), 10)
    _check_invariants(M2, Ut2.cpu().numpy(), ev2, 10)


def _signal_projector_close(Ua, Ub, k):
    A = np.asarray(Ua, np.float64)[:k]
    B = np.asarray(Ub, np.float64)[:k]
    return np.linalg.norm(A.T @ A - B.T @ B) / np.sqrt(k)


@pytest.mark.parametrize("cfg,proj", [("qwen_gate", "gate"), ("qwen_layer", "down")])
def test_synthetic_cross_expert_gram(cfg, proj):
    """M = sum_e W_e W_e^T of the Qwen3-30B-A3B-shaped weights (768^2 for the
    gate, 2048^2 for the down projection; r = d_out / 2): against numpy eigh
    and the host LAPACK path on the same M."""
    c = synth.CONFIGS[cfg]
    p = c.proj(proj)
    say("cross-expert Gram", cfg, proj, p.d_out, p.r)
    W = synth.expert_weights(c, proj)
    Wd = torch.from_numpy(np.ascontiguousarray(W).view(np.int16)).view(torch.bfloat16).to(DEV)
    Md = bm.gram_experts(Wd)
    M = Md.cpu().numpy()
    Ut, ev, ms = bm.shared_basis_gpu(Md, p.r)
    say("gpu eigensolve ms", round(ms, 1))
    Ut = Ut.cpu().numpy()
    _check_invariants(M, Ut, ev, p.r)
    Uh, evh, msh = bm.shared_basis(Md, p.r)
    say("host eigensolve ms", round(msh, 1))
    assert np.max(np.abs(ev - evh)) <= 1e-11 * evh[0]
    Uref, _ = oracle.shared_basis(M, p.r)
    k0 = c.k0 if hasattr(c, "k0") else 128
    # the shared component's directions are separated from the noise bulk
    assert _signal_projector_close(Ut, Uref, k0) <= 1e-6
    assert _signal_projector_close(Ut, Uh.cpu().numpy(), k0) <= 1e-6


def test_non_finite_m_is_rejected():
    M = _separated(16, 0)
    M[3, 5] = M[5, 3] = np.nan
    with pytest.raises(bm.BitsmoeError):
        bm.shared_basis_gpu(torch.from_numpy(M).to(DEV), 4)
