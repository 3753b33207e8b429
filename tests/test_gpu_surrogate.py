"""GPU parity of the surrogate cost table (bitsmoe_surrogate) against the
fp64 oracle (oracle.surrogate), through the C ABI.

Stage-wise: the oracle is fed the same fp32 rows C and the same H as the
device.  Bar: every entry of the table within 1e-3 relative (beta enters
through the fp16 matrix-core form of the loss table), the row statistics
alpha^2, rho and cos theta within 1e-5, and the ILP over the surrogate's
widths bit-exact against the oracle's dynamic program on the same table.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import surrogate as sg

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)
import paper_2606_00079_amd as bm  # noqa: E402

REL = 1e-3
KAPPA = [sg.KAPPA_PRINTED[b] for b in (2, 3, 4)]


def say(*a):
    print("[surrogate]", *a, flush=True)


def _inputs(units, d, seed, heavy):
    C = synth.random_rows(units, d, seed=seed, scale=0.05, heavy=heavy)
    C[0] = 0.0                      # evicted-only row: costs 0
    C[1] = 0.125                    # constant row: rho = cos = 1/sqrt(d)
    C[2, :] = 0.0
    C[2, 7] = -3.0                  # one-hot row: rho = cos * sqrt(d) = 1
    X = synth.random_rows(2 * d, d, seed=seed + 1, scale=1.0, heavy=heavy)
    X[:, ::13] *= 8.0
    H = oracle.gram(X.astype(np.float64)).astype(np.float32)
    return C, H


def _rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-30)))


@pytest.mark.parametrize("units,d,gamma,heavy", [
    (257, 256, 0.7, False),
    (130, 704, 0.5, True),      # three row tiles, partial last K block
    (4096, 2048, 0.7, False),   # Qwen3-30B-A3B gate row length
    (515, 768, 1.0, True),
    (64, 128, 0.0, False),
])
def test_surrogate_matches_oracle(units, d, gamma, heavy):
    say("case", units, d, gamma, heavy)
    C, H = _inputs(units, d, seed=units + d, heavy=heavy)
    Cd, Hd = torch.from_numpy(C).cuda(), torch.from_numpy(H).cuda()
    stats = torch.empty((units, 4), dtype=torch.float32, device="cuda")
    L = bm.surrogate(Cd, Hd, gamma, KAPPA, stats=stats).cpu().numpy()
    st = stats.cpu().numpy()
    ref = sg.surrogate_table(C.astype(np.float64), H.astype(np.float64), gamma)
    a2, rho, cos = sg.unit_stats(C.astype(np.float64))
    beta = sg.beta(C.astype(np.float64), H.astype(np.float64))
    say("max rel L", _rel(L, ref), "beta", _rel(st[3:, 1], beta[3:]))
    assert np.all(np.isfinite(L)) and np.all(L >= 0)
    assert np.all(L[0] == 0.0)
    assert _rel(L, ref) <= REL
    assert _rel(st[:, 0], a2) <= 1e-5
    assert _rel(st[3:, 1], beta[3:]) <= REL
    assert _rel(st[:, 2], rho) <= 1e-5
    assert _rel(st[:, 3], cos) <= 1e-5


def test_surrogate_eviction_column_is_the_loss_table_at_delta_c():
    """With gamma = 1 the eviction column is c H c^T: the quadratic form the
    loss table evaluates for delta = c (App. B.2, exact under eviction)."""
    C, H = _inputs(300, 512, seed=5, heavy=False)
    L = bm.surrogate(torch.from_numpy(C).cuda(), torch.from_numpy(H).cuda(), 1.0, KAPPA).cpu().numpy()
    q = np.sum((C.astype(np.float64) @ H.astype(np.float64)) * C, axis=1)
    assert _rel(L[3:, 0], q[3:]) <= REL


def test_surrogate_allocation_matches_oracle():
    """ILP over widths {0..16} on the device table vs the oracle DP on it, with
    the paper's equivalent-bit budget."""
    E, n_out, d, r = 8, 256, 512, 128
    C, H = _inputs(E * r, d, seed=11, heavy=True)
    L = bm.surrogate(torch.from_numpy(C).cuda(), torch.from_numpy(H).cuda(), 0.7, KAPPA).cpu().numpy()
    B = bm.surrogate_budget(E, n_out, d, r, 2.0)
    assert B == sg.budget_equivalent(E, n_out, d, 2.0, r)
    got, obj = bm.allocate(L, sg.WIDTHS, B)
    ref, _ = oracle.allocate_dp(L, sg.WIDTHS, B)
    assert np.array_equal(got, ref)
    assert int(got.astype(np.int64).sum()) <= B
    assert got[0] == 0  # the zero row is evicted: it costs nothing at any width


def test_surrogate_full_size_qwen_down_sampled():
    """The launch shape of the Qwen3-30B-A3B down projection (131072 units of
    length 768): sampled rows against the oracle."""
    from synth import device as sdev
    units, d = 131072, 768
    g = torch.Generator(device="cuda").manual_seed(7)
    C = torch.randn(units, d, device="cuda", generator=g) * 0.05
    C[5] = 0.0
    X = torch.randn(4096, d, device="cuda", generator=g)
    H = (X.T @ X) / 4096
    L = bm.surrogate(C, H, 0.7, KAPPA).cpu().numpy()
    rows = np.r_[0, 5, units - 1, np.random.default_rng(1).choice(units, 256, replace=False)]
    Cs = C[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    ref = sg.surrogate_table(Cs, H.cpu().numpy().astype(np.float64), 0.7)
    assert _rel(L[rows], ref) <= REL
    assert np.all(L[5] == 0.0)
    del sdev
