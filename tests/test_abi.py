"""CPU tests of the C ABI: symbols, host-side solvers, argument checking.

No device work runs here: the device entry points are only called with
arguments that are rejected before anything is enqueued.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from oracle.ilp import Infeasible

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bitsmoe.h")

pkg = pytest.importorskip("paper_2606_00079_amd")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pkg.LIB_PATH):
        pytest.skip("libbitsmoe.so not built")
    return pkg.lib()


def _declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(bitsmoe_[a-z_0-9]+)\s*\(", txt)))


def test_header_declares_and_library_exports_everything(lib):
    names = _declared()
    assert "bitsmoe_score" in names and "bitsmoe_pack" in names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(pkg.EXPORTS)


def test_version(lib):
    assert "gfx950" in pkg.version()


# ------------------------------------------------------------------ allocate
def _rand_L(g, U, nb, ties=False):
    L = g.gamma(2.0, 1.0, size=(U, nb)) * np.logspace(0, -3, nb)[None, :] * g.uniform(0.1, 10, (U, 1))
    if ties:
        L = np.round(L * 8) / 8
        for _ in range(max(1, U // 10)):
            L[g.integers(0, U)] = L[g.integers(0, U)]
        L[g.integers(0, U)] = 0.0
    return L.astype(np.float32)


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("force_core", [False, True])
def test_allocate_matches_oracle_dp(lib, seed, force_core):
    g = np.random.default_rng(500 + seed)
    U = int(g.integers(1, 300))
    bits = [[1, 2, 3, 4], [1, 2, 3, 4, 8], [2, 3], [1]][seed % 4]
    L = _rand_L(g, U, len(bits), ties=seed % 2 == 1)
    for frac in (0.0, 0.3, 0.5, 0.77, 1.0):
        budget = int(U * bits[0] + frac * U * (bits[-1] - bits[0]))
        ref, _ = oracle.allocate_dp(L, bits, budget)
        got, obj, core = pkg.allocate(L, bits, budget, full_dp_limit=0 if force_core else -1,
                                      return_core=True)
        assert np.array_equal(got, ref), (U, bits, budget)
        assert np.isclose(obj, oracle.objective(L, bits, ref), rtol=1e-12)
        assert int(got.astype(np.int64).sum()) <= budget


def test_allocate_matches_exhaustive_tiny(lib):
    g = np.random.default_rng(9)
    for _ in range(30):
        U = int(g.integers(1, 7))
        bits = [1, 2, 3, 4]
        L = _rand_L(g, U, 4, ties=True)
        budget = int(g.integers(U, 4 * U + 1))
        ref, _ = oracle.allocate_exhaustive(L, bits, budget)
        for lim in (-1, 0):
            got, _ = pkg.allocate(L, bits, budget, full_dp_limit=lim)
            assert np.array_equal(got, ref)


def test_allocate_core_path_mid_size(lib):
    # Large enough that the default solver reduces to a core; checked against
    # the oracle's full dynamic program.
    g = np.random.default_rng(21)
    U = 6000
    bits = [1, 2, 3, 4]
    L = _rand_L(g, U, 4)
    budget = 2 * U
    ref, _ = oracle.allocate_dp(L, bits, budget)
    got, obj, core = pkg.allocate(L, bits, budget, full_dp_limit=0, return_core=True)
    assert np.array_equal(got, ref)
    assert core < U // 4


def _layer_like_L(g, E, r, bits):
    """Costs shaped like a loss table of E experts x r spectral units:
    energy decaying along each expert's spectrum, error falling about 4x per
    extra bit, log-normal spread; with forced ties (duplicated units, units
    equal to another expert's, all-zero units, units whose widths all cost
    the same) so that the lexicographic tie rule decides many of them."""
    k = np.arange(r)
    energy = (1.0 / (1.0 + k / 16.0))[None, :] * g.lognormal(0.0, 0.3, (E, r))
    per_bit = np.power(4.0, -np.asarray(bits, np.float64))[None, :]
    L = (energy.reshape(-1, 1) * per_bit * g.lognormal(0.0, 0.2, (E * r, len(bits))))
    U = E * r
    L = np.round(L * 2**14) / 2**14             # coarse values: many exact equalities
    dup = g.integers(0, U, size=(U // 20, 2))
    L[dup[:, 0]] = L[dup[:, 1]]
    L[g.integers(0, U, size=U // 100)] = 0.0
    flat = g.integers(0, U, size=U // 100)
    L[flat] = L[flat, :1]
    L[r:2 * r] = L[:r]                           # expert 1 repeats expert 0
    return L.astype(np.float32)


@pytest.mark.slow
@pytest.mark.parametrize("E,r", [(128, 384), (128, 1024)], ids=["qwen_gate_49152", "qwen_down_131072"])
def test_allocate_full_size_matches_oracle_dp(lib, E, r):
    """The ILP at the Qwen3-30B-A3B-shaped layer's sizes (bits 1-4, 2.0 bits
    per unit on average), as the benchmark runs it, against the oracle's
    exact dynamic program: the same widths, bit for bit."""
    g = np.random.default_rng(7000 + r)
    bits = [1, 2, 3, 4]
    L = _layer_like_L(g, E, r, bits)
    U = E * r
    budget = 2 * U
    got, obj = pkg.allocate(L, bits, budget)
    ref, _ = oracle.allocate_dp(L, bits, budget)
    assert np.array_equal(got, ref)
    assert int(got.astype(np.int64).sum()) <= budget
    assert np.isclose(obj, oracle.objective(L, bits, ref), rtol=1e-12)


def test_allocate_errors(lib):
    L = np.ones((4, 2), dtype=np.float32)
    with pytest.raises(pkg.BitsmoeError) as e:
        pkg.allocate(L, [1, 2], 3)
    assert e.value.code == "ERR_INFEASIBLE"
    with pytest.raises(Infeasible):
        oracle.allocate_dp(L, [1, 2], 3)
    L2 = L.copy()
    L2[1, 1] = np.nan
    with pytest.raises(pkg.BitsmoeError) as e:
        pkg.allocate(L2, [1, 2], 6)
    assert e.value.code == "ERR_NUMERIC"
    with pytest.raises(pkg.BitsmoeError) as e:
        pkg.allocate(L, [2, 1], 6)
    assert e.value.code == "ERR_ARG"
    with pytest.raises(pkg.BitsmoeError) as e:
        pkg.allocate(L, [1, 17], 6)
    assert e.value.code == "ERR_ARG"
    with pytest.raises(pkg.BitsmoeError) as e:
        pkg.allocate(L, [-1, 2], 6)
    assert e.value.code == "ERR_ARG"


@pytest.mark.parametrize("seed,force_core", [(0, False), (1, True), (2, True)])
def test_allocate_surrogate_widths_match_oracle(lib, seed, force_core):
    """Widths 0 (eviction) .. 16 (fp16), as the surrogate mode uses them."""
    from oracle import surrogate as sg
    g = np.random.default_rng(50 + seed)
    U = 300
    C = (g.standard_normal((U, 64)) * np.exp(g.standard_normal((U, 1)))).astype(np.float32)
    H = oracle.gram(g.standard_normal((256, 64)))
    L = sg.surrogate_table(C.astype(np.float64), H, gamma=0.7).astype(np.float32)
    for budget in (0, 150, 2 * U, 5 * U):
        ref, _ = oracle.allocate_dp(L, sg.WIDTHS, budget)
        got, _ = pkg.allocate(L, sg.WIDTHS, budget, full_dp_limit=0 if force_core else -1)
        assert np.array_equal(got, ref), budget
        assert int(got.astype(np.int64).sum()) <= budget


def test_surrogate_budget_matches_oracle(lib):
    from oracle import surrogate as sg
    g = np.random.default_rng(8)
    for _ in range(50):
        E = int(g.integers(1, 300))
        n_out = int(g.integers(8, 8192))
        m = int(g.integers(8, 16384))
        r = int(g.integers(1, n_out + 1))
        b_eq = float(g.choice([1.5, 2.0, 2.5, 3.0, 4.0]))
        ref = sg.budget_equivalent(E, n_out, m, b_eq, r)
        if ref < 0:
            with pytest.raises(pkg.BitsmoeError) as e:
                pkg.surrogate_budget(E, n_out, m, r, b_eq)
            assert e.value.code == "ERR_INFEASIBLE"
        else:
            assert pkg.surrogate_budget(E, n_out, m, r, b_eq) == ref
    assert pkg.surrogate_budget(128, 2048, 768, 2048, 2.0) == 436906
    with pytest.raises(pkg.BitsmoeError):
        pkg.surrogate_budget(4, 64, 64, 65, 2.0)


def test_pack_layout_matches_oracle(lib):
    g = np.random.default_rng(3)
    bits_u = g.choice([1, 2, 3, 4, 8], size=77).astype(np.uint8)
    for d in (64, 256, 2048):
        assert np.array_equal(pkg.pack_layout(bits_u, d), oracle.pack_layout(bits_u, d))
    with pytest.raises(pkg.BitsmoeError) as e:
        pkg.pack_layout(bits_u, 100)
    assert e.value.code == "ERR_SHAPE"
    bad = bits_u.copy()
    bad[5] = 9
    with pytest.raises(pkg.BitsmoeError):
        pkg.pack_layout(bad, 64)
    surr = g.choice([0, 1, 2, 3, 4, 6, 8, 16], size=77).astype(np.uint8)
    assert np.array_equal(pkg.pack_layout(surr, 128), oracle.pack_layout(surr, 128))


# ------------------------------------------------- device calls, rejected early
def test_device_entry_points_validate_before_launch(lib):
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: every call below is rejected first
    null = ctypes.c_void_p(0)
    s = ctypes.c_void_p(0)
    bits = (ctypes.c_int * 4)(1, 2, 3, 4)
    bad_bits = (ctypes.c_int * 2)(3, 2)
    assert lib.bitsmoe_gram(null, 1, 10, 64, fake, s) == 1
    assert lib.bitsmoe_gram(fake, 1, 10, 100, fake, s) == 2
    assert lib.bitsmoe_gram(fake, 7, 10, 64, fake, s) == 3
    assert lib.bitsmoe_gram(fake, 1, 0, 64, fake, s) == 1
    assert lib.bitsmoe_gram_experts(fake, 1, 2, 96, 64, fake, s) == 2
    assert lib.bitsmoe_gram_experts(fake, 1, 0, 64, 64, fake, s) == 1
    assert lib.bitsmoe_project(fake, fake, 1, 2, 64, 64, 65, fake, s) == 2
    assert lib.bitsmoe_project(fake, fake, 1, 2, 64, 100, 8, fake, s) == 2
    assert lib.bitsmoe_score(fake, 10, 256, fake, bits, 4, 48, fake, s) == 2
    assert lib.bitsmoe_score(fake, 10, 320, fake, bits, 4, 128, fake, s) == 2
    assert lib.bitsmoe_score(fake, 10, 256, fake, bad_bits, 2, 64, fake, s) == 1
    assert lib.bitsmoe_score(fake, 10, 256, fake, bits, 0, 64, fake, s) == 1
    assert lib.bitsmoe_score(fake, 0, 256, fake, bits, 4, 64, fake, s) == 1
    assert lib.bitsmoe_pack(fake, 10, 256, 48, fake, fake, 10, fake, fake, s) == 2
    assert lib.bitsmoe_pack(null, 10, 256, 64, fake, fake, 10, fake, fake, s) == 1
    assert lib.bitsmoe_unpack(fake, fake, fake, fake, 10, 10, 200, 64, fake, s) == 2
    assert lib.bitsmoe_shared_basis(fake, 64, 65, fake, null, null, s) == 2
    assert "r > d_out" in pkg.last_error()
    assert lib.bitsmoe_shared_basis(null, 64, 4, fake, null, null, s) == 1
    assert lib.bitsmoe_shared_basis_gpu(fake, 64, 65, fake, null, null, s) == 2
    assert lib.bitsmoe_shared_basis_gpu(fake, 70000, 4, fake, null, null, s) == 2
    assert lib.bitsmoe_shared_basis_gpu(null, 64, 4, fake, null, null, s) == 1
    assert lib.bitsmoe_shared_basis_gpu(fake, 64, 0, fake, null, null, s) == 1
    assert lib.bitsmoe_set_lapack(b"/nonexistent/liblapack.so") == 8
    kap = (ctypes.c_double * 3)(0.149492, 0.0406789, 0.01184786)
    badk = (ctypes.c_double * 3)(0.149492, -1.0, 0.01184786)
    assert lib.bitsmoe_surrogate(null, 10, 256, fake, 0.7, kap, fake, null, s) == 1
    assert lib.bitsmoe_surrogate(fake, 10, 200, fake, 0.7, kap, fake, null, s) == 2
    assert lib.bitsmoe_surrogate(fake, 0, 256, fake, 0.7, kap, fake, null, s) == 1
    assert lib.bitsmoe_surrogate(fake, 10, 256, fake, 1.5, kap, fake, null, s) == 1
    assert lib.bitsmoe_surrogate(fake, 10, 256, fake, 0.7, badk, fake, null, s) == 1
    assert lib.bitsmoe_gram_experts_in(fake, 1, 2, 96, 64, fake, s) == 2
    assert lib.bitsmoe_gram_experts_in(null, 1, 2, 64, 64, fake, s) == 1
    assert lib.bitsmoe_gram_experts_in(fake, 5, 2, 64, 64, fake, s) == 3
    assert lib.bitsmoe_project_in(fake, fake, 1, 2, 64, 64, 65, fake, s) == 2
    assert lib.bitsmoe_project_in(fake, fake, 1, 2, 100, 64, 8, fake, s) == 2
    assert lib.bitsmoe_basis_importance(fake, 8, 100, fake, fake, s) == 2
    assert lib.bitsmoe_basis_importance(null, 8, 64, fake, fake, s) == 1
    assert lib.bitsmoe_score_diag(fake, 10, 256, fake, 0, bits, 4, 64, fake, s) == 1
    assert lib.bitsmoe_score_diag(fake, 10, 256, fake, 4, bits, 4, 48, fake, s) == 2
    assert lib.bitsmoe_score_diag(fake, 10, 256, fake, 4, bad_bits, 2, 64, fake, s) == 1
    off = (ctypes.c_int64 * 3)(0, 2, 3)
    badoff = (ctypes.c_int64 * 3)(0, 2, 1)
    rows = (ctypes.c_int32 * 3)(0, 5, 9)
    badrows = (ctypes.c_int32 * 3)(0, 5, 10)
    wts = (ctypes.c_float * 3)(0.5, 0.5, 1.0)
    badw = (ctypes.c_float * 3)(0.5, -0.5, 1.0)
    assert lib.bitsmoe_gram_routed(fake, 1, 10, 64, 2, badoff, rows, wts, fake, s) == 1
    assert lib.bitsmoe_gram_routed(fake, 1, 10, 64, 2, off, badrows, wts, fake, s) == 1
    assert lib.bitsmoe_gram_routed(fake, 1, 10, 64, 2, off, rows, badw, fake, s) == 1
    assert lib.bitsmoe_gram_routed(fake, 1, 10, 100, 2, off, rows, wts, fake, s) == 2
    assert lib.bitsmoe_score_routed(fake, 10, 256, fake, 3, bits, 4, 64, fake, s) == 2
    assert lib.bitsmoe_score_routed(fake, 128, 256, fake, 32, bits, 4, 64, fake, s) == 2
    assert lib.bitsmoe_score_routed(fake, 128, 256, fake, 0, bits, 4, 64, fake, s) == 2
    dtok = (ctypes.c_int32 * 3)(0, 1, 1)
    dbad = (ctypes.c_int32 * 3)(0, 1, 2)
    dw = (ctypes.c_float * 3)(0.5, 0.5, 1.0)
    assert lib.bitsmoe_moe_decode(fake, fake, fake, fake, 10, 2, 8, 100, 64, fake, 64, fake, 2,
                                  off, dtok, dw, fake, s) == 2
    assert lib.bitsmoe_moe_decode(fake, fake, fake, fake, 10, 2, 8, 128, 48, fake, 64, fake, 2,
                                  off, dtok, dw, fake, s) == 2
    assert lib.bitsmoe_moe_decode(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, fake, 2,
                                  off, dbad, dw, fake, s) == 1
    assert lib.bitsmoe_moe_decode(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, fake, 2,
                                  badoff, dtok, dw, fake, s) == 1
    assert lib.bitsmoe_moe_decode(null, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, fake, 2,
                                  off, dtok, dw, fake, s) == 1
    # misaligned device pointers are refused before any launch
    odd = ctypes.c_void_p(0x1008)
    assert lib.bitsmoe_moe_decode(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, odd, 2,
                                  off, dtok, dw, fake, s) == 1
    assert lib.bitsmoe_moe_decode_topk(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, fake,
                                       2, 2, odd, fake, fake, s) == 1
    # input-space decode: the units' length (d_out) follows the pack rules
    assert lib.bitsmoe_moe_decode_in(fake, fake, fake, fake, 10, 2, 8, 100, 64, fake, 64, fake, 2,
                                     off, dtok, dw, fake, s) == 2
    assert lib.bitsmoe_moe_decode_in(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, fake, 2,
                                     off, dbad, dw, fake, s) == 1
    assert lib.bitsmoe_moe_decode_in(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 0, fake, 2,
                                     off, dtok, dw, fake, s) == 1
    assert lib.bitsmoe_moe_decode_in(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, odd, 2,
                                     off, dtok, dw, fake, s) == 1
    # top-k decode: k outside [1, E], B k above 65535, shape rules, nulls
    assert lib.bitsmoe_moe_decode_topk(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, fake,
                                       2, 0, fake, fake, fake, s) == 1
    assert lib.bitsmoe_moe_decode_topk(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, fake,
                                       2, 3, fake, fake, fake, s) == 2
    assert lib.bitsmoe_moe_decode_topk(fake, fake, fake, fake, 10, 8, 8, 128, 64, fake, 64, fake,
                                       10000, 8, fake, fake, fake, s) == 2
    assert lib.bitsmoe_moe_decode_topk(fake, fake, fake, fake, 10, 2, 8, 100, 64, fake, 64, fake,
                                       2, 2, fake, fake, fake, s) == 2
    assert lib.bitsmoe_moe_decode_topk(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64, fake,
                                       2, 2, null, fake, fake, s) == 1
    # the allocation-free top-k decode: the same checks, plus its buffer limit
    assert lib.bitsmoe_moe_decode_topk_noalloc(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64,
                                               fake, 2, 0, fake, fake, fake, s) == 1
    assert lib.bitsmoe_moe_decode_topk_noalloc(fake, fake, fake, fake, 10, 2, 8, 128, 64, fake, 64,
                                               fake, 2, 2, odd, fake, fake, s) == 1
    assert lib.bitsmoe_moe_decode_topk_noalloc(fake, fake, fake, fake, 10, 8, 8192, 128, 64, fake,
                                               64, fake, 520, 1, fake, fake, fake, s) == 2
    assert "fixed scratch" in pkg.last_error()
    assert lib.bitsmoe_gram(odd, 1, 64, 64, fake, s) == 1
    assert "aligned" in pkg.last_error()
    assert lib.bitsmoe_gram_experts(fake, 1, 2, 64, 64, odd, s) == 1
    assert lib.bitsmoe_project(fake, odd, 1, 2, 64, 64, 8, fake, s) == 1
    assert lib.bitsmoe_score(fake, 10, 256, fake, bits, 4, 64, odd, s) == 1
    assert lib.bitsmoe_pack(fake, 10, 256, 64, fake, odd, 10, fake, fake, s) == 1
    assert lib.bitsmoe_unpack(fake, fake, fake, fake, 10, 10, 256, 64, odd, s) == 1
    assert lib.bitsmoe_shared_basis(odd, 64, 4, fake, null, null, s) == 1
    assert lib.bitsmoe_shared_basis_gpu(odd, 64, 4, fake, null, null, s) == 1
    assert lib.bitsmoe_surrogate(fake, 10, 256, fake, 0.7, kap, odd, null, s) == 1
    assert lib.bitsmoe_surrogate(fake, 10, 256, fake, 0.7, kap, fake, odd, s) == 1
