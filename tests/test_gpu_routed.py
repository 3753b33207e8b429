"""GPU parity of the routed per-expert calibration Grams and the loss table
against them (bitsmoe_gram_routed, bitsmoe_score_routed) vs oracle.routed.

Bars: every H_e within 1e-3 relative Frobenius; L within 1e-3 relative per
entry (1e-4 measured for the shared-H table).
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from conftest import gpu_available
from oracle import routed

pytestmark = pytest.mark.gpu

if not gpu_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2606_00079_amd as bm  # noqa: E402

DEV = "cuda:0"
REL = 1e-3


def say(*a):
    print("[gpu-routed]", *a, flush=True)
    sys.stdout.flush()


def dev(a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def relfro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.mark.parametrize("config", ["tiny", "qwen_gate"])
def test_gram_routed(config):
    say("gram_routed", config)
    cfg = synth.CONFIGS[config]
    X = synth.calibration_input(cfg, cfg.projs[0].name)
    off, tok, w = synth.routing(cfg, X)
    Hs = bm.gram_routed(dev(X, cfg.dtype), off, tok, w).cpu().numpy()
    X64 = synth.as_f64(X, cfg.dtype)
    experts = range(cfg.E) if cfg.E <= 8 else [0, 1, 17, 63, 127]
    ref = routed.gram_routed(X64, off, tok, w)
    for e in experts:
        err = relfro(Hs[e], ref[e])
        assert err <= REL, (e, err)
        assert np.array_equal(Hs[e], Hs[e].T)
    # every token's weights sum to 1: the experts' Grams add up to the shared one
    Hsum = Hs.astype(np.float64).sum(axis=0)
    assert relfro(Hsum, oracle.gram(X64)) <= REL
    say("max rel fro", max(relfro(Hs[e], ref[e]) for e in experts))


def test_gram_routed_empty_expert_and_ragged_rows():
    g = np.random.default_rng(3)
    X = synth.random_rows(150, 192, seed=3, scale=1.0, heavy=True)
    off = np.array([0, 40, 40, 107, 150], dtype=np.int64)
    tok = np.concatenate([np.sort(g.choice(150, 40, replace=False)), np.sort(g.choice(150, 67, replace=False)),
                          np.sort(g.choice(150, 43, replace=False))]).astype(np.int32)
    w = g.random(150).astype(np.float32)
    Hs = bm.gram_routed(dev(X, "f32"), off, tok, w).cpu().numpy()
    ref = routed.gram_routed(X.astype(np.float64), off, tok, w)
    assert np.all(Hs[1] == 0.0)
    for e in (0, 2, 3):
        assert relfro(Hs[e], ref[e]) <= REL


@pytest.mark.parametrize("E,upe,d,bits,group", [
    (4, 64, 256, (1, 2, 3, 4), 64),     # tiny shape: one 256-row tile per expert
    (3, 128, 768, (1, 2, 3, 4), 128),   # two tiles per expert, three row tiles of H
    (2, 256, 320, (1, 2, 4, 8), 64),    # ragged K block
])
def test_score_routed(E, upe, d, bits, group):
    say("score_routed", E, upe, d, bits, group)
    g = np.random.default_rng(E + upe + d)
    C = synth.random_rows(E * upe, d, seed=d, scale=0.05, heavy=True)
    C[0] = 0.0
    X = synth.random_rows(4 * d, d, seed=d + 1, scale=1.0, heavy=True)
    Hs = np.stack([oracle.gram(X[g.choice(4 * d, 2 * d, replace=False)].astype(np.float64)) *
                   (1.0 + e) for e in range(E)]).astype(np.float32)
    L = bm.score_routed(dev(C, "f32"), dev(Hs, "f32"), upe, bits, group).cpu().numpy()
    ref = routed.score_routed(C, Hs.astype(np.float64), upe, bits, group)
    assert np.all(L[0] == 0.0)
    err = float(np.max(np.abs(L[1:] - ref[1:]) / np.maximum(np.abs(ref[1:]), 1e-30)))
    say("max rel", err)
    assert err <= REL
    # the shared-H entry point agrees with the routed one when all H_e are equal
    Lsh = bm.score(dev(C, "f32"), dev(Hs[0], "f32"), bits, group).cpu().numpy()
    Lr = bm.score_routed(dev(C, "f32"), dev(np.stack([Hs[0]] * E), "f32"), upe, bits, group).cpu().numpy()
    assert np.array_equal(Lsh, Lr)


def test_routed_qwen_gate_full_size_sampled():
    """The Qwen3-30B-A3B gate shape: 128 routed Grams of 2048^2, the loss table
    of 49152 units against them, sampled rows checked."""
    cfg = synth.CONFIGS["qwen_gate"]
    X = synth.calibration_input(cfg, "gate")
    off, tok, w = synth.routing(cfg, X)
    Hs = bm.gram_routed(dev(X, cfg.dtype), off, tok, w)
    units, d, upe = 128 * 384, 2048, 384
    gen = torch.Generator(device="cuda").manual_seed(5)
    C = torch.randn(units, d, device="cuda", generator=gen) * 0.05
    L = bm.score_routed(C, Hs, upe, cfg.bits, cfg.group).cpu().numpy()
    rows = np.sort(np.random.default_rng(2).choice(units, 96, replace=False))
    Cs = C[torch.from_numpy(rows).cuda()].cpu().numpy()
    H64 = Hs.cpu().numpy().astype(np.float64)
    for i, u in enumerate(rows):
        ref = oracle.score_rows(Cs[i:i + 1], H64[u // upe], cfg.bits, cfg.group)[0]
        err = float(np.max(np.abs(L[u] - ref) / np.abs(ref)))
        assert err <= REL, (u, err)
