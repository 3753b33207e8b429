"""GPU parity of stage-3 decode (bitsmoe_moe_decode) against oracle.decode.

The packed units are made by the oracle's own pack from seeded rows (no
input comes from the device path), uploaded, and decoded on the device.
Bar: y within 1e-4 relative Frobenius of the fp64 oracle (fp32 sums over
d_in and r terms).
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from conftest import gpu_available
from oracle import decode

pytestmark = pytest.mark.gpu

if not gpu_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

import torch  # noqa: E402

import paper_2606_00079_amd as bm  # noqa: E402

DEV = "cuda:0"
REL = 1e-4


def say(*a):
    print("[gpu-decode]", *a, flush=True)
    sys.stdout.flush()


def relfro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def _case(E, r, d_in, d_out, B, k, G, widths, seed):
    g = np.random.default_rng(seed)
    C = (g.standard_normal((E * r, d_in)) * np.exp(g.standard_normal((E * r, 1)))).astype(np.float32)
    bits_u = g.choice(widths, size=E * r).astype(np.uint8)
    codes, params, off = oracle.pack(C, bits_u, G)
    Ut = np.ascontiguousarray(np.linalg.qr(g.standard_normal((d_out, r)))[0].T, dtype=np.float32)
    X = g.standard_normal((B, d_in)).astype(np.float32)
    # top-k routing of B tokens over E experts, grouped by expert
    logits = g.standard_normal((B, E))
    top = np.argsort(-logits, axis=1)[:, :k]
    wts = np.exp(np.take_along_axis(logits, top, 1))
    wts = (wts / wts.sum(1, keepdims=True)).astype(np.float32)
    tok = np.repeat(np.arange(B, dtype=np.int32), k)
    ex = top.reshape(-1)
    order = np.lexsort((tok, ex))
    offs = np.r_[0, np.cumsum(np.bincount(ex, minlength=E))].astype(np.int64)
    return C, bits_u, codes, params, off, Ut, X, (offs, tok[order], wts.reshape(-1)[order])


def assert_close(Y, ref, rel=REL):
    """Relative Frobenius within `rel`, and element by element within rel of
    the entry plus rel / 10 of the largest entry (entries near zero come
    from cancelling sums)."""
    Y = np.asarray(Y, np.float64)
    ref = np.asarray(ref, np.float64)
    assert relfro(Y, ref) <= rel
    bound = rel * np.abs(ref) + 0.1 * rel * np.max(np.abs(ref))
    bad = np.abs(Y - ref) > bound
    assert not bad.any(), (int(bad.sum()), float(np.max(np.abs(Y - ref) - bound)))


def _run(E, r, d_in, d_out, B, k, G, widths, seed, drop_token=None):
    C, bits_u, codes, params, off, Ut, X, (offs, tok, w) = _case(E, r, d_in, d_out, B, k, G, widths, seed)
    if drop_token is not None:
        keep = tok != drop_token
        offs = np.r_[0, np.cumsum([np.sum(keep[offs[e]:offs[e + 1]]) for e in range(E)])].astype(np.int64)
        tok, w = tok[keep], w[keep]
    cd = torch.from_numpy(codes.view(np.int64).copy() if len(codes) else np.zeros(1, np.int64)).to(DEV)
    pd = torch.from_numpy(params.view(np.int16).copy()).to(DEV)
    bd = torch.from_numpy(bits_u).to(DEV)
    od = torch.from_numpy(off).to(DEV)
    Y = bm.moe_decode(cd, pd, bd, od, int(off[-1]), E, r, d_in, G, torch.from_numpy(Ut).to(DEV),
                      torch.from_numpy(X).to(DEV), (offs, tok, w)).cpu().numpy()
    Chat = decode.dequantized_factors(codes, params, bits_u, d_in, G)
    ref = decode.moe_decode(Chat, r, Ut, X, offs, tok, w)
    return Y, ref


@pytest.mark.parametrize("E,r,d_in,d_out,B,k,G,widths", [
    (4, 64, 256, 128, 24, 2, 64, (1, 2, 3, 4)),
    (6, 40, 192, 96, 17, 3, 32, (0, 1, 2, 4, 8, 16)),   # eviction and fp16 rows
    (3, 8, 768, 64, 1, 1, 128, (2, 3)),                 # one token, one expert
    (8, 33, 512, 256, 40, 8, 256, (1, 2, 3, 4, 6, 8)),  # every token on every expert
    (5, 24, 2560, 128, 1, 2, 64, (0, 1, 2, 16)),        # rows in two slices, one token
    (4, 20, 4096, 64, 9, 2, 128, (2, 3, 4, 16)),        # rows in two slices, chunks of four
    (2, 70, 64, 96, 5, 1, 32, (1, 3, 5, 7)),            # 32 rows per wave pass
])
def test_moe_decode_matches_oracle(E, r, d_in, d_out, B, k, G, widths):
    say("decode", E, r, d_in, d_out, B, k, G, widths)
    Y, ref = _run(E, r, d_in, d_out, B, k, G, widths, seed=E + r + B)
    err = relfro(Y, ref)
    say("rel fro", err)
    assert_close(Y, ref)


def test_moe_decode_unrouted_token_is_zero():
    Y, ref = _run(4, 32, 256, 64, 10, 2, 64, (2, 4), seed=3, drop_token=4)
    assert np.all(Y[4] == 0.0)
    assert relfro(Y, ref) <= REL


def test_moe_decode_qwen_gate_rows():
    """The Qwen3-30B-A3B gate projection's unit shape (r = 384 units of length
    2048 per expert, d_out = 768, group 128) on 16 experts, 64 tokens, top-2."""
    Y, ref = _run(16, 384, 2048, 768, 64, 2, 128, (1, 2, 3, 4), seed=11)
    err = relfro(Y, ref)
    say("qwen rows rel fro", err)
    assert err <= REL


def _topk_run(E, r, d_in, d_out, B, k, G, widths, seed, bad=()):
    """Decode from a device top-k table; `bad` = (token, slot, expert) entries
    with an expert outside [0, E), which must contribute nothing."""
    C, bits_u, codes, params, off, Ut, X, _ = _case(E, r, d_in, d_out, B, k, G, widths, seed)
    g = np.random.default_rng(seed + 1)
    logits = g.standard_normal((B, E))
    top = np.argsort(-logits, axis=1)[:, :k].astype(np.int32)
    w = np.exp(np.take_along_axis(logits, top, 1))
    w = (w / w.sum(1, keepdims=True)).astype(np.float32)
    for b, j, e in bad:
        top[b, j] = e
    ok = (top >= 0) & (top < E)
    ex, tok, wt = top[ok], np.nonzero(ok)[0].astype(np.int32), w[ok]
    order = np.lexsort((tok, ex))
    offs = np.r_[0, np.cumsum(np.bincount(ex, minlength=E))].astype(np.int64)
    routing = (offs, tok[order], wt[order])
    cd = torch.from_numpy(codes.view(np.int64).copy() if len(codes) else np.zeros(1, np.int64)).to(DEV)
    pd = torch.from_numpy(params.view(np.int16).copy()).to(DEV)
    bd = torch.from_numpy(bits_u).to(DEV)
    od = torch.from_numpy(off).to(DEV)
    Utd, Xd = torch.from_numpy(Ut).to(DEV), torch.from_numpy(X).to(DEV)
    Y = bm.moe_decode_topk(cd, pd, bd, od, int(off[-1]), E, r, d_in, G, Utd, Xd,
                           torch.from_numpy(top).to(DEV), torch.from_numpy(w).to(DEV)).cpu().numpy()
    Yg = bm.moe_decode(cd, pd, bd, od, int(off[-1]), E, r, d_in, G, Utd, Xd, routing).cpu().numpy()
    Chat = decode.dequantized_factors(codes, params, bits_u, d_in, G)
    ref = decode.moe_decode(Chat, r, Ut, X, *routing)
    return Y, Yg, ref


@pytest.mark.parametrize("E,r,d_in,d_out,B,k,G,widths", [
    (16, 384, 2048, 768, 1, 8, 128, (1, 2, 3, 4)),      # Qwen3-30B-A3B gate rows, one token
    (16, 256, 768, 512, 3, 8, 128, (0, 1, 2, 3, 16)),   # down-projection row length
    (6, 40, 2560, 96, 5, 2, 64, (1, 2, 4)),              # rows in two slices
])
def test_moe_decode_topk_matches_oracle(E, r, d_in, d_out, B, k, G, widths):
    say("decode topk", E, r, d_in, d_out, B, k, G, widths)
    Y, Yg, ref = _topk_run(E, r, d_in, d_out, B, k, G, widths, seed=E + B)
    assert relfro(Y, ref) <= REL
    assert relfro(Y, Yg) <= 1e-5


def test_moe_decode_topk_skips_experts_out_of_range():
    Y, Yg, ref = _topk_run(8, 32, 256, 64, 4, 3, 64, (2, 3), seed=5,
                           bad=((0, 1, -1), (2, 0, 8), (3, 2, 1 << 30)))
    assert relfro(Y, ref) <= REL
    assert relfro(Y, Yg) <= 1e-5


# Batches of 16 tokens or more take the matrix-core z step, the top-k form
# with its routing grouped by expert on the device.  Jobs hold up to 8
# routing entries of an expert while the experts average at most 8, else 16:
# the first cases below have 16 per job, the 8-entry cases follow.
@pytest.mark.parametrize("E,r,d_in,d_out,B,k,G,widths", [
    (16, 384, 2048, 768, 64, 8, 128, (1, 2, 3, 4)),     # Qwen3-30B-A3B gate units, 64 tokens, top-8
    (16, 1024, 768, 2048, 64, 8, 128, (1, 2, 3, 4)),    # down units
    # 8-entry jobs: the benchmarked routing (128 experts, 64 tokens, top-8)
    # and row lengths (gate 2048, down 768), fewer rows per expert
    (128, 32, 2048, 256, 64, 8, 128, (1, 2, 3, 4)),
    (128, 80, 768, 512, 64, 8, 128, (1, 2, 3, 4)),
    (64, 96, 768, 128, 32, 6, 64, (1, 2, 3, 4, 5)),     # group 64, a 5-bit row past the prefetched planes
    (48, 64, 512, 64, 24, 4, 256, (2, 3, 16)),          # group 256, fp16 rows
    (40, 48, 256, 96, 20, 3, 32, (0, 1, 4, 8)),         # group 32, eviction, 8-bit rows
    (12, 40, 256, 96, 33, 5, 32, (0, 1, 2, 4, 8, 16)),  # ragged row blocks, eviction, fp16 rows
    (5, 17, 512, 64, 16, 5, 256, (3, 5, 7, 8)),         # every token on every expert, group 256
    (3, 64, 64, 64, 40, 2, 64, (1, 2)),                 # one group per row, many tokens per expert
])
def test_moe_decode_topk_batch_matches_oracle(E, r, d_in, d_out, B, k, G, widths):
    say("decode topk batch", E, r, d_in, d_out, B, k, G, widths)
    Y, Yg, ref = _topk_run(E, r, d_in, d_out, B, k, G, widths, seed=E + B + 7)
    say("rel fro", relfro(Y, ref))
    assert_close(Y, ref)
    assert_close(Yg, ref)
    assert relfro(Y, Yg) <= 1e-5


def test_moe_decode_topk_batch_out_of_range_and_deterministic():
    bad = ((0, 1, -1), (5, 0, 8), (17, 2, 1 << 30), (17, 1, 9))
    Y, Yg, ref = _topk_run(8, 48, 256, 64, 20, 3, 64, (2, 3, 16), seed=9, bad=bad)
    assert_close(Y, ref)
    Y2, _, _ = _topk_run(8, 48, 256, 64, 20, 3, 64, (2, 3, 16), seed=9, bad=bad)
    assert np.array_equal(Y, Y2)


# ---- input-space form (gate/up): y = sum_j g_j C^_e^T (Vt x) ----

def _run_in(E, r, d_out, d_in, B, k, G, widths, seed):
    g = np.random.default_rng(seed)
    C = (g.standard_normal((E * r, d_out)) * np.exp(g.standard_normal((E * r, 1)))).astype(np.float32)
    bits_u = g.choice(widths, size=E * r).astype(np.uint8)
    codes, params, off = oracle.pack(C, bits_u, G)
    Vt = np.ascontiguousarray(np.linalg.qr(g.standard_normal((d_in, r)))[0].T, dtype=np.float32)
    X = g.standard_normal((B, d_in)).astype(np.float32)
    logits = g.standard_normal((B, E))
    top = np.argsort(-logits, axis=1)[:, :k]
    wts = np.exp(np.take_along_axis(logits, top, 1))
    wts = (wts / wts.sum(1, keepdims=True)).astype(np.float32)
    tok = np.repeat(np.arange(B, dtype=np.int32), k)
    ex = top.reshape(-1)
    order = np.lexsort((tok, ex))
    offs = np.r_[0, np.cumsum(np.bincount(ex, minlength=E))].astype(np.int64)
    routing = (offs, tok[order], wts.reshape(-1)[order])
    cd = torch.from_numpy(codes.view(np.int64).copy() if len(codes) else np.zeros(1, np.int64)).to(DEV)
    pd = torch.from_numpy(params.view(np.int16).copy()).to(DEV)
    Y = bm.moe_decode_in(cd, pd, torch.from_numpy(bits_u).to(DEV), torch.from_numpy(off).to(DEV),
                         int(off[-1]), E, r, d_out, G, torch.from_numpy(Vt).to(DEV),
                         torch.from_numpy(X).to(DEV), routing).cpu().numpy()
    Chat = decode.dequantized_factors(codes, params, bits_u, d_out, G)
    return Y, decode.moe_decode_in(Chat, r, Vt, X, *routing)


@pytest.mark.parametrize("E,r,d_out,d_in,B,k,G,widths", [
    (4, 64, 128, 256, 24, 2, 64, (1, 2, 3, 4)),
    (6, 40, 192, 96, 17, 3, 32, (0, 1, 2, 4, 8, 16)),   # eviction and fp16 rows
    (3, 8, 64, 768, 1, 1, 32, (2, 3)),                  # 64-entry units, one token
    (4, 30, 9216, 64, 5, 2, 128, (1, 2, 16)),           # two segment blocks
    (16, 384, 768, 2048, 1, 8, 128, (1, 2, 3, 4)),      # Qwen3-30B-A3B gate, one token
    (16, 384, 768, 2048, 64, 8, 128, (1, 2, 3, 4)),     # the same, 64 tokens
])
def test_moe_decode_in_matches_oracle(E, r, d_out, d_in, B, k, G, widths):
    say("decode_in", E, r, d_out, d_in, B, k, G, widths)
    Y, ref = _run_in(E, r, d_out, d_in, B, k, G, widths, seed=E + r + B)
    assert relfro(Y, ref) <= REL
