"""The top-k decode entry point that allocates nothing
(bitsmoe_moe_decode_topk_noalloc), called through the C ABI, against the
allocating entry point (bitsmoe_moe_decode_topk) on the same inputs: calls
in a row, each smaller than the one before (the fixed scratch buffer keeps
the previous call's contents), every one bit-identical to the allocating
call and within the decode bar (1e-4 relative Frobenius) of the fp64
oracle."""
import ctypes
import sys

import numpy as np
import pytest

import oracle
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
    print("[gpu-noalloc]", *a, flush=True)
    sys.stdout.flush()


def relfro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def _case(E, r, d_in, d_out, B, k, G, widths, seed):
    """Packed units (by the oracle), basis, tokens and a top-k table."""
    g = np.random.default_rng(seed)
    C = (g.standard_normal((E * r, d_in)) * np.exp(g.standard_normal((E * r, 1)))).astype(np.float32)
    bits_u = g.choice(widths, size=E * r).astype(np.uint8)
    codes, params, off = oracle.pack(C, bits_u, G)
    Ut = np.ascontiguousarray(np.linalg.qr(g.standard_normal((d_out, r)))[0].T, dtype=np.float32)
    X = g.standard_normal((B, d_in)).astype(np.float32)
    logits = g.standard_normal((B, E))
    top = np.argsort(-logits, axis=1)[:, :k].astype(np.int32)
    w = np.exp(np.take_along_axis(logits, top, 1))
    w = (w / w.sum(1, keepdims=True)).astype(np.float32)
    ex, tok = top.reshape(-1), np.repeat(np.arange(B, dtype=np.int32), k)
    order = np.lexsort((tok, ex))
    offs = np.r_[0, np.cumsum(np.bincount(ex, minlength=E))].astype(np.int64)
    Chat = decode.dequantized_factors(codes, params, bits_u, d_in, G)
    ref = decode.moe_decode(Chat, r, Ut, X, offs, tok[order], w.reshape(-1)[order])
    t = {
        "codes": torch.from_numpy(codes.view(np.int64).copy() if len(codes) else np.zeros(1, np.int64)).to(DEV),
        "params": torch.from_numpy(params.view(np.int16).copy()).to(DEV),
        "bits": torch.from_numpy(bits_u).to(DEV),
        "off": torch.from_numpy(off).to(DEV),
        "Ut": torch.from_numpy(Ut).to(DEV),
        "X": torch.from_numpy(X).to(DEV),
        "top": torch.from_numpy(top).to(DEV),
        "w": torch.from_numpy(w).to(DEV),
    }
    return t, int(off[-1]), ref


def _call(fn, t, words, E, r, d_in, d_out, G, Y):
    B, k = t["top"].shape
    p = lambda x: ctypes.c_void_p(x.data_ptr())  # noqa: E731
    return fn(p(t["codes"]), p(t["params"]), p(t["bits"]), p(t["off"]), words, E, r, d_in, G,
              p(t["Ut"]), d_out, p(t["X"]), B, k, p(t["top"]), p(t["w"]), p(Y),
              ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_allocating_entry_point(order):
    L = bm.lib()
    # first call: a large batch (matrix-core path, about 9 MiB of the fixed
    # buffer: down-projection rows, 256 tokens, top-8); then smaller calls
    # that reuse (and overwrite only part of) the same buffer: a gate-shaped
    # batch of 20 tokens (matrix-core path, other layout) and 3 tokens (the
    # one-token-per-slot path)
    cases = [dict(E=16, r=1024, d_in=768, d_out=2048, B=256, k=8, G=128, widths=(1, 2, 3, 4, 16),
                  seed=31),
             dict(E=8, r=384, d_in=2048, d_out=768, B=20, k=2, G=128, widths=(0, 1, 2, 3, 4),
                  seed=32),
             dict(E=8, r=384, d_in=2048, d_out=768, B=3, k=2, G=64, widths=(0, 1, 2, 3, 16),
                  seed=33)]
    for c in cases:
        say("case", {k: v for k, v in c.items() if k != "widths"})
        t, words, ref = _case(**c)
        B, d_out = c["B"], c["d_out"]
        Ya = torch.full((B, d_out), float("nan"), dtype=torch.float32, device=DEV)
        Yn = torch.full((B, d_out), float("nan"), dtype=torch.float32, device=DEV)
        args = (t, words, c["E"], c["r"], c["d_in"], d_out, c["G"])
        assert _call(L.bitsmoe_moe_decode_topk, *args, Ya) == 0, bm.last_error()
        assert _call(L.bitsmoe_moe_decode_topk_noalloc, *args, Yn) == 0, bm.last_error()
        torch.cuda.synchronize()
        ya, yn = Ya.cpu().numpy(), Yn.cpu().numpy()
        assert np.all(np.isfinite(yn))
        assert np.array_equal(yn, ya), "noalloc and allocating decode differ"
        err = relfro(yn, ref)
        say("rel fro vs oracle", err)
        assert err <= REL


def test_noalloc_rejects_sizes_above_the_buffer():
    L = bm.lib()
    t, words, _ = _case(E=4, r=64, d_in=128, d_out=64, B=2, k=2, G=64, widths=(1, 2), seed=33)
    Y = torch.empty((2, 64), dtype=torch.float32, device=DEV)
    # r = 8192, B * k = 520: the partials alone (17 MB) exceed the 16 MiB
    big_B = 520
    bt = dict(t)
    bt["top"] = torch.zeros((big_B, 1), dtype=torch.int32, device=DEV)
    bt["w"] = torch.zeros((big_B, 1), dtype=torch.float32, device=DEV)
    bt["X"] = torch.zeros((big_B, 128), dtype=torch.float32, device=DEV)
    Yb = torch.empty((big_B, 64), dtype=torch.float32, device=DEV)
    st = _call(L.bitsmoe_moe_decode_topk_noalloc, bt, words, 4, 8192, 128, 64, 64, Yb)
    assert st == 2 and "fixed scratch" in bm.last_error()
    # a call that fits still works afterwards
    assert _call(L.bitsmoe_moe_decode_topk_noalloc, t, words, 4, 64, 128, 64, 64, Y) == 0
    torch.cuda.synchronize()
