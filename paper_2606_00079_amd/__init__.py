"""MI355X (gfx950) BitsMoE spectral quantizer: Python binding of libbitsmoe.

Thin ctypes marshalling over the C ABI declared in ``include/bitsmoe.h``.
Every step runs in the library (HIP kernels on the device, LAPACK and the
exact ILP on the host); torch is used only to allocate device memory and to
name the current stream.  There is no fallback: if the library is not built,
importing the functions raises.

Steps, in order (one projection type of one MoE layer):

    H      = gram(X)                         # X^T X / n
    M      = gram_experts(W)                 # sum_e W_e W_e^T (fp64)
    Ut, ev = shared_basis(M, r)              # top-r eigenvectors (host)
    C      = project(Ut, W)                  # C_e = U^T W_e, [E*r][d_in]
    L      = score(C, H, bits, group)        # delta H delta^T per (unit, width)
    b, obj = allocate(L, bits, budget)       # exact ILP (host)
    off    = pack_layout(b, d)
    codes, params = pack(C, b, off, group)
"""
from __future__ import annotations

import ctypes
import glob
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# BITSMOE_LIB selects another build of the same library (e.g. the
# host-sanitized libbitsmoe_san.so of ``build --sanitize``)
LIB_PATH = os.environ.get("BITSMOE_LIB") or os.path.join(_HERE, "libbitsmoe.so")

OK = 0
_STATUS = {0: "OK", 1: "ERR_ARG", 2: "ERR_SHAPE", 3: "ERR_DTYPE", 4: "ERR_DEVICE",
           5: "ERR_NOMEM", 6: "ERR_NUMERIC", 7: "ERR_INFEASIBLE", 8: "ERR_UNAVAILABLE"}
F32, BF16 = 0, 1

EXPORTS = [
    "bitsmoe_gram", "bitsmoe_gram_experts", "bitsmoe_shared_basis", "bitsmoe_project",
    "bitsmoe_score", "bitsmoe_allocate", "bitsmoe_allocate_ex", "bitsmoe_pack_layout",
    "bitsmoe_pack", "bitsmoe_unpack", "bitsmoe_set_lapack", "bitsmoe_last_error",
    "bitsmoe_release", "bitsmoe_version", "bitsmoe_timing", "bitsmoe_timing_only",
    "bitsmoe_kernel_time",
    "bitsmoe_surrogate", "bitsmoe_surrogate_budget", "bitsmoe_gram_experts_in",
    "bitsmoe_project_in", "bitsmoe_basis_importance", "bitsmoe_score_diag",
    "bitsmoe_gram_routed", "bitsmoe_score_routed", "bitsmoe_moe_decode",
    "bitsmoe_moe_decode_topk", "bitsmoe_shared_basis_gpu", "bitsmoe_moe_decode_in",
    "bitsmoe_moe_decode_topk_noalloc",
]
# Candidate widths of the surrogate table, in column order.
SURROGATE_WIDTHS = (0, 1, 2, 3, 4, 6, 8, 16)


class BitsmoeError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        self.status = status
        self.code = _STATUS.get(status, str(status))
        super().__init__(f"{where}: {self.code}: {msg}")


_lib = None


def _find_lapack() -> Optional[str]:
    """A LAPACK shared library for the host eigensolve: the one bundled with
    numpy/scipy (OpenBLAS), else the system one."""
    import numpy
    cands = []
    for mod_dir in (os.path.dirname(numpy.__file__),):
        parent = os.path.dirname(mod_dir)
        cands += sorted(glob.glob(os.path.join(parent, "numpy.libs", "libscipy_openblas*.so")))
        cands += sorted(glob.glob(os.path.join(parent, "scipy.libs", "libscipy_openblas*.so")))
    cands += ["liblapack.so.3"]
    return cands[0] if cands else None


def lib() -> ctypes.CDLL:
    """Loads libbitsmoe.so (built by ``paper_2606_00079_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_00079_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    L.bitsmoe_gram.argtypes = [vp, i32, i64, i64, vp, vp]
    L.bitsmoe_gram_experts.argtypes = [vp, i32, i64, i64, i64, vp, vp]
    L.bitsmoe_shared_basis.argtypes = [vp, i64, i64, vp, vp, vp, vp]
    L.bitsmoe_project.argtypes = [vp, vp, i32, i64, i64, i64, i64, vp, vp]
    L.bitsmoe_score.argtypes = [vp, i64, i64, vp, vp, i32, i32, vp, vp]
    L.bitsmoe_allocate.argtypes = [vp, i64, vp, i32, i64, vp, vp]
    L.bitsmoe_allocate_ex.argtypes = [vp, i64, vp, i32, i64, vp, vp, i64, vp]
    L.bitsmoe_pack_layout.argtypes = [vp, i64, i64, vp]
    L.bitsmoe_pack.argtypes = [vp, i64, i64, i32, vp, vp, i64, vp, vp, vp]
    L.bitsmoe_unpack.argtypes = [vp, vp, vp, vp, i64, i64, i64, i32, vp, vp]
    L.bitsmoe_surrogate.argtypes = [vp, i64, i64, vp, ctypes.c_double, vp, vp, vp, vp]
    L.bitsmoe_surrogate_budget.argtypes = [i64, i64, i64, i64, ctypes.c_double, vp]
    L.bitsmoe_gram_experts_in.argtypes = [vp, i32, i64, i64, i64, vp, vp]
    L.bitsmoe_project_in.argtypes = [vp, vp, i32, i64, i64, i64, i64, vp, vp]
    L.bitsmoe_basis_importance.argtypes = [vp, i64, i64, vp, vp, vp]
    L.bitsmoe_score_diag.argtypes = [vp, i64, i64, vp, i64, vp, i32, i32, vp, vp]
    L.bitsmoe_gram_routed.argtypes = [vp, i32, i64, i64, i64, vp, vp, vp, vp, vp]
    L.bitsmoe_score_routed.argtypes = [vp, i64, i64, vp, i64, vp, i32, i32, vp, vp]
    L.bitsmoe_moe_decode.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i32, vp, i64, vp, i64,
                                     vp, vp, vp, vp, vp]
    L.bitsmoe_shared_basis_gpu.argtypes = [vp, i64, i64, vp, vp, vp, vp]
    L.bitsmoe_moe_decode_in.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i32, vp, i64, vp, i64,
                                        vp, vp, vp, vp, vp]
    L.bitsmoe_moe_decode_topk.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i32, vp, i64, vp,
                                          i64, i64, vp, vp, vp, vp]
    L.bitsmoe_moe_decode_topk_noalloc.argtypes = L.bitsmoe_moe_decode_topk.argtypes
    L.bitsmoe_set_lapack.argtypes = [ctypes.c_char_p]
    L.bitsmoe_timing.argtypes = [i32]
    L.bitsmoe_timing_only.argtypes = [ctypes.c_char_p]
    L.bitsmoe_kernel_time.argtypes = [ctypes.c_char_p, vp, vp]
    L.bitsmoe_last_error.restype = ctypes.c_char_p
    L.bitsmoe_version.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("bitsmoe_last_error", "bitsmoe_version", "bitsmoe_release"):
            getattr(L, name).restype = ctypes.c_int
    L.bitsmoe_release.restype = None
    lp = _find_lapack()
    if lp and os.environ.get("BITSMOE_LAPACK") is None:
        L.bitsmoe_set_lapack(lp.encode())
    _lib = L
    return L


def _check(st: int, where: str) -> None:
    if st != OK:
        raise BitsmoeError(st, where, lib().bitsmoe_last_error().decode())


# ---------------------------------------------------------------------------
# torch glue (device memory and streams only)
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _stream():
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def _dev(t, name: str):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _dtype_code(t, name: str) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"{name} must be bfloat16 or float32")


def _bits_arr(bits: Sequence[int]):
    a = np.ascontiguousarray(np.asarray(bits, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.c_void_p)


def gram(X, out=None):
    """H = X^T X / n for calibration rows X [n][d] (bf16 or fp32) -> fp32 [d][d]."""
    torch = _torch()
    n, d = X.shape
    if out is None:
        out = torch.empty((d, d), dtype=torch.float32, device=X.device)
    _check(lib().bitsmoe_gram(_dev(X, "X"), _dtype_code(X, "X"), n, d, _dev(out, "H"), _stream()),
           "gram")
    return out


def gram_experts(W, out=None):
    """M = sum_e W_e W_e^T for W [E][d_out][d_in] -> fp64 [d_out][d_out]."""
    torch = _torch()
    E, d_out, d_in = W.shape
    if out is None:
        out = torch.empty((d_out, d_out), dtype=torch.float64, device=W.device)
    _check(lib().bitsmoe_gram_experts(_dev(W, "W"), _dtype_code(W, "W"), E, d_out, d_in,
                                      _dev(out, "M"), _stream()), "gram_experts")
    return out


def shared_basis(M, r: int, out=None) -> Tuple[object, np.ndarray, float]:
    """Top-r eigenvectors of M (host LAPACK). Returns (Ut [r][d_out] fp32, eigvals, host_ms)."""
    torch = _torch()
    d = M.shape[0]
    if M.dtype != torch.float64:
        raise TypeError("M must be float64")
    if out is None:
        out = torch.empty((r, d), dtype=torch.float32, device=M.device)
    ev = np.zeros(r, dtype=np.float64)
    ms = ctypes.c_double(0.0)
    _check(lib().bitsmoe_shared_basis(_dev(M, "M"), d, r, _dev(out, "Ut"),
                                      ev.ctypes.data_as(ctypes.c_void_p), ctypes.byref(ms),
                                      _stream()), "shared_basis")
    return out, ev, ms.value


def shared_basis_gpu(M, r: int, out=None) -> Tuple[object, np.ndarray, float]:
    """Top-r eigenvectors of M, tridiagonal reduction on the device.
    Returns (Ut [r][d_out] fp32, eigvals, wall ms of the call)."""
    torch = _torch()
    d = M.shape[0]
    if M.dtype != torch.float64:
        raise TypeError("M must be float64")
    if out is None:
        out = torch.empty((r, d), dtype=torch.float32, device=M.device)
    ev = np.zeros(r, dtype=np.float64)
    ms = ctypes.c_double(0.0)
    _check(lib().bitsmoe_shared_basis_gpu(_dev(M, "M"), d, r, _dev(out, "Ut"),
                                          ev.ctypes.data_as(ctypes.c_void_p), ctypes.byref(ms),
                                          _stream()), "shared_basis_gpu")
    return out, ev, ms.value


def project(Ut, W, out=None):
    """C_e = U^T W_e -> fp32 [E*r][d_in] (unit u = e*r + k)."""
    torch = _torch()
    r, d_out = Ut.shape
    E, d_out2, d_in = W.shape
    if d_out2 != d_out:
        raise ValueError("Ut and W disagree on d_out")
    if Ut.dtype != torch.float32:
        raise TypeError("Ut must be float32")
    if out is None:
        out = torch.empty((E * r, d_in), dtype=torch.float32, device=W.device)
    _check(lib().bitsmoe_project(_dev(Ut, "Ut"), _dev(W, "W"), _dtype_code(W, "W"), E, d_out, d_in,
                                 r, _dev(out, "C"), _stream()), "project")
    return out


def score(C, H, bits: Sequence[int], group: int, out=None):
    """L[u][j] = delta H delta^T for every unit and width -> fp32 [units][len(bits)]."""
    torch = _torch()
    units, d = C.shape
    if C.dtype != torch.float32 or H.dtype != torch.float32:
        raise TypeError("C and H must be float32")
    if tuple(H.shape) != (d, d):
        raise ValueError("H must be [d][d]")
    b, bp = _bits_arr(bits)
    if out is None:
        out = torch.empty((units, len(b)), dtype=torch.float32, device=C.device)
    _check(lib().bitsmoe_score(_dev(C, "C"), units, d, _dev(H, "H"), bp, len(b), group,
                               _dev(out, "L"), _stream()), "score")
    return out


def gram_experts_in(W, out=None):
    """M_in = sum_e W_e^T W_e for W [E][d_out][d_in] -> fp64 [d_in][d_in] (input-space basis)."""
    torch = _torch()
    E, d_out, d_in = W.shape
    if out is None:
        out = torch.empty((d_in, d_in), dtype=torch.float64, device=W.device)
    _check(lib().bitsmoe_gram_experts_in(_dev(W, "W"), _dtype_code(W, "W"), E, d_out, d_in,
                                         _dev(out, "M_in"), _stream()), "gram_experts_in")
    return out


def project_in(Vt, W, out=None):
    """C_e = Phi_r^T W_e^T -> fp32 [E*r][d_out] (unit u = e*r + k is the column W_e phi_k)."""
    torch = _torch()
    r, d_in = Vt.shape
    E, d_out, d_in2 = W.shape
    if d_in2 != d_in:
        raise ValueError("Vt and W disagree on d_in")
    if Vt.dtype != torch.float32:
        raise TypeError("Vt must be float32")
    if out is None:
        out = torch.empty((E * r, d_out), dtype=torch.float32, device=W.device)
    _check(lib().bitsmoe_project_in(_dev(Vt, "Vt"), _dev(W, "W"), _dtype_code(W, "W"), E, d_out,
                                    d_in, r, _dev(out, "C"), _stream()), "project_in")
    return out


def basis_importance(Vt, H, out=None):
    """beta_k = phi_k^T H phi_k for the rows of Vt -> fp32 [r]."""
    torch = _torch()
    r, d = Vt.shape
    if Vt.dtype != torch.float32 or H.dtype != torch.float32:
        raise TypeError("Vt and H must be float32")
    if tuple(H.shape) != (d, d):
        raise ValueError("H must be [d][d]")
    if out is None:
        out = torch.empty((r,), dtype=torch.float32, device=Vt.device)
    _check(lib().bitsmoe_basis_importance(_dev(Vt, "Vt"), r, d, _dev(H, "H"), _dev(out, "beta"),
                                          _stream()), "basis_importance")
    return out


def score_diag(C, beta, bits: Sequence[int], group: int, out=None):
    """L[u][j] = beta[u % r] ||c_u - Q_{bits[j]}(c_u)||^2 -> fp32 [units][len(bits)]."""
    torch = _torch()
    units, d = C.shape
    if C.dtype != torch.float32 or beta.dtype != torch.float32:
        raise TypeError("C and beta must be float32")
    b, bp = _bits_arr(bits)
    if out is None:
        out = torch.empty((units, len(b)), dtype=torch.float32, device=C.device)
    _check(lib().bitsmoe_score_diag(_dev(C, "C"), units, d, _dev(beta, "beta"), beta.shape[0], bp,
                                    len(b), group, _dev(out, "L"), _stream()), "score_diag")
    return out


def gram_routed(X, offsets, rows, weights, out=None):
    """Per-expert routed Grams H_e = (1/n) sum w x x^T -> fp32 [E][d][d]; the
    routing tables (offsets [E+1], rows [nnz], weights [nnz]) are host arrays."""
    torch = _torch()
    n, d = X.shape
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int64))
    rw = np.ascontiguousarray(np.asarray(rows, dtype=np.int32))
    wt = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    E = off.shape[0] - 1
    if rw.shape[0] < off[-1] or wt.shape[0] < off[-1]:
        raise ValueError("rows and weights need offsets[-1] entries")
    if out is None:
        out = torch.empty((E, d, d), dtype=torch.float32, device=X.device)
    _check(lib().bitsmoe_gram_routed(_dev(X, "X"), _dtype_code(X, "X"), n, d, E,
                                     off.ctypes.data_as(ctypes.c_void_p),
                                     rw.ctypes.data_as(ctypes.c_void_p),
                                     wt.ctypes.data_as(ctypes.c_void_p), _dev(out, "H"),
                                     _stream()), "gram_routed")
    return out


def score_routed(C, Hs, units_per_h: int, bits: Sequence[int], group: int, out=None):
    """Loss table with one H per block of units_per_h units -> fp32 [units][len(bits)]."""
    torch = _torch()
    units, d = C.shape
    if C.dtype != torch.float32 or Hs.dtype != torch.float32:
        raise TypeError("C and H must be float32")
    if Hs.dim() != 3 or tuple(Hs.shape[1:]) != (d, d) or Hs.shape[0] * units_per_h != units:
        raise ValueError("Hs must be [units / units_per_h][d][d]")
    b, bp = _bits_arr(bits)
    if out is None:
        out = torch.empty((units, len(b)), dtype=torch.float32, device=C.device)
    _check(lib().bitsmoe_score_routed(_dev(C, "C"), units, d, _dev(Hs, "H"), units_per_h, bp, len(b),
                                      group, _dev(out, "L"), _stream()), "score_routed")
    return out


def moe_decode(codes, params, bits_dev, offsets_dev, total_words: int, E: int, r: int, d_in: int,
               group: int, Ut, X, routing, out=None):
    """y = U sum_j g_j C^_e x for every token of X [B][d_in] (fp32) from the packed
    units; routing = (offsets [E+1], tokens, weights) host arrays -> fp32 [B][d_out]."""
    torch = _torch()
    B = X.shape[0]
    d_out = Ut.shape[1]
    if X.dtype != torch.float32 or Ut.dtype != torch.float32:
        raise TypeError("X and Ut must be float32")
    if X.dim() != 2 or X.shape[1] != d_in or Ut.dim() != 2 or Ut.shape[0] != r:
        raise ValueError("X must be [B][d_in] and Ut [r][d_out]")
    off = np.ascontiguousarray(np.asarray(routing[0], dtype=np.int64))
    tok = np.ascontiguousarray(np.asarray(routing[1], dtype=np.int32))
    wt = np.ascontiguousarray(np.asarray(routing[2], dtype=np.float32))
    if off.shape[0] != E + 1 or tok.shape[0] < off[-1] or wt.shape[0] < off[-1]:
        raise ValueError("routing tables do not match E")
    if out is None:
        out = torch.empty((B, d_out), dtype=torch.float32, device=X.device)
    _check(lib().bitsmoe_moe_decode(_dev(codes, "codes"), _dev(params, "params"),
                                    _dev(bits_dev, "bits"), _dev(offsets_dev, "offsets"),
                                    int(total_words), E, r, d_in, group, _dev(Ut, "Ut"), d_out,
                                    _dev(X, "X"), B, off.ctypes.data_as(ctypes.c_void_p),
                                    tok.ctypes.data_as(ctypes.c_void_p),
                                    wt.ctypes.data_as(ctypes.c_void_p), _dev(out, "Y"), _stream()),
           "moe_decode")
    return out


def moe_decode_in(codes, params, bits_dev, offsets_dev, total_words: int, E: int, r: int,
                  d_out: int, group: int, Vt, X, routing, out=None):
    """Input-space (gate/up) decode: y = sum_j g_j C^_e^T (Vt x) for every token
    of X [B][d_in] (fp32); Vt [r][d_in] fp32; units of length d_out ->
    fp32 [B][d_out]."""
    torch = _torch()
    B = X.shape[0]
    if X.dtype != torch.float32 or Vt.dtype != torch.float32:
        raise TypeError("X and Vt must be float32")
    if X.dim() != 2 or Vt.dim() != 2 or Vt.shape[0] != r or Vt.shape[1] != X.shape[1]:
        raise ValueError("Vt must be [r][d_in] and X [B][d_in]")
    off = np.ascontiguousarray(np.asarray(routing[0], dtype=np.int64))
    tok = np.ascontiguousarray(np.asarray(routing[1], dtype=np.int32))
    wt = np.ascontiguousarray(np.asarray(routing[2], dtype=np.float32))
    if off.shape[0] != E + 1 or tok.shape[0] < off[-1] or wt.shape[0] < off[-1]:
        raise ValueError("routing tables do not match E")
    if out is None:
        out = torch.empty((B, d_out), dtype=torch.float32, device=X.device)
    _check(lib().bitsmoe_moe_decode_in(_dev(codes, "codes"), _dev(params, "params"),
                                       _dev(bits_dev, "bits"), _dev(offsets_dev, "offsets"),
                                       int(total_words), E, r, d_out, group, _dev(Vt, "Vt"),
                                       X.shape[1], _dev(X, "X"), B,
                                       off.ctypes.data_as(ctypes.c_void_p),
                                       tok.ctypes.data_as(ctypes.c_void_p),
                                       wt.ctypes.data_as(ctypes.c_void_p), _dev(out, "Y"), _stream()),
           "moe_decode_in")
    return out


def moe_decode_topk(codes, params, bits_dev, offsets_dev, total_words: int, E: int, r: int,
                    d_in: int, group: int, Ut, X, topk_experts, topk_weights, out=None,
                    noalloc: bool = False):
    """moe_decode from the router's device top-k table: topk_experts int32
    [B][k], topk_weights fp32 [B][k] (both on the device) -> fp32 [B][d_out].
    noalloc=True calls bitsmoe_moe_decode_topk_noalloc (no device allocation
    in the library; pass ``out`` to allocate nothing here either)."""
    torch = _torch()
    B = X.shape[0]
    d_out = Ut.shape[1]
    if X.dtype != torch.float32 or Ut.dtype != torch.float32 or topk_weights.dtype != torch.float32:
        raise TypeError("X, Ut and topk_weights must be float32")
    if topk_experts.dtype != torch.int32:
        raise TypeError("topk_experts must be int32")
    if X.dim() != 2 or X.shape[1] != d_in or Ut.dim() != 2 or Ut.shape[0] != r:
        raise ValueError("X must be [B][d_in] and Ut [r][d_out]")
    if topk_experts.dim() != 2 or topk_experts.shape[0] != B or \
            tuple(topk_weights.shape) != tuple(topk_experts.shape):
        raise ValueError("topk_experts and topk_weights must both be [B][k]")
    k = topk_experts.shape[1]
    if out is None:
        out = torch.empty((B, d_out), dtype=torch.float32, device=X.device)
    fn = lib().bitsmoe_moe_decode_topk_noalloc if noalloc else lib().bitsmoe_moe_decode_topk
    _check(fn(_dev(codes, "codes"), _dev(params, "params"), _dev(bits_dev, "bits"),
              _dev(offsets_dev, "offsets"), int(total_words), E, r, d_in, group, _dev(Ut, "Ut"),
              d_out, _dev(X, "X"), B, k, _dev(topk_experts, "topk_experts"),
              _dev(topk_weights, "topk_weights"), _dev(out, "Y"), _stream()),
           "moe_decode_topk_noalloc" if noalloc else "moe_decode_topk")
    return out


def surrogate(C, H, gamma: float, kappa: Sequence[float], out=None, stats=None):
    """The paper's surrogate costs alpha^2 beta^gamma E(b) for the widths
    SURROGATE_WIDTHS -> fp32 [units][8]; ``stats`` (optional, [units][4]) gets
    {alpha^2, beta, rho, cos theta}."""
    torch = _torch()
    units, d = C.shape
    if C.dtype != torch.float32 or H.dtype != torch.float32:
        raise TypeError("C and H must be float32")
    if tuple(H.shape) != (d, d):
        raise ValueError("H must be [d][d]")
    k = np.ascontiguousarray(np.asarray(kappa, dtype=np.float64))
    if k.shape != (3,):
        raise ValueError("kappa holds the coefficients of widths 2, 3, 4")
    if out is None:
        out = torch.empty((units, len(SURROGATE_WIDTHS)), dtype=torch.float32, device=C.device)
    sp = _dev(stats, "stats") if stats is not None else None
    _check(lib().bitsmoe_surrogate(_dev(C, "C"), units, d, _dev(H, "H"), float(gamma),
                                   k.ctypes.data_as(ctypes.c_void_p), _dev(out, "L"), sp,
                                   _stream()), "surrogate")
    return out


def surrogate_budget(E: int, n_out: int, m: int, r: int, b_eq: float) -> int:
    """Equivalent-bit ILP budget of one projection (host)."""
    b = ctypes.c_int64(0)
    _check(lib().bitsmoe_surrogate_budget(E, n_out, m, r, float(b_eq), ctypes.byref(b)),
           "surrogate_budget")
    return b.value


def allocate(L, bits: Sequence[int], budget: int, full_dp_limit: int = -1,
             return_core: bool = False):
    """Exact ILP on the host. L: host array [units][len(bits)] fp32."""
    Lh = np.ascontiguousarray(np.asarray(L, dtype=np.float32))
    units = Lh.shape[0]
    b, bp = _bits_arr(bits)
    out = np.zeros(units, dtype=np.uint8)
    obj = ctypes.c_double(0.0)
    core = ctypes.c_int64(0)
    _check(lib().bitsmoe_allocate_ex(Lh.ctypes.data_as(ctypes.c_void_p), units, bp, len(b),
                                     int(budget), out.ctypes.data_as(ctypes.c_void_p),
                                     ctypes.byref(obj), int(full_dp_limit), ctypes.byref(core)),
           "allocate")
    if return_core:
        return out, obj.value, core.value
    return out, obj.value


def pack_layout(bits_u, d: int) -> np.ndarray:
    bu = np.ascontiguousarray(np.asarray(bits_u, dtype=np.uint8))
    off = np.zeros(bu.shape[0] + 1, dtype=np.int64)
    _check(lib().bitsmoe_pack_layout(bu.ctypes.data_as(ctypes.c_void_p), bu.shape[0], d,
                                     off.ctypes.data_as(ctypes.c_void_p)), "pack_layout")
    return off


def pack(C, bits_dev, offsets_dev, group: int, total_words: int, codes=None, params=None):
    """Bit-plane codes (uint64 words, as int64 tensor) and fp16 params (as int16 [units][d/G][2])."""
    torch = _torch()
    units, d = C.shape
    if codes is None:
        codes = torch.empty((max(int(total_words), 1),), dtype=torch.int64, device=C.device)
    if params is None:
        params = torch.empty((units, d // group, 2), dtype=torch.int16, device=C.device)
    _check(lib().bitsmoe_pack(_dev(C, "C"), units, d, group, _dev(bits_dev, "bits"),
                              _dev(offsets_dev, "offsets"), int(total_words), _dev(codes, "codes"),
                              _dev(params, "params"), _stream()), "pack")
    return codes, params


def unpack(codes, params, bits_dev, offsets_dev, units: int, d: int, group: int,
           total_words: int, out=None):
    torch = _torch()
    if out is None:
        out = torch.empty((units, d), dtype=torch.float32, device=codes.device)
    _check(lib().bitsmoe_unpack(_dev(codes, "codes"), _dev(params, "params"), _dev(bits_dev, "bits"),
                                _dev(offsets_dev, "offsets"), int(total_words), units, d, group,
                                _dev(out, "Chat"), _stream()), "unpack")
    return out


def timing(enable: bool, only: Optional[str] = None) -> None:
    """Records HIP events around every main kernel while enabled (``only``:
    just around the kernels timed under that name)."""
    _check(lib().bitsmoe_timing_only((only or "").encode()), "timing")
    _check(lib().bitsmoe_timing(1 if enable else 0), "timing")


def kernel_time(name: str) -> Tuple[float, int]:
    """(summed ms, launches) of the kernel ``name`` since it was last read."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib().bitsmoe_kernel_time(name.encode(), ctypes.byref(ms), ctypes.byref(n)), "kernel_time")
    return ms.value, n.value


def release() -> None:
    lib().bitsmoe_release()


def version() -> str:
    return lib().bitsmoe_version().decode()


def last_error() -> str:
    return lib().bitsmoe_last_error().decode()
