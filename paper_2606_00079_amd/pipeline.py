"""End-to-end driver: one projection, or a whole MoE layer, through the C ABI.

A projection runs three device segments separated by the two host steps:

    device:  gram (H), gram_experts (M)
    host:    shared_basis (LAPACK eigensolve of M)
    device:  project (C), score (L)
    host:    allocate (exact ILP over L)
    device:  pack (codes, params)

Device segments are timed with HIP events on the current stream; the host
steps with a wall clock.  Gate and up projections of a layer read the same
calibration input, so their H is computed once.

``surrogate_allocation`` runs the paper's own allocation on the same spectral
units: the closed-form surrogate costs on the device, then the ILP over the
widths {0, 1, 2, 3, 4, 6, 8, 16} under the equivalent-bit budget.
"""
from __future__ import annotations

import dataclasses
import time
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import (SURROGATE_WIDTHS, allocate, basis_importance, gram, gram_experts, gram_experts_in,
               gram_routed, pack, pack_layout, project, project_in, score, score_diag,
               score_routed, shared_basis, shared_basis_gpu, surrogate, surrogate_budget)


@dataclasses.dataclass
class ProjectionResult:
    H: object
    M: object
    Ut: object
    eigvals: np.ndarray
    C: object
    L: object
    bits_u: np.ndarray
    objective: float
    offsets: np.ndarray
    codes: object
    params: object
    times: Dict[str, float]


class _Seg:
    """HIP-event timer for one device segment on the current stream."""

    def __init__(self):
        import torch
        self.t = torch
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def __enter__(self):
        self.a.record()
        return self

    def __exit__(self, *exc):
        self.b.record()

    def ms(self) -> float:
        self.b.synchronize()
        return float(self.a.elapsed_time(self.b))


def _allocate_timed(seg: "_Seg", L, bits, budget: int, d: int, dev, times: Dict[str, float],
                    seg_key: str):
    """Waits for the device segment ``seg`` (its end event), copies L to the
    host, then times the ILP alone (host_ilp_ms).  The L copy and the copy
    of the widths and offsets back to the device are timed apart
    (host_copy_ms), so that neither device time nor transfers are counted as
    ILP time."""
    import torch
    times[seg_key] = seg.ms()              # synchronizes on the segment's end
    t0 = time.perf_counter()
    Lh = L.cpu().numpy()
    t1 = time.perf_counter()
    bits_u, obj = allocate(Lh, bits, budget)
    off = pack_layout(bits_u, d)
    t2 = time.perf_counter()
    bits_d = torch.from_numpy(bits_u).to(dev, non_blocking=False)
    off_d = torch.from_numpy(off).to(dev, non_blocking=False)
    t3 = time.perf_counter()
    times["host_ilp_ms"] = (t2 - t1) * 1e3
    times["host_copy_ms"] = ((t1 - t0) + (t3 - t2)) * 1e3
    return bits_u, obj, off, bits_d, off_d


def quantize_projection(W, X, r: int, bits: Sequence[int], group: int, budget: int,
                        H=None, eig: str = "host") -> ProjectionResult:
    """The hot path on one projection.  eig = "host" (LAPACK on M copied to
    the host) or "gpu" (tridiagonal reduction on the device); the eigensolve
    is timed apart from the device segments either way (host_eig_ms)."""
    import torch
    times: Dict[str, float] = {}
    dev = W.device
    E, d_out, d_in = W.shape
    # outputs are allocated before each segment's start event, so that the
    # segments time device work and launches only
    Hbuf = None
    if H is None:
        Hbuf = torch.empty((X.shape[1], X.shape[1]), dtype=torch.float32, device=dev)
    M = torch.empty((d_out, d_out), dtype=torch.float64, device=dev)
    s1 = _Seg()
    with s1:
        if H is None:
            H = gram(X, out=Hbuf)
        gram_experts(W, out=M)
    if eig == "gpu":
        Ut, ev, eig_ms = shared_basis_gpu(M, r)  # synchronizes the stream first
    elif eig == "host":
        Ut, ev, eig_ms = shared_basis(M, r)      # synchronizes the stream first
    else:
        raise ValueError("eig must be 'host' or 'gpu'")
    times["gpu_gram_ms"] = s1.ms()
    times["host_eig_ms"] = eig_ms
    C = torch.empty((E * r, d_in), dtype=torch.float32, device=dev)
    L = torch.empty((E * r, len(bits)), dtype=torch.float32, device=dev)
    s2 = _Seg()
    with s2:
        project(Ut, W, out=C)
        score(C, H, bits, group, out=L)
    bits_u, obj, off, bits_d, off_d = _allocate_timed(s2, L, bits, budget, C.shape[1], dev, times,
                                                      "gpu_score_ms")
    codes = torch.empty((max(int(off[-1]), 1),), dtype=torch.int64, device=dev)
    params = torch.empty((C.shape[0], d_in // group, 2), dtype=torch.int16, device=dev)
    s3 = _Seg()
    with s3:
        pack(C, bits_d, off_d, group, int(off[-1]), codes=codes, params=params)
    times["gpu_pack_ms"] = s3.ms()
    times["gpu_ms"] = times["gpu_gram_ms"] + times["gpu_score_ms"] + times["gpu_pack_ms"]
    return ProjectionResult(H, M, Ut, ev, C, L, bits_u, obj, off, codes, params, times)


def quantize_projection_in(W, X, r: int, bits: Sequence[int], group: int, budget: int,
                           H=None) -> ProjectionResult:
    """The paper's input-space construction of a gate/up projection (Sec. 3.2):
    basis Phi from M_in = sum W_e^T W_e, units W_e phi_k (rows of C, length
    d_out), loss beta_k ||c - Q_b(c)||^2 (diagonal approximation), exact ILP,
    pack.  ``Ut`` of the result holds Phi_r^T and ``M`` holds M_in."""
    import torch
    times: Dict[str, float] = {}
    dev = W.device
    E, d_out, d_in = W.shape
    Hbuf = None
    if H is None:
        Hbuf = torch.empty((d_in, d_in), dtype=torch.float32, device=dev)
    M = torch.empty((d_in, d_in), dtype=torch.float64, device=dev)
    s1 = _Seg()
    with s1:
        if H is None:
            H = gram(X, out=Hbuf)
        gram_experts_in(W, out=M)
    Vt, ev, eig_ms = shared_basis(M, r)
    times["gpu_gram_ms"] = s1.ms()
    times["host_eig_ms"] = eig_ms
    C = torch.empty((E * r, d_out), dtype=torch.float32, device=dev)
    beta = torch.empty((r,), dtype=torch.float32, device=dev)
    L = torch.empty((E * r, len(bits)), dtype=torch.float32, device=dev)
    s2 = _Seg()
    with s2:
        project_in(Vt, W, out=C)
        basis_importance(Vt, H, out=beta)
        score_diag(C, beta, bits, group, out=L)
    bits_u, obj, off, bits_d, off_d = _allocate_timed(s2, L, bits, budget, d_out, dev, times,
                                                      "gpu_score_ms")
    codes = torch.empty((max(int(off[-1]), 1),), dtype=torch.int64, device=dev)
    params = torch.empty((C.shape[0], d_out // group, 2), dtype=torch.int16, device=dev)
    s3 = _Seg()
    with s3:
        pack(C, bits_d, off_d, group, int(off[-1]), codes=codes, params=params)
    times["gpu_pack_ms"] = s3.ms()
    times["gpu_ms"] = times["gpu_gram_ms"] + times["gpu_score_ms"] + times["gpu_pack_ms"]
    res = ProjectionResult(H, M, Vt, ev, C, L, bits_u, obj, off, codes, params, times)
    res.beta = beta
    return res


def quantize_projection_routed(W, X, routing, r: int, bits: Sequence[int], group: int,
                               budget: int, Hs=None) -> ProjectionResult:
    """The hot path with the paper's routed calibration: one affinity-weighted
    Gram H_e per expert (App. B.2, Eq. app_affinity_gram) from ``routing`` =
    (offsets, rows, weights) over the rows of X, and every unit scored
    against its own expert's H_e.  ``H`` of the result holds the [E][d][d]
    Grams."""
    import torch
    times: Dict[str, float] = {}
    dev = W.device
    E, d_out, d_in = W.shape
    offsets, rows, weights = routing
    Hbuf = None
    if Hs is None:
        Hbuf = torch.empty((E, d_in, d_in), dtype=torch.float32, device=dev)
    M = torch.empty((d_out, d_out), dtype=torch.float64, device=dev)
    s1 = _Seg()
    with s1:
        if Hs is None:
            Hs = gram_routed(X, offsets, rows, weights, out=Hbuf)
        gram_experts(W, out=M)
    Ut, ev, eig_ms = shared_basis(M, r)
    times["gpu_gram_ms"] = s1.ms()
    times["host_eig_ms"] = eig_ms
    C = torch.empty((E * r, d_in), dtype=torch.float32, device=dev)
    L = torch.empty((E * r, len(bits)), dtype=torch.float32, device=dev)
    s2 = _Seg()
    with s2:
        project(Ut, W, out=C)
        score_routed(C, Hs, r, bits, group, out=L)
    bits_u, obj, off, bits_d, off_d = _allocate_timed(s2, L, bits, budget, d_in, dev, times,
                                                      "gpu_score_ms")
    codes = torch.empty((max(int(off[-1]), 1),), dtype=torch.int64, device=dev)
    params = torch.empty((C.shape[0], d_in // group, 2), dtype=torch.int16, device=dev)
    s3 = _Seg()
    with s3:
        pack(C, bits_d, off_d, group, int(off[-1]), codes=codes, params=params)
    times["gpu_pack_ms"] = s3.ms()
    times["gpu_ms"] = times["gpu_gram_ms"] + times["gpu_score_ms"] + times["gpu_pack_ms"]
    return ProjectionResult(Hs, M, Ut, ev, C, L, bits_u, obj, off, codes, params, times)


def quantize_layer(projs: List[dict], eig: str = "host") -> List[ProjectionResult]:
    """projs: dicts with W, X, r, bits, group, budget.  X objects that are the
    same tensor share one H."""
    cache = {}
    out = []
    for p in projs:
        key = id(p["X"])
        res = quantize_projection(p["W"], p["X"], p["r"], p["bits"], p["group"], p["budget"],
                                  H=cache.get(key), eig=eig)
        cache[key] = res.H
        out.append(res)
    return out


@dataclasses.dataclass
class SurrogateResult:
    L: object            # device [units][8] surrogate costs
    stats: object        # device [units][4] {alpha^2, beta, rho, cos theta}
    bits_u: np.ndarray   # chosen widths (0 = evicted, 16 = fp16)
    budget: int
    objective: float
    offsets: np.ndarray
    codes: object
    params: object
    times: Dict[str, float]


def surrogate_allocation(C, H, gamma: float, kappa: Sequence[float], E: int, n_out: int, r: int,
                         b_eq: float, group: int) -> SurrogateResult:
    """Surrogate costs of the units C (rows of U^T W_e), the ILP over the
    widths {0..16} under the equivalent-bit budget, and the packed units."""
    import torch
    units, d = C.shape
    dev = C.device
    L = torch.empty((units, len(SURROGATE_WIDTHS)), dtype=torch.float32, device=dev)
    st = torch.empty((units, 4), dtype=torch.float32, device=dev)
    budget = surrogate_budget(E, n_out, d, r, b_eq)
    seg = _Seg()
    with seg:
        surrogate(C, H, gamma, kappa, out=L, stats=st)
    times: Dict[str, float] = {}
    bits_u, obj, off, bits_d, off_d = _allocate_timed(seg, L, SURROGATE_WIDTHS, budget, d, dev,
                                                      times, "gpu_cost_ms")
    codes = torch.empty((max(int(off[-1]), 1),), dtype=torch.int64, device=dev)
    params = torch.empty((units, d // group, 2), dtype=torch.int16, device=dev)
    sp = _Seg()
    with sp:
        pack(C, bits_d, off_d, group, int(off[-1]), codes=codes, params=params)
    times["gpu_pack_ms"] = sp.ms()
    times["gpu_ms"] = times["gpu_cost_ms"] + times["gpu_pack_ms"]
    return SurrogateResult(L, st, bits_u, budget, obj, off, codes, params, times)
