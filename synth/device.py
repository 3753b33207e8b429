"""Seeded synthetic inputs generated directly in device memory.

The same recipes as the host generators in ``synth`` (shared low-rank
component plus noise for the expert weights; Gaussian or Student-t calibration
rows with scaled outlier columns; the SiLU-gated intermediate activation for
down projections), drawn with torch's device RNG so that inputs of the largest
configurations (several GB per projection) never pass through host memory.
The values are not bit-identical to the host generators' (a different RNG),
only identically distributed.  Nothing here computes any step of the
quantizer.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np

from . import CONFIGS, ConfigSpec, shared_component, _proj_id


def _gen(device, *key: int):
    import torch
    g = torch.Generator(device=device)
    h = 0
    for k in key:  # fold the key into one 63-bit seed
        h = (h * 1_000_003 + int(k) + 0x9E3779B97F4A7C15) % (1 << 63)
    g.manual_seed(h)
    return g


def normal(shape, seed: int, scale: float = 1.0, dtype: str = "f32", device: str = "cuda"):
    """Gaussian N(0, scale^2) tensor of the given shape, drawn in fp32 and rounded."""
    import torch
    out = torch.empty(shape, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32,
                      device=device)
    g = _gen(device, seed, 7)
    flat = out.view(shape[0], -1) if len(shape) > 1 else out.view(1, -1)
    step = max(1, (1 << 26) // flat.shape[1])  # row blocks: no full-size fp32 temporary
    for i in range(0, flat.shape[0], step):
        blk = flat[i:i + step]
        blk.copy_((torch.randn(blk.shape, generator=g, device=device) * scale).to(out.dtype))
    return out


def expert_weights(cfg: ConfigSpec, pname: str, experts: Optional[Sequence[int]] = None,
                   seed: int = 0, device: str = "cuda"):
    """[len(experts)][d_out][d_in] bf16 (or fp32) expert weights U0 A_e + noise N."""
    import torch
    p = cfg.proj(pname)
    pid = _proj_id(cfg, pname)
    experts = list(range(cfg.E) if experts is None else experts)
    U0 = torch.from_numpy(shared_component(cfg, pname, seed)).to(device)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    out = torch.empty((len(experts), p.d_out, p.d_in), dtype=dt, device=device)
    a_std = 1.0 / math.sqrt(p.d_in)
    for i, e in enumerate(experts):
        g = _gen(device, seed, cfg.config_id, pid, e)
        A = torch.randn((cfg.k0, p.d_in), generator=g, device=device) * a_std
        N = torch.randn((p.d_out, p.d_in), generator=g, device=device) * cfg.noise
        out[i] = (U0 @ A + N).to(dt)
    return out


def _layer_input(cfg: ConfigSpec, seed: int, device: str):
    import torch
    d_in = next(p.d_in for p in cfg.projs if p.input == "x")
    g = _gen(device, seed, cfg.config_id, 99)
    n = cfg.n_tokens
    X = torch.randn((n, d_in), generator=g, device=device)
    if cfg.x_dist == "t4":  # Student-t, 4 degrees of freedom: z / sqrt(chi2_4 / 4)
        chi2 = sum(torch.randn((n, d_in), generator=g, device=device) ** 2 for _ in range(4))
        X = X / torch.sqrt(chi2 / 4.0)
    elif cfg.x_dist != "normal":
        raise ValueError(cfg.x_dist)
    n_out = cfg.outlier_count or int(math.ceil(cfg.outlier_frac * d_in))
    if n_out > 0 and cfg.outlier_scale != 1.0:
        cols = np.sort(np.random.default_rng([seed, cfg.config_id, 98]).choice(
            d_in, size=n_out, replace=False))
        X[:, torch.from_numpy(cols).to(device)] *= cfg.outlier_scale
    return X


def calibration_input(cfg: ConfigSpec, pname: str, seed: int = 0, device: str = "cuda"):
    """Calibration rows [n][d_in] (bf16, or fp32 for fp32 configurations).

    Projections reading the layer input get X; down projections get the
    SiLU-gated intermediate activation of expert 0,
    SiLU(X W_gate,0^T) * (X W_up,0^T), computed in fp32 and then rounded.
    """
    import torch
    p = cfg.proj(pname)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    X = _layer_input(cfg, seed, device)
    if p.input == "x":
        return X.to(dt)
    gate = next(q.name for q in cfg.projs if q.input == "x" and q.name in ("gate", "w1"))
    up = next(q.name for q in cfg.projs if q.input == "x" and q.name in ("up", "w3"))
    Xr = X.to(dt).float()
    Wg = expert_weights(cfg, gate, experts=[0], seed=seed, device=device)[0].float()
    Wu = expert_weights(cfg, up, experts=[0], seed=seed, device=device)[0].float()
    A = torch.nn.functional.silu(Xr @ Wg.T) * (Xr @ Wu.T)
    return A.to(dt)
