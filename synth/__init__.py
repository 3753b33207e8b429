"""Seeded synthetic MoE projections and calibration activations.

This module only draws inputs.  It holds none of the quantizer's arithmetic:
no Gram, no basis, no fake-quant, no loss, no allocation.  Both the fp64
oracle (``oracle/``) and the HIP path (``paper_2606_00079_amd``) consume what
it returns; neither is imported here.

The paper measures on real checkpoints (Qwen3-30B-A3B, Mixtral-8x7B,
DeepSeek) calibrated with C4 samples (Sec. 4.1).  Neither the weights nor
the corpus are available, so seeded stand-ins of the same shapes are drawn:

* expert weights  W_e = U0 @ A_e + sigma * N(0, 1)   (a shared rank-k0
  component, which is what makes a cross-expert basis worthwhile, plus
  independent noise), U0 orthonormal (QR of a Gaussian, diag(R) > 0),
  A_e ~ N(0, 1/d_in);
* calibration rows X ~ N(0, 1) (Student-t nu=4 for the Mixtral shape) with a
  few outlier input channels scaled up, as LLM activations have;
* the down-projection calibration input is the SiLU-gated intermediate
  activation of expert 0: SiLU(X W_gate,0^T) * (X W_up,0^T).

Every expert has its own PCG64 stream ``[seed, config_id, proj_id, expert]``
so any subset of experts can be regenerated on its own.  Gaussians are drawn
in fp32; bf16 tensors are rounded to nearest-even and returned as their raw
uint16 bit patterns.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence

import numpy as np

__all__ = [
    "ProjSpec", "ConfigSpec", "CONFIGS", "Projection", "make_projection",
    "make_layer", "expert_weights", "calibration_input", "f32_to_bf16_bits",
    "bf16_bits_to_f32", "as_f64", "random_rows", "TOP_K", "routing",
]


# ----------------------------------------------------------------------------
# bf16 encoding (input encoding only)
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def as_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 values of a 'bf16' (uint16 bits) or 'f32' array."""
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------
# configuration table
# ----------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class ProjSpec:
    name: str          # gate / up / down / w1 / w2 / w3
    d_out: int
    d_in: int
    r: int             # shared-basis rank
    input: str         # "x" (layer input) or "act" (SiLU-gated intermediate)


@dataclasses.dataclass(frozen=True)
class ConfigSpec:
    name: str
    config_id: int
    E: int
    projs: Sequence[ProjSpec]
    n_tokens: int            # calibration rows
    dtype: str               # "bf16" or "f32" for W and X
    k0: int                  # rank of the planted shared component
    noise: float             # std of the independent weight noise
    x_dist: str              # "normal" or "t4"
    outlier_frac: float      # fraction of input channels that are outliers
    outlier_count: int       # used instead of the fraction when > 0
    outlier_scale: float
    bits: Sequence[int]
    group: int
    budget: float            # average bits per spectral unit

    def proj(self, name: str) -> ProjSpec:
        for p in self.projs:
            if p.name == name:
                return p
        raise KeyError(name)

    def budget_bits(self, p: ProjSpec) -> int:
        """Total bit budget of one projection's ILP: floor(avg * E * r)."""
        return int(math.floor(self.budget * self.E * p.r))


def _qwen_projs():
    return (ProjSpec("gate", 768, 2048, 384, "x"),
            ProjSpec("up", 768, 2048, 384, "x"),
            ProjSpec("down", 2048, 768, 1024, "act"))


CONFIGS: Dict[str, ConfigSpec] = {
    # E=4, W_e 128x256 fp32, shared U0 128x32, X 512x256 with 4 outliers x20.
    "tiny": ConfigSpec("tiny", 0, 4, (ProjSpec("gate", 128, 256, 64, "x"),),
                       512, "f32", 32, 0.05, "normal", 0.0, 4, 20.0,
                       (1, 2, 3, 4), 64, 2.0),
    # Qwen3-30B-A3B-shaped gate_proj alone.
    "qwen_gate": ConfigSpec("qwen_gate", 1, 128, (ProjSpec("gate", 768, 2048, 384, "x"),),
                            4096, "bf16", 128, 0.02, "normal", 0.01, 0, 20.0,
                            (1, 2, 3, 4), 128, 2.0),
    # Qwen3-30B-A3B-shaped full MoE layer (gate, up, down).
    "qwen_layer": ConfigSpec("qwen_layer", 2, 128, _qwen_projs(),
                             4096, "bf16", 128, 0.02, "normal", 0.01, 0, 20.0,
                             (1, 2, 3, 4), 128, 2.0),
    # Mixtral-8x7B-shaped layer, heavy-tailed X.
    "mixtral": ConfigSpec("mixtral", 3, 8,
                          (ProjSpec("w1", 14336, 4096, 3584, "x"),
                           ProjSpec("w3", 14336, 4096, 3584, "x"),
                           ProjSpec("w2", 4096, 14336, 1024, "act")),
                          8192, "bf16", 128, 0.02, "t4", 0.0, 0, 1.0,
                          (1, 2, 3, 4), 128, 2.5),
    # DeepSeek-V3-shaped layer.
    "dsv3": ConfigSpec("dsv3", 4, 256,
                       (ProjSpec("gate", 2048, 7168, 1024, "x"),
                        ProjSpec("up", 2048, 7168, 1024, "x"),
                        ProjSpec("down", 7168, 2048, 3584, "act")),
                       8192, "bf16", 128, 0.02, "normal", 0.005, 0, 30.0,
                       (1, 2, 3, 4, 8), 128, 2.0),
}


def _proj_id(cfg: ConfigSpec, pname: str) -> int:
    return [p.name for p in cfg.projs].index(pname)


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng([int(k) for k in key])


def _encode(a32: np.ndarray, dtype: str) -> np.ndarray:
    return f32_to_bf16_bits(a32) if dtype == "bf16" else np.ascontiguousarray(a32, np.float32)


def _decode32(a: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits_to_f32(a) if dtype == "bf16" else np.asarray(a, np.float32)


def shared_component(cfg: ConfigSpec, pname: str, seed: int = 0) -> np.ndarray:
    """U0: d_out x k0 with orthonormal columns (QR, diag(R) made positive)."""
    p = cfg.proj(pname)
    g = _rng(seed, cfg.config_id, _proj_id(cfg, pname), 1_000_000)
    G = g.standard_normal((p.d_out, cfg.k0), dtype=np.float32).astype(np.float64)
    Q, R = np.linalg.qr(G)
    Q = Q * np.sign(np.diag(R))[None, :]
    return Q.astype(np.float32)


def expert_weights(cfg: ConfigSpec, pname: str, experts: Optional[Sequence[int]] = None,
                   seed: int = 0, threads: Optional[int] = None) -> np.ndarray:
    """Stacked expert weights [len(experts)][d_out][d_in] (bf16 bits or fp32)."""
    p = cfg.proj(pname)
    pid = _proj_id(cfg, pname)
    if experts is None:
        experts = range(cfg.E)
    experts = list(experts)
    U0 = shared_component(cfg, pname, seed)
    dt = np.uint16 if cfg.dtype == "bf16" else np.float32
    out = np.empty((len(experts), p.d_out, p.d_in), dtype=dt)
    a_std = np.float32(1.0 / math.sqrt(p.d_in))
    noise = np.float32(cfg.noise)

    def one(i: int) -> None:
        e = experts[i]
        g = _rng(seed, cfg.config_id, pid, e)
        A = g.standard_normal((cfg.k0, p.d_in), dtype=np.float32) * a_std
        N = g.standard_normal((p.d_out, p.d_in), dtype=np.float32) * noise
        out[i] = _encode(U0 @ A + N, cfg.dtype)

    nthr = threads or min(16, os.cpu_count() or 1)
    if len(experts) <= 2 or nthr <= 1:
        for i in range(len(experts)):
            one(i)
    else:
        with ThreadPoolExecutor(nthr) as ex:
            list(ex.map(one, range(len(experts))))
    return out


def _layer_input_f32(cfg: ConfigSpec, seed: int) -> np.ndarray:
    d_in = next(p.d_in for p in cfg.projs if p.input == "x")
    g = _rng(seed, cfg.config_id, 99, 0)
    n = cfg.n_tokens
    if cfg.x_dist == "normal":
        X = g.standard_normal((n, d_in), dtype=np.float32)
    elif cfg.x_dist == "t4":
        X = g.standard_t(4.0, size=(n, d_in)).astype(np.float32)
    else:
        raise ValueError(cfg.x_dist)
    n_out = cfg.outlier_count or int(math.ceil(cfg.outlier_frac * d_in))
    if n_out > 0 and cfg.outlier_scale != 1.0:
        cols = np.sort(g.choice(d_in, size=n_out, replace=False))
        X[:, cols] *= np.float32(cfg.outlier_scale)
    return X


# Routed experts per token of the model families the configurations stand in
# for (Qwen3-30B-A3B: 8 of 128; Mixtral-8x7B: 2 of 8; DeepSeek-V3: 8 of 256).
TOP_K = {"tiny": 2, "qwen_gate": 8, "qwen_layer": 8, "mixtral": 2, "dsv3": 8}


def routing(cfg: ConfigSpec, X: Optional[np.ndarray] = None, seed: int = 0):
    """Synthetic top-k routing of the calibration tokens of a layer.

    A random linear router R ~ N(0, 1/d_in) [d_in][E] scores every token of
    the layer input (logits = X R in fp32); each token goes to its TOP_K
    highest-scoring experts with weights softmax-normalized over those k.
    Returned grouped by expert, tokens ascending within an expert:
    (offsets int64 [E+1], tokens int32 [n k], weights float32 [n k]).
    """
    if X is None:
        X = _decode32(_encode(_layer_input_f32(cfg, seed), cfg.dtype), cfg.dtype)
    else:
        X = _decode32(X, cfg.dtype)
    n, d_in = X.shape
    E, k = cfg.E, TOP_K[cfg.name]
    g = _rng(seed, cfg.config_id, 98, 0)
    R = (g.standard_normal((d_in, E), dtype=np.float32) / np.float32(math.sqrt(d_in)))
    logits = X @ R
    top = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    z = np.take_along_axis(logits, top, axis=1).astype(np.float64)
    w = np.exp(z - z.max(axis=1, keepdims=True))
    w = (w / w.sum(axis=1, keepdims=True)).astype(np.float32)
    tok = np.repeat(np.arange(n, dtype=np.int32), k)
    ex = top.reshape(-1)
    order = np.lexsort((tok, ex))
    counts = np.bincount(ex, minlength=E)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    return offsets, tok[order], w.reshape(-1)[order]


def calibration_input(cfg: ConfigSpec, pname: str, seed: int = 0) -> np.ndarray:
    """Calibration rows [n][d_in] for projection ``pname`` (bf16 bits or fp32).

    Up-projections read the layer input X.  The down projection reads the
    SiLU-gated intermediate activation of expert 0,
    SiLU(X W_gate,0^T) * (X W_up,0^T), formed in fp32 from the rounded X and
    weights and then rounded to the storage type.
    """
    p = cfg.proj(pname)
    X32 = _decode32(_encode(_layer_input_f32(cfg, seed), cfg.dtype), cfg.dtype)
    if p.input == "x":
        return _encode(X32, cfg.dtype)
    ins = [q.name for q in cfg.projs if q.input == "x"]
    Wg = _decode32(expert_weights(cfg, ins[0], [0], seed)[0], cfg.dtype)
    Wu = _decode32(expert_weights(cfg, ins[1], [0], seed)[0], cfg.dtype)
    G = X32 @ Wg.T
    U = X32 @ Wu.T
    A = (G / (np.float32(1.0) + np.exp(-G))) * U
    assert A.shape[1] == p.d_in
    return _encode(A.astype(np.float32), cfg.dtype)


@dataclasses.dataclass
class Projection:
    """One projection's quantizer inputs."""
    cfg: ConfigSpec
    spec: ProjSpec
    W: np.ndarray          # [E][d_out][d_in]
    X: np.ndarray          # [n][d_in]
    dtype: str

    @property
    def E(self) -> int:
        return self.W.shape[0]

    @property
    def r(self) -> int:
        return self.spec.r

    @property
    def bits(self) -> List[int]:
        return list(self.cfg.bits)

    @property
    def group(self) -> int:
        return self.cfg.group

    @property
    def budget_bits(self) -> int:
        return int(math.floor(self.cfg.budget * self.E * self.spec.r))


def make_projection(config: str, pname: Optional[str] = None, seed: int = 0,
                    experts: Optional[Sequence[int]] = None) -> Projection:
    cfg = CONFIGS[config]
    spec = cfg.projs[0] if pname is None else cfg.proj(pname)
    W = expert_weights(cfg, spec.name, experts, seed)
    X = calibration_input(cfg, spec.name, seed)
    return Projection(cfg, spec, W, X, cfg.dtype)


def make_layer(config: str, seed: int = 0) -> List[Projection]:
    cfg = CONFIGS[config]
    X = None
    out = []
    for spec in cfg.projs:
        W = expert_weights(cfg, spec.name, None, seed)
        if spec.input == "x":
            if X is None:
                X = calibration_input(cfg, spec.name, seed)
            Xp = X
        else:
            Xp = calibration_input(cfg, spec.name, seed)
        out.append(Projection(cfg, spec, W, Xp, cfg.dtype))
    return out


def random_rows(rows: int, d: int, seed: int, scale: float = 0.02,
                heavy: bool = False) -> np.ndarray:
    """Generic fp32 rows for shape and edge-case tests (Gaussian or t3)."""
    g = _rng(seed, 7_000_000, rows, d)
    if heavy:
        return (g.standard_t(3.0, size=(rows, d)) * scale).astype(np.float32)
    return (g.standard_normal((rows, d), dtype=np.float32) * np.float32(scale))
