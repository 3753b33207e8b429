"""Oracle: group-wise RTN quantizer, activation-aware loss table, packing.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The quantizer.  The paper derives its error model with a symmetric
per-vector quantizer (App. B.3, Eq. app_scalar_quantization_uk) and runs its
experiments with group size 128 (Sec. 4.1).  The hot path quantizes every
spectral unit with a group-wise *asymmetric* min/max round-to-nearest rule at
every candidate width, including 1 bit.  Zero point, scale format and
rounding are not stated in the paper; the reading fixed here is:

  for each group of G consecutive entries of the fp32 row, q_max = 2^b - 1,
  1. mn, mx = min and max of the group (exact);
  2. s32 = fl32(fl32(mx - mn) / q_max)  (IEEE fp32, round to nearest even);
     s16 = fp16(s32), m16 = fp16(mn)    (round to nearest even);
  3. if s16 == 0: q = 0, else q = clamp(rint((c - m16) / s16), 0, q_max) with
     the difference and the quotient taken in fp64 and rint rounding halves
     to even;
  4. the dequantized value is x_hat = m16 + q * s16.

The stored parameters are (s16, m16), so dequantizing packed codes gives
exactly x_hat.
"""
from __future__ import annotations

import numpy as np


def _rows32(c) -> np.ndarray:
    c = np.asarray(c)
    if c.ndim == 1:
        c = c[None, :]
    return np.ascontiguousarray(c, dtype=np.float32)


def quant_group(c, b: int, G: int):
    """Codes and group parameters of the fp32 rows ``c`` at width ``b``.

    Returns (q, s16, m16): q int64 [rows][d], s16 and m16 float16
    [rows][d/G].  The rule is the one in the module docstring.
    """
    c32 = _rows32(c)
    rows, d = c32.shape
    if d % G != 0:
        raise ValueError("quant_group: d must be a multiple of the group size")
    if not (1 <= b <= 16):
        raise ValueError("quant_group: width out of range")
    ng = d // G
    g = c32.reshape(rows, ng, G)
    mn = g.min(axis=2)
    mx = g.max(axis=2)
    qmax = (1 << b) - 1
    s32 = (mx - mn) / np.float32(qmax)            # fp32 subtract, fp32 divide
    assert s32.dtype == np.float32
    s16 = s32.astype(np.float16)
    m16 = mn.astype(np.float16)
    s = s16.astype(np.float64)[:, :, None]
    m = m16.astype(np.float64)[:, :, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = (g.astype(np.float64) - m) / s
        q = np.clip(np.rint(t), 0, qmax)
    q = np.where(s > 0, q, 0.0)
    return q.astype(np.int64).reshape(rows, d), s16, m16


def fake_quant(c, b: int, G: int) -> np.ndarray:
    """Dequantized rows x_hat = m16 + q * s16 (fp64), the value Q_b(c)."""
    q, s16, m16 = quant_group(c, b, G)
    rows, d = q.shape
    s = np.repeat(s16.astype(np.float64), G, axis=1)
    m = np.repeat(m16.astype(np.float64), G, axis=1)
    return m + q.astype(np.float64) * s


def score_rows(C, H, bits, G: int, rows=None) -> np.ndarray:
    """L[u, j] = delta H delta^T with delta = c_u - Q_{bits[j]}(c_u).

    For the output-space basis the layer loss is
    sum_k alpha_k^2 eps_k^T H eps_k (App. B.2, Eq. app_down_exact_metric);
    alpha_k eps_k is the quantization error of the unnormalized factor row
    c_k = alpha_k p_k, written delta here.  Codes are taken from fp32(c);
    delta is c (as given) minus the dequantized row, in fp64.

    ``rows`` selects a subset of units (all when None).
    """
    C = np.asarray(C)
    if rows is not None:
        C = C[np.asarray(rows)]
    H = np.asarray(H, dtype=np.float64)
    C64 = C.astype(np.float64)
    L = np.empty((C.shape[0], len(bits)), dtype=np.float64)
    for j, b in enumerate(bits):
        delta = C64 - fake_quant(C, int(b), G)
        L[:, j] = np.sum((delta @ H) * delta, axis=1)
    return L


def score(C, H, bits, G: int, chunk: int = 4096) -> np.ndarray:
    """The full loss table [units][len(bits)], computed in row chunks."""
    C = np.asarray(C)
    out = [score_rows(C[i:i + chunk], H, bits, G) for i in range(0, C.shape[0], chunk)]
    return np.concatenate(out, axis=0) if out else np.zeros((0, len(bits)))


# ----------------------------------------------------------------------------
# packing
# ----------------------------------------------------------------------------
def pack_layout(bits_u, d: int) -> np.ndarray:
    """Word offsets [units+1]: unit u holds bits_u[u] * d/64 uint64 words."""
    if d % 64 != 0:
        raise ValueError("pack_layout: d must be a multiple of 64")
    bits_u = np.asarray(bits_u, dtype=np.int64)
    off = np.zeros(bits_u.shape[0] + 1, dtype=np.int64)
    off[1:] = np.cumsum(bits_u * (d // 64))
    return off


def bit_planes(q: np.ndarray, b: int) -> np.ndarray:
    """Bit-plane words of code rows: [..., b, d/64] uint64 for q [..., d].

    Word w of plane t has bit j equal to bit t of q[64 w + j] (one row: the
    result is [b][d/64]).
    """
    q = np.asarray(q, dtype=np.uint64)
    d = q.shape[-1]
    lead = q.shape[:-1]
    shifts = np.arange(64, dtype=np.uint64)
    out = np.empty(lead + (b, d // 64), dtype=np.uint64)
    for t in range(b):
        bit = (q >> np.uint64(t)) & np.uint64(1)
        out[..., t, :] = np.sum(bit.reshape(lead + (d // 64, 64)) << shifts, axis=-1,
                                dtype=np.uint64)
    return out


def pack(C, bits_u, G: int, chunk: int = 8192):
    """Pack every unit at its assigned width.

    Widths 1..8 are codes of the group rule as bit planes.  The surrogate's
    two extra widths (Sec. 3.3, candidate set {16, 8, 6, 4, 3, 2, 1, 0}):
    16 stores the row itself in fp16 (round to nearest even), entry 4 w + i
    in bits 16 i .. 16 i + 15 of word w; 0 (eviction) stores nothing.  Their
    group parameters are zero.  Units of one width are packed together, in
    blocks of ``chunk`` units.

    Returns (codes uint64 [total words], params uint16 [units][d/G][2] holding
    the fp16 bit patterns of (s16, m16), offsets int64 [units+1]).
    """
    C32 = _rows32(C)
    units, d = C32.shape
    bits_u = np.asarray(bits_u, dtype=np.int64)
    off = pack_layout(bits_u, d)
    codes = np.zeros(int(off[-1]), dtype=np.uint64)
    params = np.zeros((units, d // G, 2), dtype=np.uint16)
    for b in np.unique(bits_u):
        if b == 0:
            continue
        if b != 16 and not 1 <= b <= 8:
            raise ValueError("pack: widths are 0, 1..8 or 16")
        for i0 in range(0, int(np.count_nonzero(bits_u == b)), chunk):
            us = np.nonzero(bits_u == b)[0][i0:i0 + chunk]
            words = int(b) * d // 64
            where = off[us][:, None] + np.arange(words)[None, :]
            if b == 16:
                codes[where] = C32[us].astype(np.float16).view(np.uint64).reshape(len(us), words)
                continue
            q, s16, m16 = quant_group(C32[us], int(b), G)
            params[us, :, 0] = s16.view(np.uint16)
            params[us, :, 1] = m16.view(np.uint16)
            codes[where] = bit_planes(q, int(b)).reshape(len(us), words)
    return codes, params, off


def unpack(codes, params, bits_u, d: int, G: int) -> np.ndarray:
    """Dequantize packed units back to rows (fp64): m16 + q * s16 (widths
    1..8), the stored fp16 row (16), zeros (0)."""
    codes = np.asarray(codes, dtype=np.uint64)
    bits_u = np.asarray(bits_u, dtype=np.int64)
    off = pack_layout(bits_u, d)
    units = bits_u.shape[0]
    out = np.empty((units, d), dtype=np.float64)
    shifts = np.arange(64, dtype=np.uint64)
    s16 = params[:, :, 0].view(np.float16).astype(np.float64)
    m16 = params[:, :, 1].view(np.float16).astype(np.float64)
    for u in range(units):
        b = int(bits_u[u])
        if b == 0:
            out[u] = 0.0
            continue
        if b == 16:
            out[u] = codes[off[u]:off[u + 1]].view(np.float16).astype(np.float64)
            continue
        words = codes[off[u]:off[u + 1]].reshape(b, d // 64)
        q = np.zeros(d, dtype=np.uint64)
        for t in range(b):
            bit = (words[t][:, None] >> shifts[None, :]) & np.uint64(1)
            q |= bit.reshape(d) << np.uint64(t)
        out[u] = np.repeat(m16[u], G) + q.astype(np.float64) * np.repeat(s16[u], G)
    return out
