"""INT4 group quantization of the linear weights (TEST INFRASTRUCTURE ONLY).

The paper's models are GPTQ-INT4 (Sec. 4.1, "Models"); GPTQ needs calibration
data, so round-to-nearest per group stands in for it.  The format:

    groups of G = 128 consecutive input columns of one output row;
    a   = max |w| over the group (w: the bf16 weight, exact in float32);
    s   = bf16( float32(a) / 7 )        float32 division, then rounding to
                                        bfloat16 (nearest, ties to even);
    q   = clamp( rint( float32(w) / s ), -8, 7 )   float32 division, rint
                                        rounding halves to even; q = 0 where s = 0;
    effective weight = q * s            (exact: 4-bit integer times bf16 scale).

The quantizer's arithmetic is part of the format (float32 steps as written,
the way the fixed-point sampler's is), so it is written here in float32; the
model that uses the effective weights is the float64 oracle of model.py.
"""
from __future__ import annotations

import numpy as np

GROUP = 128


def _f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); bit patterns."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def _bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def quantize_int4(w_bits: np.ndarray, group: int = GROUP):
    """Quantize a bf16 matrix [N, K] (bit patterns).

    Returns (q int8 [N, K] in [-8, 7], s_bits uint16 [N, ceil(K/group)])."""
    w_bits = np.asarray(w_bits, dtype=np.uint16)
    N, K = w_bits.shape
    w = _bf16_bits_to_f32(w_bits)
    G = (K + group - 1) // group
    s_bits = np.zeros((N, G), np.uint16)
    q = np.zeros((N, K), np.int8)
    for g in range(G):
        blk = w[:, g * group:(g + 1) * group]
        a = np.max(np.abs(blk), axis=1).astype(np.float32)
        sb = _f32_to_bf16_bits(a / np.float32(7.0))
        s = _bf16_bits_to_f32(sb)
        with np.errstate(divide="ignore", invalid="ignore"):
            t = np.rint(blk / s[:, None])
        t = np.where(s[:, None] == 0, 0.0, t)
        q[:, g * group:(g + 1) * group] = np.clip(t, -8, 7).astype(np.int8)
        s_bits[:, g] = sb
    return q, s_bits


def dequantize_int4(q: np.ndarray, s_bits: np.ndarray, group: int = GROUP) -> np.ndarray:
    """Effective weights q * s as float64 [N, K] (exact)."""
    q = np.asarray(q, dtype=np.int8)
    s = _bf16_bits_to_f32(s_bits).astype(np.float64)
    N, K = q.shape
    return q.astype(np.float64) * np.repeat(s, group, axis=1)[:, :K]


LINEAR = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def int4_model_weights(weights: dict, n_layers: int | None = None) -> dict:
    """The weights of the INT4 model: every layer's linear matrices replaced by
    their float64 effective weights; embedding, gains and the LM head stay bf16."""
    L = len(weights["layers"]) if n_layers is None else n_layers
    out = {k: v for k, v in weights.items() if k != "layers"}
    out["layers"] = []
    for l in range(L):
        lw = dict(weights["layers"][l])
        for name in LINEAR:
            lw[name] = dequantize_int4(*quantize_int4(lw[name]))
        out["layers"].append(lw)
    return out
