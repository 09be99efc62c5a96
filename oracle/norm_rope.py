"""Q/K RMSNorm + NeoX rotary embedding -- TEST INFRASTRUCTURE ONLY (CPU oracle).

The operators applied to queries and keys before attention in both regimes
(Section 6 Q3 lists Q RMSNorm, K RMSNorm and NeoX RoPE among the operators
whose full-sequence and token-wise outputs must agree bit for bit).  The
paper gives no formulas; this follows the usual definitions with the
rounding points the GPU path documents:

  r   = 1 / sqrt(mean_i x_i^2 + eps)
  y_i = bf16(w_i * bf16(x_i * r))
  out_i = bf16(y_i cos(a) - y_{i+d/2} sin(a)),  out_{i+d/2} = bf16(y_{i+d/2} cos(a) + y_i sin(a))
  a   = pos * theta^(-2i/d),  cos/sin rounded to fp32 (the rotary table)

Everything between the rounding points is evaluated in fp64.  Shares no code
with the GPU path.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_to_f64, round_to_bf16, to_bf16_bits


def rope_table(max_position: int, head_dim: int, theta: float) -> np.ndarray:
    """[max_position, head_dim/2, 2] float32: (cos, sin) of the fp64 angle, each rounded to fp32."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.power(np.float64(theta), -2.0 * i / head_dim)
    ang = np.arange(max_position, dtype=np.float64)[:, None] * inv_freq[None, :]
    out = np.empty((max_position, head_dim // 2, 2), dtype=np.float32)
    out[..., 0] = np.cos(ang).astype(np.float32)
    out[..., 1] = np.sin(ang).astype(np.float32)
    return out


def rms_norm_bf16(x_bits: np.ndarray, w_bits: np.ndarray, eps: float) -> np.ndarray:
    """y = bf16(w * bf16(x / sqrt(mean(x^2) + eps))) over the last axis, as float64 values."""
    x = bf16_to_f64(x_bits)
    w = bf16_to_f64(w_bits)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    n = round_to_bf16(x * r).astype(np.float64)
    return round_to_bf16(w * n).astype(np.float64)


def rope_neox(y: np.ndarray, positions: np.ndarray, cos_sin: np.ndarray) -> np.ndarray:
    """Rotate the halves (i, i + d/2) of y [T, H, d] by the table's angle for each token; bf16 bits."""
    d = y.shape[-1]
    cs = cos_sin[np.asarray(positions)].astype(np.float64)   # [T, d/2, 2]
    c = cs[:, None, :, 0]
    s = cs[:, None, :, 1]
    y1, y2 = y[..., : d // 2], y[..., d // 2:]
    out = np.concatenate([y1 * c - y2 * s, y2 * c + y1 * s], axis=-1)
    return to_bf16_bits(out)


def qk_norm_rope(x_bits: np.ndarray, positions, w_bits: np.ndarray, eps: float, cos_sin: np.ndarray) -> np.ndarray:
    """x [T, H, d] bf16 bits -> normalized, rotated [T, H, d] bf16 bits."""
    return rope_neox(rms_norm_bf16(x_bits, w_bits, eps), np.asarray(positions), cos_sin)
