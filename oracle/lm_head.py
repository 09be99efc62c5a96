"""LM-head logits -- TEST INFRASTRUCTURE ONLY (CPU oracle).

The logits the log-probability reads (Section 3.1: the same deterministic
logit processing in both regimes): z = hidden . weight^T, here in fp64 with
the library matrix product as the one step, then rounded to bf16 where the
GPU path stores bf16.  Shares no code with the GPU path.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_to_f64, to_bf16_bits


def logits_fp64(hidden_bits: np.ndarray, weight_bits: np.ndarray) -> np.ndarray:
    """hidden [T, H], weight [V, H] (bf16 bits) -> exact-as-fp64 logits [T, V]."""
    return bf16_to_f64(hidden_bits) @ bf16_to_f64(weight_bits).T


def logits_bf16(hidden_bits: np.ndarray, weight_bits: np.ndarray) -> np.ndarray:
    """The fp64 logits rounded to bf16 (bits)."""
    return to_bf16_bits(logits_fp64(hidden_bits, weight_bits))


def abs_dot(hidden_bits: np.ndarray, weight_bits: np.ndarray) -> np.ndarray:
    """sum_k |h_k w_k| per logit: the scale of fp32 accumulation error."""
    return np.abs(bf16_to_f64(hidden_bits)) @ np.abs(bf16_to_f64(weight_bits)).T
