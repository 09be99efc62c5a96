"""LM-head logits -- TEST INFRASTRUCTURE ONLY (CPU oracle).

The logits the log-probability reads (Section 3.1: the same deterministic
logit processing in both regimes): z = hidden . weight^T, here in fp64 with
the library matrix product as the one step, then rounded to bf16 where the
GPU path stores bf16.  Shares no code with the GPU path.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_to_f64, round_to_bf16, to_bf16_bits
from .logprob import logprob_fp64


def logits_fp64(hidden_bits: np.ndarray, weight_bits: np.ndarray) -> np.ndarray:
    """hidden [T, H], weight [V, H] (bf16 bits) -> exact-as-fp64 logits [T, V]."""
    return bf16_to_f64(hidden_bits) @ bf16_to_f64(weight_bits).T


def logits_bf16(hidden_bits: np.ndarray, weight_bits: np.ndarray) -> np.ndarray:
    """The fp64 logits rounded to bf16 (bits)."""
    return to_bf16_bits(logits_fp64(hidden_bits, weight_bits))


def abs_dot(hidden_bits: np.ndarray, weight_bits: np.ndarray) -> np.ndarray:
    """sum_k |h_k w_k| per logit: the scale of fp32 accumulation error."""
    return np.abs(bf16_to_f64(hidden_bits)) @ np.abs(bf16_to_f64(weight_bits)).T


def lm_head_logprob_fp64(hidden_bits: np.ndarray, weight_bits: np.ndarray, targets: np.ndarray,
                         inv_temperature: float = 1.0, fp32_slack: float = 2e-5):
    """The fused LM head + log-probability, and how far an fp32 evaluation may be from it.

    Reference: logp = x[y] - logsumexp(x) in fp64 over x = bf16(z) * inv_temperature,
    z = hidden . weight^T exact (Section 3.1: one deterministic logit
    processing, then normalization).

    Bound: an evaluation that accumulates z in fp32 (error at most
    e = H * 2^-24 * sum_k |h_k w_k| per logit) and then rounds to bf16 may
    store, for each logit, any bf16 value in [bf16(z - e), bf16(z + e)]
    (rounding is monotone); with d_v the largest such move of x_v,
    |dlogp| <= d_y + log(sum_v p_v exp(d_v)) (p the reference softmax), plus
    ``fp32_slack`` for the fp32 log-softmax itself.
    Returns (logp [T] float64, bound [T] float64).
    """
    H = hidden_bits.shape[1]
    it = float(np.float32(inv_temperature))
    z = logits_fp64(hidden_bits, weight_bits)
    e = H * 2.0 ** -24 * abs_dot(hidden_bits, weight_bits)
    zb = round_to_bf16(z.astype(np.float32)).astype(np.float64)
    lo = round_to_bf16((z - e).astype(np.float32)).astype(np.float64)
    hi = round_to_bf16((z + e).astype(np.float32)).astype(np.float64)
    d = np.maximum(np.abs(hi - zb), np.abs(zb - lo)) * it
    logp = logprob_fp64(zb, targets, inv_temperature)
    x = zb * it
    p = np.exp(x - x.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    rows = np.arange(z.shape[0])
    bound = d[rows, np.asarray(targets, dtype=np.int64)] + np.log((p * np.exp(d)).sum(axis=1)) + fp32_slack
    return logp, bound
