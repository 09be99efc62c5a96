"""Attention backward -- TEST INFRASTRUCTURE ONLY (CPU oracle).

The gradient of the causal GQA attention of Section 3.2 (scores Q K^T,
weights P = softmax, output P V), which the policy update runs after its
forward pass over every prompt+response trajectory (Section 6 Q2 times the
update's forward and backward once per trajectory).  The paper gives no
formula for it; it is fixed by the forward's definition and the chain rule.
For one (sequence, q head), with S = scale * Q K^T masked causally,
P = softmax(S) row-wise, O = P V and an upstream gradient dO:

    dV = P^T dO
    dP = dO V^T
    dS = P * (dP - D),   D_i = sum_j P_ij dP_ij = dO_i . O_i
    dQ = scale * dS K
    dK = scale * dS^T Q

and the q heads of a group, which read the same K and V, add their dK and
dV.  Everything is float64 from the exact values of the inputs (bf16 bit
patterns as handed to the GPU, or float arrays).  Shares no code with the
GPU path.
"""
from __future__ import annotations

from typing import Iterable, Optional, Sequence, Tuple

import numpy as np

from .attention import _as_f64, default_scale


def _softmax_causal(qh: np.ndarray, kh: np.ndarray, scale: float) -> np.ndarray:
    """P of one (sequence, head): row i is the softmax of scale * q_i . k_j over j <= i."""
    L = qh.shape[0]
    s = (qh @ kh.T) * scale
    s[np.triu(np.ones((L, L), dtype=bool), k=1)] = -np.inf
    e = np.exp(s - s.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def _one_head(qh, kh, vh, doh, scale):
    """Gradients of one (sequence, q head).  Returns (dq, dk, dv, p, ds)."""
    p = _softmax_causal(qh, kh, scale)
    o = p @ vh
    dv = p.T @ doh
    dp = doh @ vh.T
    dd = np.sum(doh * o, axis=1, keepdims=True)   # D_i = dO_i . O_i
    ds = p * (dp - dd)
    dq = scale * (ds @ kh)
    dk = scale * (ds.T @ qh)
    return dq, dk, dv, p, ds


def _setup(q, k, v, dout, scale):
    qf, kf, vf, df = _as_f64(q), _as_f64(k), _as_f64(v), _as_f64(dout)
    hq, hkv = qf.shape[1], kf.shape[1]
    if hq % hkv:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    if scale is None:
        scale = default_scale(qf.shape[2])
    return qf, kf, vf, df, hq // hkv, scale


def attention_backward_fp64(q: np.ndarray, k: np.ndarray, v: np.ndarray, dout: np.ndarray,
                            cu_seqlens: Sequence[int], scale: Optional[float] = None
                            ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Gradients of causal GQA attention over a packed varlen batch.

    q, dout [T,Hq,d]; k, v [T,Hkv,d]; cu_seqlens [B+1] (sequence-relative
    causal positions, as in the forward).  Returns (dq [T,Hq,d],
    dk [T,Hkv,d], dv [T,Hkv,d]) float64.
    """
    qf, kf, vf, df, g, scale = _setup(q, k, v, dout, scale)
    hq = qf.shape[1]
    dq = np.zeros_like(qf)
    dk = np.zeros_like(kf)
    dv = np.zeros_like(vf)
    cu = [int(x) for x in cu_seqlens]
    for b in range(len(cu) - 1):
        lo, hi = cu[b], cu[b + 1]
        if hi <= lo:
            continue
        for h in range(hq):
            kvh = h // g
            gq, gk, gv, _, _ = _one_head(qf[lo:hi, h], kf[lo:hi, kvh], vf[lo:hi, kvh], df[lo:hi, h], scale)
            dq[lo:hi, h] = gq
            dk[lo:hi, kvh] += gk
            dv[lo:hi, kvh] += gv
    return dq, dk, dv


def backward_error_scales(q: np.ndarray, k: np.ndarray, v: np.ndarray, dout: np.ndarray,
                          cu_seqlens: Sequence[int], scale: Optional[float] = None
                          ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Magnitudes that bound the rounding error of a bf16/fp32 evaluation.

    With a_i = sum_d |dO_id| (P |V|)_id (the size of D_i's terms, which also
    bounds how far a rounded forward output moves D_i), returns
      sv[j] = sum_h sum_i P_ij |dO_i|                      (scale of dV)
      sq[i] = scale * sum_j (|dS_ij| + a_i P_ij) |K_j|     (scale of dQ)
      sk[j] = scale * sum_h sum_i (|dS_ij| + a_i P_ij) |Q_i|   (scale of dK)
    each of the gradient's shape.  Each bounds its gradient's magnitude.
    """
    qf, kf, vf, df, g, scale = _setup(q, k, v, dout, scale)
    hq = qf.shape[1]
    sq = np.zeros_like(qf)
    sk = np.zeros_like(kf)
    sv = np.zeros_like(vf)
    cu = [int(x) for x in cu_seqlens]
    for b in range(len(cu) - 1):
        lo, hi = cu[b], cu[b + 1]
        if hi <= lo:
            continue
        for h in range(hq):
            kvh = h // g
            qh, kh, vh, doh = qf[lo:hi, h], kf[lo:hi, kvh], vf[lo:hi, kvh], df[lo:hi, h]
            _, _, _, p, ds = _one_head(qh, kh, vh, doh, scale)
            a = np.sum(np.abs(doh) * (p @ np.abs(vh)), axis=1, keepdims=True)
            w = np.abs(ds) + a * p
            sq[lo:hi, h] = scale * (w @ np.abs(kh))
            sk[lo:hi, kvh] += scale * (w.T @ np.abs(qh))
            sv[lo:hi, kvh] += p.T @ np.abs(doh)
    return sq, sk, sv


def dq_rows_fp64(q: np.ndarray, k: np.ndarray, v: np.ndarray, dout: np.ndarray, cu_seqlens: Sequence[int],
                 rows: Iterable[Tuple[int, int]], scale: Optional[float] = None, with_scale: bool = False):
    """dQ at chosen (packed token index, q head) rows, each from its own row's
    data and its sequence's keys and values: dQ_i = scale sum_j P_ij (dO_i.V_j - dO_i.O_i) K_j.

    With ``with_scale`` also returns the rows' error magnitudes (the sq of
    backward_error_scales, from the same row data)."""
    rows = list(rows)
    hq, hkv, d = q.shape[1], k.shape[1], q.shape[2]
    g = hq // hkv
    if scale is None:
        scale = default_scale(d)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    out = np.zeros((len(rows), d), dtype=np.float64)
    mag = np.zeros((len(rows), d), dtype=np.float64)
    for r, (t, h) in enumerate(rows):
        b = int(np.searchsorted(cu, t, side="right") - 1)
        lo = int(cu[b])
        qi = _as_f64(q[t, h])
        doi = _as_f64(dout[t, h])
        kj = _as_f64(k[lo:t + 1, h // g])
        vj = _as_f64(v[lo:t + 1, h // g])
        s = (kj @ qi) * scale
        e = np.exp(s - s.max())
        p = e / e.sum()
        dp = vj @ doi
        ds = p * (dp - np.dot(doi, p @ vj))
        out[r] = scale * (ds @ kj)
        if with_scale:
            a = np.dot(np.abs(doi), p @ np.abs(vj))
            mag[r] = scale * ((np.abs(ds) + a * p) @ np.abs(kj))
    return (out, mag) if with_scale else out
