"""CPU oracle for the token log-probability gather (test infrastructure only).

Only the tests, the smoke entry point and the benchmark's CPU-baseline leg
may import this module.

Section 3.1 defines the token log-probability as the result of one fixed,
deterministic logit processing followed by normalization; the reuse ratio
is exp(l_upd - l_roll).  The processing used here is a single temperature
multiply: x = logits * inv_temperature.  Then

    logp_t = x_t[y_t] - log sum_v exp(x_t[v])

evaluated in float64 from the exact bf16 logits.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from .attention import bf16_to_f64


def logprob_fp64(logits: np.ndarray, targets: np.ndarray, inv_temperature: float = 1.0,
                 rows: Optional[np.ndarray] = None) -> np.ndarray:
    """logits [T,V] (bf16 bits or float), targets [T] int -> logp [T] float64.

    ``inv_temperature`` is applied as the fp32 value the caller passes.
    With ``rows`` given, only those rows are evaluated.
    """
    idx = np.arange(logits.shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    it = float(np.float32(inv_temperature))
    out = np.empty(idx.size, dtype=np.float64)
    # one row at a time keeps memory at O(V) for any T
    for r, t in enumerate(idx):
        row = logits[t]
        x = (bf16_to_f64(row) if row.dtype == np.uint16 else np.asarray(row, dtype=np.float64)) * it
        m = x.max()
        lse = m + np.log(np.exp(x - m).sum())
        out[r] = x[int(targets[t])] - lse
    return out
