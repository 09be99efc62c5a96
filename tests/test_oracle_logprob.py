"""The fp64 log-prob oracle against closed forms, a library routine and brute force."""
import math

import numpy as np
import pytest

import oracle
from paper_2609_35140_amd import inputs


def test_constant_logits_give_minus_log_v():
    V = 1000
    logits = np.zeros((3, V), dtype=np.float64) + 2.5
    tg = np.array([0, 17, 999])
    lp = oracle.logprob_fp64(logits, tg)
    assert np.max(np.abs(lp + math.log(V))) < 1e-12


def test_probabilities_sum_to_one():
    lg = inputs.logits_bf16(4, 257, 2.0)
    V = lg.shape[1]
    for r in range(4):
        lp = oracle.logprob_fp64(np.repeat(lg[r:r + 1], V, axis=0), np.arange(V))
        assert abs(math.fsum(np.exp(lp)) - 1.0) < 1e-12


def test_against_scipy_log_softmax():
    from scipy.special import log_softmax
    lg = inputs.logits_bf16(16, 5000, 2.0)
    tg = inputs.targets(16, 5000)
    for it in [1.0, 0.7]:
        lp = oracle.logprob_fp64(lg, tg, inv_temperature=it)
        x = oracle.bf16_to_f64(lg) * float(np.float32(it))
        ref = log_softmax(x, axis=1)[np.arange(16), tg]
        assert np.max(np.abs(lp - ref)) < 1e-12


def test_bruteforce_mpmath():
    import mpmath as mp
    mp.mp.dps = 40
    lg = inputs.logits_bf16(2, 50, 3.0)
    tg = np.array([3, 49])
    lp = oracle.logprob_fp64(lg, tg, inv_temperature=0.5)
    x = oracle.bf16_to_f64(lg)
    for r in range(2):
        z = mp.fsum(mp.exp(mp.mpf(float(v)) * mp.mpf(0.5)) for v in x[r])
        ref = mp.mpf(float(x[r, tg[r]])) * mp.mpf(0.5) - mp.log(z)
        assert abs(float(ref) - lp[r]) < 1e-12


def test_rows_subset_and_row_independence():
    lg = inputs.logits_bf16(10, 300, 2.0)
    tg = inputs.targets(10, 300)
    full = oracle.logprob_fp64(lg, tg)
    sub = oracle.logprob_fp64(lg, tg, rows=np.array([7, 2]))
    assert sub[0] == full[7] and sub[1] == full[2]
    # reversing the batch reverses the results exactly
    rev = oracle.logprob_fp64(lg[::-1].copy(), tg[::-1].copy())
    assert np.array_equal(rev[::-1], full)


@pytest.mark.parametrize("shift", [-30.0, 0.0, 45.0])
def test_shift_invariance(shift):
    """log-softmax is invariant to adding a constant to every logit of a row."""
    x = np.random.default_rng(0).standard_normal((3, 64))
    tg = np.array([1, 2, 3])
    a = oracle.logprob_fp64(x, tg)
    b = oracle.logprob_fp64(x + shift, tg)
    assert np.max(np.abs(a - b)) < 1e-12
