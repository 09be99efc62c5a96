"""Pins of the oracle's LM-head logits (no GPU): a brute-force dot product on
a tiny case, selection weights that copy hidden entries exactly, and exact
power-of-two scaling."""
import numpy as np

import oracle
from paper_2609_35140_amd import inputs


def test_brute_force_dot_products():
    h = inputs.normal_bf16((3, 64), 1.0, 90, 0)
    w = inputs.normal_bf16((5, 64), 1.0, 90, 1)
    hf, wf = oracle.bf16_to_f64(h), oracle.bf16_to_f64(w)
    want = np.array([[sum(float(hf[t, k]) * float(wf[v, k]) for k in range(64)) for v in range(5)] for t in range(3)])
    assert np.allclose(oracle.logits_fp64(h, w), want, rtol=1e-12, atol=1e-12)


def test_selection_weights_copy_hidden_entries():
    h = inputs.normal_bf16((4, 128), 2.0, 91)
    sel = np.array([5, 0, 127, 64, 5])
    w = np.zeros((5, 128), dtype=np.uint16)
    w[np.arange(5), sel] = 0x3F80                      # 1.0
    w[4, 6] = 0xC000                                   # row 4 = h[5] - 2 h[6]
    got = oracle.logits_bf16(h, w)
    assert np.array_equal(got[:, :4], h[:, sel[:4]])
    want4 = oracle.bf16_to_f64(h[:, 5]) - 2.0 * oracle.bf16_to_f64(h[:, 6])
    assert np.array_equal(got[:, 4], oracle.to_bf16_bits(want4))


def test_power_of_two_scaling_is_exact():
    h = inputs.normal_bf16((6, 64), 1.0, 92)
    w = inputs.normal_bf16((7, 64), 1.0, 93)
    w4 = inputs.f32_to_bf16_bits(oracle.bf16_to_f64(w).astype(np.float32) * np.float32(0.25))
    assert np.array_equal(oracle.logits_fp64(h, w4), oracle.logits_fp64(h, w) * 0.25)


def _fp32_blocked_logits(h, w, block):
    """An fp32 evaluation of the logits in a different order from any above:
    partial dot products of `block` hidden entries in fp32, summed in fp32."""
    hf = oracle.bf16_to_f64(h).astype(np.float32)
    wf = oracle.bf16_to_f64(w).astype(np.float32)
    z = np.zeros((h.shape[0], w.shape[0]), dtype=np.float32)
    for k0 in range(0, h.shape[1], block):
        z = (z + (hf[:, k0:k0 + block] @ wf[:, k0:k0 + block].T).astype(np.float32)).astype(np.float32)
    return z


def test_fused_logprob_reference_and_bound_cover_fp32_evaluations():
    # any fp32-accumulated, bf16-rounded evaluation of the logits lands inside the bound
    T, V, H = 24, 700, 1024
    h = inputs.normal_bf16((T, H), 1.0, 94, 1)
    w = inputs.normal_bf16((V, H), float(2.0 / np.sqrt(H)), 95, 1)
    tg = inputs.targets(T, V, tag=3)
    for it in (1.0, 0.7):
        ref, bound = oracle.lm_head_logprob_fp64(h, w, tg, it)
        # the reference is the log-softmax of the correctly rounded logits
        assert np.array_equal(ref, oracle.logprob_fp64(oracle.logits_bf16(h, w), tg, it))
        for block in (1, 32, 256, H):
            alt = oracle.to_bf16_bits(_fp32_blocked_logits(h, w, block))
            lp = oracle.logprob_fp64(alt, tg, it)
            assert np.all(np.abs(lp - ref) <= bound), (it, block, float(np.max(np.abs(lp - ref) - bound)))
        assert np.all(bound < 0.2) and np.median(bound) < 0.05


def test_fused_logprob_bound_is_the_slack_when_logits_are_exact():
    # small integers (|z| <= 64): the logits are bf16 values, so the bound reduces to the
    # fp32 slack of the log-softmax itself plus the a-priori accumulation bound near z = 0
    g = np.random.default_rng(5)
    T, V, H = 6, 300, 64
    hi = g.integers(-1, 2, size=(T, H)).astype(np.float32)
    wi = g.integers(-1, 2, size=(V, H)).astype(np.float32)
    h, w = inputs.f32_to_bf16_bits(hi), inputs.f32_to_bf16_bits(wi)
    tg = g.integers(0, V, size=T)
    ref, bound = oracle.lm_head_logprob_fp64(h, w, tg, 0.125)
    x = (hi @ wi.T).astype(np.float64) * 0.125
    want = x[np.arange(T), tg] - (x.max(1) + np.log(np.exp(x - x.max(1, keepdims=True)).sum(1)))
    assert np.allclose(ref, want, rtol=0, atol=1e-12)
    e = 64 * 2.0 ** -24 * oracle.abs_dot(h, w)
    assert np.all(bound <= 2e-5 + 0.125 * 1.01 * e.max())


def test_fused_logprob_bound_catches_a_shifted_target_logit():
    # a mistake of one bf16 step in the target logit where the logits are exact is outside the bound
    g = np.random.default_rng(6)
    T, V, H = 4, 200, 64
    hi = g.integers(-3, 4, size=(T, H)).astype(np.float32)
    wi = g.integers(-2, 3, size=(V, H)).astype(np.float32)
    h, w = inputs.f32_to_bf16_bits(hi), inputs.f32_to_bf16_bits(wi)
    tg = g.integers(0, V, size=T)
    ref, bound = oracle.lm_head_logprob_fp64(h, w, tg)
    z = oracle.logits_fp64(h, w)
    z[np.arange(T), tg] += np.maximum(np.abs(z[np.arange(T), tg]), 1.0) * 2.0 ** -7
    bad = oracle.logprob_fp64(oracle.to_bf16_bits(z), tg)
    assert np.all(np.abs(bad - ref) > bound)
