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
