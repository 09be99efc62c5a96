"""Pins of the oracle's Q/K RMSNorm + NeoX RoPE (no GPU).

Against textbook values of the rotary table, the rotation written with
complex numbers (the halves as real and imaginary parts), position 0 as the
identity, exact normalization cases and scale invariance.
"""
import numpy as np

import oracle
from paper_2609_35140_amd import inputs


def test_rope_table_closed_forms():
    t = oracle.rope_table(201, 128, 10000.0)
    assert np.array_equal(t[0, :, 0], np.ones(64, dtype=np.float32))
    assert np.array_equal(t[0, :, 1], np.zeros(64, dtype=np.float32))
    # i = 0: inv_freq 1, angle = position; i = 32 (= d/4): inv_freq = 10000^-0.5 = 0.01
    assert t[1, 0, 0] == np.float32(0.5403023058681398) and t[1, 0, 1] == np.float32(0.8414709848078965)
    assert t[100, 32, 0] == np.float32(0.5403023058681398) and t[100, 32, 1] == np.float32(0.8414709848078965)
    assert t[200, 32, 0] == np.float32(-0.4161468365471424) and t[200, 32, 1] == np.float32(0.9092974268256817)
    assert np.allclose(t[..., 0].astype(np.float64) ** 2 + t[..., 1].astype(np.float64) ** 2, 1.0, atol=1e-6)


def _x(T, H, d, sigma=1.0, key=0):
    return inputs.normal_bf16((T, H, d), sigma, 70, key)


def test_rotation_is_complex_multiplication_of_the_halves():
    T, H, d = 7, 3, 64
    y = oracle.bf16_to_f64(_x(T, H, d))
    pos = np.array([0, 1, 5, 77, 1000, 4095, 31999])
    cs = oracle.rope_table(32000, d, 1e6)
    z = (y[..., : d // 2] + 1j * y[..., d // 2:]) * (cs[pos, :, 0] + 1j * cs[pos, :, 1]).astype(np.complex128)[:, None, :]
    want = inputs.f32_to_bf16_bits(np.concatenate([z.real, z.imag], axis=-1).astype(np.float32))
    assert np.array_equal(oracle.rope_neox(y, pos, cs), want)


def test_position_zero_is_the_normalization_alone():
    x = _x(4, 2, 128, key=1)
    w = inputs.normal_bf16((128,), 1.0, 71)
    cs = oracle.rope_table(8, 128, 10000.0)
    out = oracle.qk_norm_rope(x, np.zeros(4, dtype=np.int64), w, 1e-6, cs)
    assert np.array_equal(out, oracle.to_bf16_bits(oracle.rms_norm_bf16(x, w, 1e-6)))


def test_rms_norm_exact_cases():
    one = np.full(64, 0x3F80, dtype=np.uint16)                   # weight 1.0
    c = inputs.f32_to_bf16_bits(np.array([[-3.0] * 64, [0.5] * 64, [2.0 ** -20] * 64], dtype=np.float32))
    y = oracle.rms_norm_bf16(c, one, 0.0)
    assert np.array_equal(y, np.array([[-1.0] * 64, [1.0] * 64, [1.0] * 64]))
    # with eps = 0 the normalization ignores a power-of-two scale exactly
    x = _x(5, 1, 64, key=2)
    x2 = inputs.f32_to_bf16_bits(oracle.bf16_to_f64(x).astype(np.float32) * np.float32(4.0))
    assert np.array_equal(oracle.rms_norm_bf16(x, one, 0.0), oracle.rms_norm_bf16(x2, one, 0.0))
    # unit weights: the mean square of the result is 1 up to bf16 rounding
    ms = np.mean(oracle.rms_norm_bf16(_x(50, 1, 128, key=3), np.full(128, 0x3F80, dtype=np.uint16), 1e-6) ** 2, axis=-1)
    assert np.all(np.abs(ms - 1.0) < 2 ** -7)


def test_rotation_keeps_pair_norms():
    y = oracle.rms_norm_bf16(_x(16, 4, 128, key=4), inputs.normal_bf16((128,), 1.0, 72), 1e-6)
    cs = oracle.rope_table(40000, 128, 1e6)
    pos = inputs.rng(73).integers(0, 40000, size=16)
    o = oracle.bf16_to_f64(oracle.rope_neox(y, pos, cs))
    n_in = y[..., :64] ** 2 + y[..., 64:] ** 2
    n_out = o[..., :64] ** 2 + o[..., 64:] ** 2
    assert np.all(np.abs(np.sqrt(n_out) - np.sqrt(n_in)) <= 2 ** -7 * np.sqrt(n_in) + 1e-30)
