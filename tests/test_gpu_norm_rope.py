"""GPU Q/K RMSNorm + NeoX RoPE: oracle parity, and the same bits for a row
whether it is computed in a full-sequence call or token by token
(Section 6 Q3's prescribed checks for these operators)."""
import numpy as np
import pytest

import oracle
from paper_2609_35140_amd import inputs

pytestmark = pytest.mark.gpu
gu = pytest.importorskip("gpu_util")


@pytest.fixture(scope="module")
def ua():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35140_amd import uattn
    uattn.lib()
    return uattn


def _ulps_bf16(a_bits, b_bits):
    """Distance in bf16 units of the larger magnitude (0 for equal bits)."""
    a = oracle.bf16_to_f64(a_bits)
    b = oracle.bf16_to_f64(b_bits)
    mag = np.maximum(np.abs(a), np.abs(b))
    ulp = np.where(mag > 0, 2.0 ** (np.floor(np.log2(np.where(mag > 0, mag, 1.0))) - 7), 2.0 ** -133)
    return np.where(a_bits == b_bits, 0.0, np.abs(a - b) / ulp)


@pytest.mark.parametrize("max_pos,d,theta", [(4096, 128, 1e6), (33000, 64, 10000.0), (131072, 128, 5e5)])
def test_rope_cache_matches_oracle(ua, max_pos, d, theta):
    got = ua.rope_cache(max_pos, d, theta).cpu().numpy()
    want = oracle.rope_table(max_pos, d, theta)
    # both sides round cos/sin of an fp64 angle to fp32; the angle p * theta^(-2i/d)
    # is itself uncertain by a few fp64 ulps of p (different pow/cos implementations),
    # which near a zero of cos or sin can exceed one fp32 ulp of the tiny result
    err = np.abs(got.astype(np.float64) - want.astype(np.float64))
    bound = 2.0 ** -24 + np.arange(max_pos, dtype=np.float64)[:, None, None] * 2.0 ** -50
    exact = np.mean(got.view(np.int32) == want.view(np.int32))
    print(f"rope table {max_pos}x{d}: {exact:.6f} exact, max abs err {err.max():.3g}", flush=True)
    assert np.all(err <= bound) and exact > 0.999


@pytest.mark.parametrize("T,hq,hkv,d,sigma,eps", [(300, 32, 8, 128, 1.0, 1e-6), (77, 10, 2, 64, 3.0, 1e-5),
                                                  (1, 64, 8, 128, 0.5, 1e-6)])
def test_matches_oracle(ua, T, hq, hkv, d, sigma, eps):
    import torch
    q = inputs.normal_bf16((T, hq, d), sigma, 74, T)
    k = inputs.normal_bf16((T, hkv, d), sigma, 75, T)
    qw = inputs.normal_bf16((d,), 1.0, 76, T)
    kw = inputs.normal_bf16((d,), 1.0, 77, T)
    pos = inputs.rng(78, T).integers(0, 40000, size=T).astype(np.int32)
    cs = ua.rope_cache(40000, d, 1e6)
    qo, ko = ua.qk_norm_rope(gu.dev(q), gu.dev(k), gu.dev_i32(pos), gu.dev(qw), gu.dev(kw), cs, eps=eps)
    cs_host = cs.cpu().numpy()            # the table itself is checked against the oracle above
    for got, x, w in ((qo, q, qw), (ko, k, kw)):
        want = oracle.qk_norm_rope(x, pos, w, eps, cs_host)
        u = _ulps_bf16(gu.host_bits(got), want)
        print(f"T={T} d={d}: {np.mean(u == 0):.5f} exact, max {u.max():.2f} bf16 units", flush=True)
        # the GPU evaluates x * r and the rotation in fp32, the oracle in fp64: an
        # intermediate bf16 rounding (x * r) can land one unit apart, which moves
        # the rotated value by at most one unit (|cos|, |sin| <= 1) before the
        # final rounding adds at most one more
        assert u.max() <= 2.0 and np.mean(u == 0) > 0.999
    torch.cuda.synchronize()


def test_full_sequence_and_token_wise_rows_are_identical(ua):
    """One call over a whole pack vs one call per decode step (a token of each
    sequence, in shuffled order) and in-place: the same bits for every row."""
    import torch
    T, hq, hkv, d = 512, 16, 4, 128
    q = gu.dev(inputs.normal_bf16((T, hq, d), 1.0, 79))
    k = gu.dev(inputs.normal_bf16((T, hkv, d), 1.0, 80))
    qw = gu.dev(inputs.normal_bf16((d,), 1.0, 81))
    kw = gu.dev(inputs.normal_bf16((d,), 1.0, 82))
    pos_h = np.concatenate([np.arange(200), np.arange(312)]).astype(np.int32)   # two sequences
    pos = gu.dev_i32(pos_h)
    cs = ua.rope_cache(4096, d, 1e6)
    qf, kf = ua.qk_norm_rope(q, k, pos, qw, kw, cs)
    g = inputs.rng(83)
    for step in range(40):
        idx = g.permutation(T)[: 1 + step % 9]
        it = torch.from_numpy(idx).cuda()
        qs, ks = ua.qk_norm_rope(q[it].contiguous(), k[it].contiguous(), pos[it].contiguous(), qw, kw, cs)
        assert torch.equal(qs.view(torch.int16), qf[it].view(torch.int16))
        assert torch.equal(ks.view(torch.int16), kf[it].view(torch.int16))
    qi, ki = q.clone(), k.clone()
    ua.qk_norm_rope(qi, ki, pos, qw, kw, cs, q_out=qi, k_out=ki)
    assert torch.equal(qi.view(torch.int16), qf.view(torch.int16)) and torch.equal(ki.view(torch.int16), kf.view(torch.int16))


def test_position_outside_the_table_gives_nan_rows(ua):
    import torch
    d = 64
    q = gu.dev(inputs.normal_bf16((3, 2, d), 1.0, 84))
    k = gu.dev(inputs.normal_bf16((3, 1, d), 1.0, 85))
    w = gu.dev(np.full(d, 0x3F80, dtype=np.uint16))
    cs = ua.rope_cache(16, d, 1e4)
    qo, ko = ua.qk_norm_rope(q, k, gu.dev_i32([3, 16, -1]), w, w, cs)
    assert not torch.isnan(qo[0]).any() and torch.isnan(qo[1]).all() and torch.isnan(ko[2]).all()
