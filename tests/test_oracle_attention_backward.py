"""Pins of the attention-backward oracle (no GPU).

The oracle writes out the chain rule of the Section 3.2 attention; these
tests tie it to things other than itself: central finite differences of the
forward definition, torch's autograd through its own causal attention, and
identities the gradient must satisfy (keys' gradients sum to zero, a shift
of every value row leaves dQ and dK alone, a one-token sequence copies dO
into dV, identical keys give the uniform-weights closed form).
"""
import numpy as np
import pytest

import oracle
from paper_2609_35140_amd import inputs


def _case(lens, hq, hkv, d, tag, sigma=1.0):
    cu = inputs.cu_seqlens(lens)
    T = int(cu[-1])
    g = inputs.rng(70, tag)
    q = g.normal(0, sigma, size=(T, hq, d))
    k = g.normal(0, sigma, size=(T, hkv, d))
    v = g.normal(0, sigma, size=(T, hkv, d))
    do = g.normal(0, 1.0, size=(T, hq, d))
    return q, k, v, do, cu


def test_finite_differences():
    """Every gradient entry against a central difference of sum(dO * O)."""
    q, k, v, do, cu = _case([3, 0, 5], 4, 2, 6, 0)
    scale = 0.37
    dq, dk, dv = oracle.attention_backward_fp64(q, k, v, do, cu, scale)

    def loss(q_, k_, v_):
        o, _ = oracle.causal_attention_fp64(q_, k_, v_, cu, scale)
        return float(np.sum(o * do))

    h = 1e-6
    for x, grad in ((q, dq), (k, dk), (v, dv)):
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            x0 = x[idx]
            x[idx] = x0 + h
            up = loss(q, k, v)
            x[idx] = x0 - h
            dn = loss(q, k, v)
            x[idx] = x0
            fd[idx] = (up - dn) / (2 * h)
        assert np.max(np.abs(fd - grad)) < 1e-7, np.max(np.abs(fd - grad))


def test_matches_torch_autograd():
    """torch's causal scaled-dot-product attention, differentiated by autograd
    in float64 on the CPU, with K/V repeated per q head (GQA)."""
    torch = pytest.importorskip("torch")
    lens = [37, 1, 70, 0, 64]
    hq, hkv, d = 6, 2, 16
    cu = inputs.cu_seqlens(lens)
    T = int(cu[-1])
    qb = inputs.normal_bf16((T, hq, d), 1.0, 71, 0)
    kb = inputs.normal_bf16((T, hkv, d), 1.0, 71, 1)
    vb = inputs.normal_bf16((T, hkv, d), 1.0, 71, 2)
    db = inputs.normal_bf16((T, hq, d), 1.0, 71, 3)
    scale = oracle.default_scale(d)
    dq, dk, dv = oracle.attention_backward_fp64(qb, kb, vb, db, cu, scale)
    f = oracle.bf16_to_f64
    Q = torch.tensor(f(qb), requires_grad=True)
    K = torch.tensor(f(kb), requires_grad=True)
    V = torch.tensor(f(vb), requires_grad=True)
    dO = torch.tensor(f(db))
    g = hq // hkv
    outs = []
    for b in range(len(lens)):
        lo, hi = int(cu[b]), int(cu[b + 1])
        if hi == lo:
            continue
        qs = Q[lo:hi].transpose(0, 1)                                  # [Hq, L, d]
        ks = K[lo:hi].transpose(0, 1).repeat_interleave(g, dim=0)
        vs = V[lo:hi].transpose(0, 1).repeat_interleave(g, dim=0)
        o = torch.nn.functional.scaled_dot_product_attention(qs, ks, vs, is_causal=True, scale=scale)
        outs.append((o.transpose(0, 1) * dO[lo:hi]).sum())
    torch.stack(outs).sum().backward()
    for got, want in ((dq, Q.grad), (dk, K.grad), (dv, V.grad)):
        assert np.allclose(got, want.numpy(), rtol=1e-10, atol=1e-12)


def test_key_gradients_sum_to_zero():
    """Each row of dS sums to zero (sum_j P_ij dP_ij = D_i), so the keys' dK of
    one (sequence, kv head) sum to zero."""
    q, k, v, do, cu = _case([50, 1, 129], 4, 1, 8, 2)
    _, dk, _ = oracle.attention_backward_fp64(q, k, v, do, cu)
    _, sk, _ = oracle.backward_error_scales(q, k, v, do, cu)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        tot = dk[lo:hi].sum(axis=0)
        assert np.max(np.abs(tot)) <= 1e-12 * max(1.0, sk[lo:hi].sum())


def test_value_shift_leaves_dq_dk_and_dv():
    """O moves by c when every value row moves by c (rows of P sum to 1), and
    dP - D does not change: dQ, dK and dV stay put."""
    q, k, v, do, cu = _case([20, 33], 4, 2, 8, 3)
    a = oracle.attention_backward_fp64(q, k, v, do, cu)
    v2 = v.copy()
    shift = inputs.rng(72).normal(0, 3.0, size=(2, 2, 8))
    for b in range(2):
        v2[int(cu[b]):int(cu[b + 1])] += shift[b]
    b_ = oracle.attention_backward_fp64(q, k, v2, do, cu)
    for x, y in zip(a, b_):
        assert np.allclose(x, y, rtol=1e-9, atol=1e-11)


def test_single_token_sequences():
    """A one-token sequence has P = [1]: dV is the sum of its group's dO, and
    dQ, dK vanish."""
    q, k, v, do, cu = _case([1, 1, 1], 6, 2, 8, 4)
    dq, dk, dv = oracle.attention_backward_fp64(q, k, v, do, cu)
    assert np.max(np.abs(dq)) < 1e-14 and np.max(np.abs(dk)) < 1e-14
    want = do.reshape(3, 2, 3, 8).sum(axis=2)
    assert np.allclose(dv, want, rtol=0, atol=1e-15)


def test_identical_keys_uniform_weights():
    """All keys of a sequence equal: P_ij = 1/(i+1) for j <= i, so
    dV_j = sum_h sum_{i>=j} dO_i/(i+1), and dQ = 0 (its keys' weights dS_ij sum to 0)."""
    L, hq, d = 17, 2, 8
    q, k, v, do, cu = _case([L], hq, 1, d, 5)
    k[:] = k[0]
    dq, _, dv = oracle.attention_backward_fp64(q, k, v, do, cu)
    want = np.zeros((L, d))
    for j in range(L):
        for i in range(j, L):
            want[j] += do[i].sum(axis=0) / (i + 1)
    assert np.allclose(dv[:, 0], want, rtol=1e-12, atol=1e-13)
    assert np.max(np.abs(dq)) < 1e-12


def test_error_scales_bound_the_gradients():
    """Each magnitude dominates its gradient (triangle inequality)."""
    q, k, v, do, cu = _case([40, 7], 4, 2, 16, 6)
    g = oracle.attention_backward_fp64(q, k, v, do, cu)
    s = oracle.backward_error_scales(q, k, v, do, cu)
    for x, m in zip(g, s):
        assert np.all(np.abs(x) <= m * (1 + 1e-12) + 1e-15)


def test_dq_rows_match_full_gradient():
    lens = [30, 65]
    q, k, v, do, cu = _case(lens, 4, 2, 16, 7)
    dq, _, _ = oracle.attention_backward_fp64(q, k, v, do, cu)
    rows = [(0, 0), (29, 3), (30, 1), (94, 2), (60, 0)]
    got, mag = oracle.dq_rows_fp64(q, k, v, do, cu, rows, with_scale=True)
    sq, _, _ = oracle.backward_error_scales(q, k, v, do, cu)
    for r, (t, h) in enumerate(rows):
        assert np.allclose(got[r], dq[t, h], rtol=1e-12, atol=1e-14)
        assert np.allclose(mag[r], sq[t, h], rtol=1e-12, atol=1e-14)
