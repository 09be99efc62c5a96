"""Checks that pin the CPU oracle to facts other than itself.

Each check takes the oracle entry point as an argument so that the same
check can be run against the real oracle (it must pass) and against copies
with a planted mistake (at least one check must fail for each).

What pins what:
  * brute force -- an independent high-precision (mpmath, 50 digits) loop
    over (query, key) pairs on tiny inputs;
  * a library routine -- torch's float64 scaled_dot_product_attention with
    is_causal=True, K/V expanded per query-head group;
  * closed forms -- a zero query gives the prefix mean of V with
    lse = log(i+1) + 0; a one-token context returns v_0 exactly; scores
    {0, ln 2} weight two keys 1/3 and 2/3; one-hot V rows expose P itself,
    whose rows must sum to one, vanish above the diagonal, and equal
    exp(score - lse);
  * invariants -- packing order does not change a sequence's rows; the GQA
    map sends q head h to kv head h // (Hq/Hkv).
"""
from __future__ import annotations

import math

import numpy as np

TOL = 1e-10


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def check_bruteforce(attn):
    """mpmath loop over pairs, 50 significant digits, on a 2-sequence GQA pack."""
    import mpmath as mp
    mp.mp.dps = 50
    lens = [5, 3]
    hq, hkv, d = 4, 2, 6
    T = sum(lens)
    q, k, v = _rand((T, hq, d), 1), _rand((T, hkv, d), 2), _rand((T, hkv, d), 3)
    scale = 0.37
    cu = [0, 5, 8]
    o, lse = attn(q, k, v, cu, scale)
    for b in range(2):
        lo, hi = cu[b], cu[b + 1]
        for h in range(hq):
            g = h // (hq // hkv)
            for i in range(hi - lo):
                sc = [mp.mpf(scale) * mp.fsum(mp.mpf(q[lo + i, h, e]) * mp.mpf(k[lo + j, g, e]) for e in range(d))
                      for j in range(i + 1)]
                w = [mp.exp(s) for s in sc]
                z = mp.fsum(w)
                for e in range(d):
                    ref = mp.fsum(w[j] * mp.mpf(v[lo + j, g, e]) for j in range(i + 1)) / z
                    assert abs(float(ref) - o[lo + i, h, e]) < TOL, ("bruteforce o", b, h, i, e)
                assert abs(float(mp.log(z)) - lse[lo + i, h]) < TOL, ("bruteforce lse", b, h, i)


def check_torch_sdpa(attn):
    """torch float64 SDPA (is_causal) per sequence with K/V expanded per group."""
    import torch
    lens = [17, 1, 40]
    hq, hkv, d = 6, 2, 16
    T = sum(lens)
    q, k, v = _rand((T, hq, d), 4), _rand((T, hkv, d), 5), _rand((T, hkv, d), 6)
    scale = 1.0 / math.sqrt(d)
    cu = np.concatenate([[0], np.cumsum(lens)])
    o, lse = attn(q, k, v, cu, scale)
    for b in range(len(lens)):
        lo, hi = int(cu[b]), int(cu[b + 1])
        qt = torch.from_numpy(q[lo:hi]).permute(1, 0, 2)
        kt = torch.from_numpy(k[lo:hi]).permute(1, 0, 2).repeat_interleave(hq // hkv, dim=0)
        vt = torch.from_numpy(v[lo:hi]).permute(1, 0, 2).repeat_interleave(hq // hkv, dim=0)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, scale=scale)
        ref = ref.permute(1, 0, 2).numpy()
        assert np.max(np.abs(ref - o[lo:hi])) < 1e-10, ("sdpa", b)
        sc = torch.einsum("hid,hjd->hij", qt, kt) * scale
        sc = sc.masked_fill(torch.triu(torch.ones(hi - lo, hi - lo, dtype=torch.bool), 1), float("-inf"))
        ref_lse = torch.logsumexp(sc, dim=-1).permute(1, 0).numpy()
        assert np.max(np.abs(ref_lse - lse[lo:hi])) < 1e-10, ("sdpa lse", b)


def check_closed_forms(attn):
    hq, hkv, d = 2, 1, 8
    # zero query: uniform weights over the prefix -> prefix mean, lse = log(i+1)
    L = 9
    q = np.zeros((L, hq, d))
    k, v = _rand((L, hkv, d), 7), _rand((L, hkv, d), 8)
    o, lse = attn(q, k, v, [0, L], 0.5)
    for i in range(L):
        assert np.max(np.abs(o[i, 0] - v[:i + 1, 0].mean(axis=0))) < TOL, ("prefix mean", i)
        assert abs(lse[i, 1] - math.log(i + 1)) < TOL, ("prefix lse", i)
    # one-token context returns v_0 exactly, lse = scaled score
    q, k, v = _rand((1, hq, d), 9), _rand((1, hkv, d), 10), _rand((1, hkv, d), 11)
    o, lse = attn(q, k, v, [0, 1], 0.25)
    assert np.array_equal(o[0, 0], v[0, 0]) and np.array_equal(o[0, 1], v[0, 0]), "one token"
    assert abs(lse[0, 0] - 0.25 * float(q[0, 0] @ k[0, 0])) < TOL, "one token lse"
    # scores {0, ln 2}: weights 1/3 and 2/3
    q = np.zeros((2, 1, 2)); q[1, 0, 0] = 1.0
    k = np.zeros((2, 1, 2)); k[1, 0, 0] = math.log(2.0)
    v = _rand((2, 1, 2), 12)
    o, lse = attn(q, k, v, [0, 2], 1.0)
    assert np.max(np.abs(o[1, 0] - (v[0, 0] + 2 * v[1, 0]) / 3)) < TOL, "1/3-2/3"
    assert abs(lse[1, 0] - math.log(3.0)) < TOL, "log 3"
    # one-hot V exposes P: rows sum to 1, zero above the diagonal, P = exp(s - lse)
    L, d = 12, 12
    q, k = _rand((L, 1, d), 13), _rand((L, 1, d), 14)
    v = np.eye(L).reshape(L, 1, L)
    o, lse = attn(q, k, v, [0, L], 0.3)
    P = o[:, 0, :]
    assert np.max(np.abs(P.sum(axis=1) - 1.0)) < TOL, "rows sum to one"
    assert np.all(P[np.triu_indices(L, 1)] == 0.0), "causal: no weight above the diagonal"
    s = 0.3 * (q[:, 0] @ k[:, 0].T)
    for i in range(L):
        assert np.max(np.abs(P[i, :i + 1] - np.exp(s[i, :i + 1] - lse[i, 0]))) < TOL, ("P = exp(s - lse)", i)
    # dominant key: output ~ that key's value
    L = 6
    q = np.zeros((L, 1, 4)); q[:, 0, 0] = 1.0
    k = np.zeros((L, 1, 4)); k[3, 0, 0] = 200.0
    v = _rand((L, 1, 4), 15)
    o, _ = attn(q, k, v, [0, L], 1.0)
    assert np.max(np.abs(o[5, 0] - v[3, 0])) < 1e-12, "dominant key"


def check_invariants(attn):
    # packing order: a sequence's rows do not depend on its neighbours or position
    lens = [7, 13, 4]
    hq, hkv, d = 4, 2, 8
    seqs = [(_rand((L, hq, d), 20 + s), _rand((L, hkv, d), 30 + s), _rand((L, hkv, d), 40 + s)) for s, L in enumerate(lens)]

    def pack(order):
        q = np.concatenate([seqs[s][0] for s in order])
        k = np.concatenate([seqs[s][1] for s in order])
        v = np.concatenate([seqs[s][2] for s in order])
        cu = np.concatenate([[0], np.cumsum([lens[s] for s in order])])
        return q, k, v, cu

    o1, l1 = attn(*pack([0, 1, 2]), 0.35)
    o2, l2 = attn(*pack([2, 0, 1]), 0.35)
    cu1 = np.concatenate([[0], np.cumsum(lens)])
    cu2 = np.concatenate([[0], np.cumsum([lens[s] for s in [2, 0, 1]])])
    pos2 = {2: 0, 0: 1, 1: 2}
    for s in range(3):
        a = o1[cu1[s]:cu1[s + 1]]
        b = o2[cu2[pos2[s]]:cu2[pos2[s] + 1]]
        assert np.array_equal(a, b), ("pack order", s)
    # GQA map: q head h reads kv head h // G; compare with per-head expansion
    q, k, v, cu = pack([0, 1, 2])
    o_g, _ = attn(q, k, v, cu, 0.35)
    kx = np.repeat(k, hq // hkv, axis=1)
    vx = np.repeat(v, hq // hkv, axis=1)
    o_x, _ = attn(q, kx, vx, cu, 0.35)
    assert np.max(np.abs(o_g - o_x)) < TOL, "gqa map"


ALL_CHECKS = [check_bruteforce, check_torch_sdpa, check_closed_forms, check_invariants]


def run_all(attn):
    failures = []
    for chk in ALL_CHECKS:
        try:
            chk(attn)
        except AssertionError as e:  # noqa: PERF203
            failures.append((chk.__name__, str(e)))
    return failures
