"""GPU attention backward: parity of dQ, dK, dV with the fp64 oracle, and the
determinism the policy update needs (the same bits on every call and for a
sequence in any batch).

Inputs to the backward are what the training step feeds it: the GPU forward's
own bf16 output and fp32 log-sum-exp.  The bound is derived from the
kernels' arithmetic (fp32 scores and exp2, bf16 P and dS as matrix operands,
fp32 accumulation, one bf16 rounding per result) plus the forward's bf16
output entering D_i = dO_i . O_i; per element

    |got - ref| <= 2^-7 * scale_elem + 2^-8 * |ref|

with scale_elem from oracle.backward_error_scales (sum of |terms| of each
gradient, with D's term size a_i).  The relative error of P from the saved
log-sum-exp (whose normalizer sums bf16 weights) and its bf16 rounding are
each at most 2^-9; the 2^-7 coefficient leaves a factor two over their sum.
"""
import numpy as np
import pytest

import oracle
from paper_2609_35140_amd import inputs

pytestmark = pytest.mark.gpu
gu = pytest.importorskip("gpu_util")

A_COEF = 2.0 ** -7
R_COEF = 2.0 ** -8


@pytest.fixture(scope="module")
def ua():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35140_amd import uattn
    uattn.lib()
    return uattn


def _inputs(lens, hq, hkv, d, sigma, tag):
    cu = inputs.cu_seqlens(lens)
    T = int(cu[-1])
    key = (tag, hq, hkv, d, len(lens))
    q = inputs.normal_bf16((T, hq, d), sigma, 81, *key, 0)
    k = inputs.normal_bf16((T, hkv, d), sigma, 81, *key, 1)
    v = inputs.normal_bf16((T, hkv, d), sigma, 81, *key, 2)
    do = inputs.normal_bf16((T, hq, d), 1.0, 81, *key, 3)
    return q, k, v, do, cu


def _run(ua, q, k, v, do, cu, max_seqlen=None):
    qd, kd, vd, dod = gu.dev(q), gu.dev(k), gu.dev(v), gu.dev(do)
    cud = gu.dev_i32(cu)
    ms = int(np.max(np.diff(cu))) if max_seqlen is None else max_seqlen
    out, lse = ua.prefill(qd, kd, vd, cud, ms, return_lse=True)
    return ua.prefill_backward(qd, kd, vd, out, dod, lse, cud, ms)


def _check(name, got_bits, ref, scale):
    got = oracle.bf16_to_f64(got_bits)
    err = np.abs(got - ref)
    bound = A_COEF * scale + R_COEF * np.abs(ref)
    ratio = float(np.max(err / np.maximum(bound, 1e-300)))
    print(f"  {name}: max err {err.max():.3e}  mean err {err.mean():.2e}  max err/bound {ratio:.3f}", flush=True)
    assert np.all(np.isfinite(got)), name
    assert np.all(err <= bound), (name, ratio)


CASES = [  # (sequence lengths, Hq, Hkv, d, sigma)
    ([300, 1, 129, 64, 0, 513], 8, 2, 128, 1.0),
    ([77, 200], 4, 4, 64, 1.0),
    ([257, 31, 1, 1], 16, 2, 64, 1.0),
    ([1000, 390], 32, 8, 128, 0.25),
    ([1], 4, 1, 128, 1.0),
]


@pytest.mark.parametrize("lens,hq,hkv,d,sigma", CASES)
def test_matches_oracle(ua, lens, hq, hkv, d, sigma):
    q, k, v, do, cu = _inputs(lens, hq, hkv, d, sigma, 0)
    print(f"lens={lens} hq={hq} hkv={hkv} d={d} sigma={sigma}", flush=True)
    dq, dk, dv = _run(ua, q, k, v, do, cu)
    ref = oracle.attention_backward_fp64(q, k, v, do, cu)
    sc = oracle.backward_error_scales(q, k, v, do, cu)
    for name, got, r, s in zip(("dq", "dk", "dv"), (dq, dk, dv), ref, sc):
        _check(name, gu.host_bits(got), r, s)


def test_repeated_calls_are_bitwise_equal(ua):
    q, k, v, do, cu = _inputs([700, 333, 64], 8, 2, 128, 1.0, 1)
    first = [gu.host_bits(x) for x in _run(ua, q, k, v, do, cu)]
    for _ in range(2):
        again = [gu.host_bits(x) for x in _run(ua, q, k, v, do, cu)]
        for a, b in zip(first, again):
            assert np.array_equal(a, b)


def test_batch_invariance(ua):
    """A sequence's gradients do not depend on the other sequences, their
    order, its place in the pack or max_seqlen."""
    hq, hkv, d = 8, 2, 128
    q, k, v, do, cu = _inputs([130, 517, 64, 1, 300], hq, hkv, d, 1.0, 2)
    batch = [gu.host_bits(x) for x in _run(ua, q, k, v, do, cu, max_seqlen=1024)]
    for s in (1, 4, 3):
        lo, hi = int(cu[s]), int(cu[s + 1])
        alone = [gu.host_bits(x) for x in _run(ua, q[lo:hi], k[lo:hi], v[lo:hi], do[lo:hi],
                                                np.array([0, hi - lo], dtype=np.int32))]
        for a, b in zip(batch, alone):
            assert np.array_equal(a[lo:hi], b), s
    # reversed order
    order = [4, 3, 2, 1, 0]
    parts = [(int(cu[s]), int(cu[s + 1])) for s in order]
    cat = lambda x: np.concatenate([x[lo:hi] for lo, hi in parts])
    cu2 = inputs.cu_seqlens([hi - lo for lo, hi in parts])
    rev = [gu.host_bits(x) for x in _run(ua, cat(q), cat(k), cat(v), cat(do), cu2)]
    for j, (lo, hi) in enumerate(parts):
        for a, b in zip(batch, rev):
            assert np.array_equal(a[lo:hi], b[int(cu2[j]):int(cu2[j + 1])])


def test_sum_of_key_gradients_is_small(ua):
    """The keys' dK of one (sequence, kv head) sum to zero exactly in the
    definition; the GPU's sum stays within the accumulated bound."""
    q, k, v, do, cu = _inputs([400, 97], 8, 2, 128, 1.0, 3)
    _, dk, _ = _run(ua, q, k, v, do, cu)
    _, sk, _ = oracle.backward_error_scales(q, k, v, do, cu)
    got = gu.host_f64(dk)
    for b in range(2):
        lo, hi = int(cu[b]), int(cu[b + 1])
        tot = np.abs(got[lo:hi].sum(axis=0))
        assert np.all(tot <= (A_COEF + R_COEF) * sk[lo:hi].sum(axis=0)), b


def _full_size(ua, w, tag, n_rows, full, alone):
    """Full-size backward in the launch configuration the benchmark times:
    n_rows sampled dQ rows against the oracle; all keys of one (sequence, kv
    head) = `full` for dK and dV (None to skip); sequence `alone` run by
    itself equal bit for bit to its rows in the batch."""
    import torch
    cfg = pytest.importorskip("config_util")
    pk = cfg.DevicePack(w, tag=tag)
    hq, hkv = w.num_q_heads, w.num_kv_heads
    grp = hq // hkv
    dout = inputs.normal_bf16_device(tuple(pk.q.shape), 1.0, tag, 9)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    dq, dk, dv = ua.prefill_backward(pk.q, pk.k, pk.v, out, dout, lse, pk.cu_dev, pk.max_seqlen)
    torch.cuda.synchronize()

    def seq_host(s, positions=None):
        """Host bits of sequence s: K and V in full; Q and dO in full, or only at
        `positions` (the other rows left zero, unread by the row oracle)."""
        lo, hi = int(pk.cu[s]), int(pk.cu[s + 1])
        ks, vs = gu.host_bits(pk.k[lo:hi]), gu.host_bits(pk.v[lo:hi])
        if positions is None:
            return lo, hi, [gu.host_bits(pk.q[lo:hi]), ks, vs, gu.host_bits(dout[lo:hi])]
        qs = np.zeros((hi - lo, hq, w.head_dim), dtype=np.uint16)
        ds = np.zeros_like(qs)
        ti = torch.from_numpy(np.array([lo + p for p in positions], dtype=np.int64)).cuda()
        qs[positions] = gu.host_bits(pk.q[ti])
        ds[positions] = gu.host_bits(dout[ti])
        return lo, hi, [qs, ks, vs, ds]

    g = inputs.rng(51, tag)
    picks = {}
    for _ in range(n_rows):
        s = int(g.integers(0, w.num_seqs))
        picks.setdefault(s, []).append((int(g.integers(0, w.seq_lens[s])), int(g.integers(0, hq))))
    got, ref, mag = [], [], []
    for s, rows in sorted(picks.items()):
        lo, hi, (qs, ks, vs, ds) = seq_host(s, sorted({p for p, _ in rows}))
        r, m = oracle.dq_rows_fp64(qs, ks, vs, ds, [0, hi - lo], rows, with_scale=True)
        ti = torch.from_numpy(np.array([lo + p for p, _ in rows], dtype=np.int64)).cuda()
        bits = gu.host_bits(dq[ti])
        ref.append(r)
        mag.append(m)
        got.append(np.stack([bits[i, h] for i, (_, h) in enumerate(rows)]))
        del qs, ks, vs, ds
    print(f"{w.name}: {n_rows} sampled dQ rows:", flush=True)
    _check("dq", np.concatenate(got), np.concatenate(ref), np.concatenate(mag))

    if full is not None:
        s, kvh = full
        lo, hi, (qs, ks, vs, ds) = seq_host(s)
        heads = list(range(kvh * grp, (kvh + 1) * grp))
        args = (qs[:, heads], ks[:, kvh:kvh + 1], vs[:, kvh:kvh + 1], ds[:, heads], [0, hi - lo])
        _, rk, rv = oracle.attention_backward_fp64(*args)
        _, sk, sv = oracle.backward_error_scales(*args)
        print(f"{w.name}: sequence {s}, kv head {kvh}, all {hi - lo} keys:", flush=True)
        _check("dk", gu.host_bits(dk[lo:hi, kvh:kvh + 1]), rk, sk)
        _check("dv", gu.host_bits(dv[lo:hi, kvh:kvh + 1]), rv, sv)

    lo, hi = int(pk.cu[alone]), int(pk.cu[alone + 1])
    cu1 = gu.dev_i32([0, hi - lo])
    sl = [x[lo:hi].contiguous() for x in (pk.q, pk.k, pk.v, dout)]
    o1, l1 = ua.prefill(sl[0], sl[1], sl[2], cu1, hi - lo, return_lse=True)
    one = ua.prefill_backward(sl[0], sl[1], sl[2], o1, sl[3], l1, cu1, hi - lo)
    for a, b in zip((dq, dk, dv), one):
        assert torch.equal(a[lo:hi].view(torch.int16), b.view(torch.int16))
    print(f"{w.name}: sequence {alone} ({hi - lo} tokens) alone == in the batch, bit for bit", flush=True)


def test_full_size_qwen_gqa(ua):
    """Benchmark shape: 8 x 4096 tokens, 32 q / 8 kv heads, d 128, N(0,0.25)
    inputs, N(0,1) upstream gradient."""
    _full_size(ua, inputs.qwen_gqa(), 106, 256, (3, 5), 6)


def test_full_size_varlen_pack(ua):
    """Varlen training pack: 64 sequences ~U[512, 8192] (278K tokens), 40 q /
    8 kv heads (group 5), N(0,1) inputs; dK/dV in full for the shortest
    sequence."""
    w = inputs.varlen_pack()
    short = int(np.argmin(w.seq_lens))
    _full_size(ua, w, 107, 256, (short, 3), int(np.argmax(w.seq_lens)))


def test_full_size_long_context(ua):
    """Long context: 8 x 32768 tokens, 64 q / 8 kv heads (group 8), N(0,0.25)
    inputs: sampled dQ rows (dK/dV of a 32K sequence is beyond the oracle's
    budget here) and one 32K sequence alone == in the batch."""
    _full_size(ua, inputs.long_context(), 108, 64, None, 2)


def test_graph_replay_with_varying_inputs(ua):
    """The forward and backward captured in one HIP graph, replayed with new
    inputs written into the captured buffers, with eager work between the
    replays: every replay equals the eager calls bit for bit."""
    import torch
    lens = [300, 129, 1, 513]
    hq, hkv, d = 8, 2, 128
    cu = inputs.cu_seqlens(lens)
    T = int(cu[-1])
    cud = gu.dev_i32(cu)
    bufs = [torch.empty((T, h, d), dtype=torch.bfloat16, device="cuda") for h in (hq, hkv, hkv, hq)]
    q, k, v, do = bufs
    ws = torch.empty(ua.prefill_backward_workspace_bytes(T, hq), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(q)
    lse = torch.empty((T, hq), dtype=torch.float32, device="cuda")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s):
            ua.prefill(q, k, v, cud, 513, out=out, lse=lse, stream=s)
            ua.prefill_backward(q, k, v, out, do, lse, cud, 513, dq=dq, dk=dk, dv=dv, workspace=ws, stream=s)
    torch.cuda.synchronize()
    for rep in range(4):
        for i, b in enumerate(bufs):
            b.copy_(gu.dev(inputs.normal_bf16(tuple(b.shape), 1.0, 82, rep, i)))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        o2, l2 = ua.prefill(q, k, v, cud, 513, return_lse=True)
        e = ua.prefill_backward(q, k, v, o2, do, l2, cud, 513)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), o2.view(torch.int16)), rep
        for a, b in zip((dq, dk, dv), e):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), rep
