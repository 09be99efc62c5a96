"""GPU indexed KV-cache write: exact post-write cache state, and the rollout
step it serves (write the new token's K/V, then decode it) staying bitwise
equal to the full-sequence path (Section 6 Q3's prescribed checks)."""
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


CASES = [  # (P, Hkv, page, d, B, maxp, N, token stride padding)
    (40, 8, 64, 128, 6, 9, 300, 0),
    (25, 1, 16, 64, 3, 12, 120, 8),
    (64, 2, 128, 128, 4, 4, 1000, 16),
    (7, 4, 16, 64, 2, 5, 1, 0),
]


@pytest.mark.parametrize("P,hkv,page,d,B,maxp,N,pad", CASES)
def test_post_write_state_is_exact(ua, P, hkv, page, d, B, maxp, N, pad):
    import torch
    g = inputs.rng(60, P, N)
    kp = g.integers(0, 2 ** 16, size=(P, hkv, page, d), dtype=np.uint16)
    vp = g.integers(0, 2 ** 16, size=(P, hkv, page, d), dtype=np.uint16)
    # block table over a shuffled pool, with -1 and out-of-pool entries mixed in
    table = g.integers(-2, P + 2, size=(B, maxp)).astype(np.int32)
    # distinct (sequence, position) slots, plus padding and out-of-range tokens
    slots = g.choice(B * maxp * page, size=min(N, B * maxp * page), replace=False)
    seq = (slots // (maxp * page)).astype(np.int32)
    pos = (slots % (maxp * page)).astype(np.int32)
    if N >= 8:
        pos[:2] = -1                  # padding
        seq[2] = B                    # no such sequence
        pos[3] = maxp * page + 5      # past the table
    # distinct logical slots can still share a physical slot when the table
    # repeats an entry; keep only the first token per physical slot
    phys = np.where((pos >= 0) & (seq < B) & (pos // page < maxp),
                    table[np.minimum(seq, B - 1), np.minimum(pos // page, maxp - 1)], -1)
    key = phys.astype(np.int64) * page + pos % page
    dup = np.zeros(len(key), dtype=bool)
    seen = set()
    for i, k_ in enumerate(key):
        if phys[i] >= 0 and phys[i] < P:
            if k_ in seen:
                dup[i] = True
            seen.add(k_)
    pos[dup] = -1
    n = len(pos)
    row = hkv * d + pad
    k_rows = g.integers(0, 2 ** 16, size=(n, row), dtype=np.uint16)
    v_rows = g.integers(0, 2 ** 16, size=(n, row), dtype=np.uint16)
    k_new = gu.dev(k_rows)[:, : hkv * d].unflatten(1, (hkv, d))   # token rows `row` elements apart
    v_new = gu.dev(v_rows)[:, : hkv * d].unflatten(1, (hkv, d))
    kd, vd = gu.dev(kp), gu.dev(vp)
    ua.kv_write(k_new, v_new, gu.dev_i32(table), gu.dev_i32(seq), gu.dev_i32(pos), kd, vd)
    want_k, want_v = oracle.kv_write(kp, vp, k_rows[:, : hkv * d].reshape(n, hkv, d),
                                     v_rows[:, : hkv * d].reshape(n, hkv, d), table, seq, pos)
    got_k, got_v = gu.host_bits(kd), gu.host_bits(vd)
    print(f"P={P} hkv={hkv} page={page} d={d}: {int((pos >= 0).sum())} tokens, "
          f"{int((got_k != kp).any(axis=-1).sum())} rows changed", flush=True)
    assert np.array_equal(got_k, want_k)
    assert np.array_equal(got_v, want_v)
    torch.cuda.synchronize()


def test_rollout_step_write_then_decode_equals_prefill(ua):
    """Prompt K/V written into an empty cache, then each response token's K/V
    written just before it is decoded: every decoded row equals the full
    prefill row bit for bit (the Eq. (1) replay with the write in the loop)."""
    import torch
    w = inputs.custom(8, 2, 128, [64 + 40, 150 + 70, 33 + 20], sigma=1.0, page_size=16, prompt_lens=[64, 150, 33])
    pk = gu.Pack(w, seed=11)
    full = gu.host_bits(ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen))
    kp = torch.full_like(pk.kp, float("nan"))
    vp = torch.full_like(pk.vp, float("nan"))
    table = pk.table_dev
    P = w.prompt_lens
    seq = np.concatenate([np.full(P[b], b) for b in range(w.num_seqs)]).astype(np.int32)
    pos = np.concatenate([np.arange(P[b]) for b in range(w.num_seqs)]).astype(np.int32)
    tok = pk.cu[seq] + pos
    it = torch.from_numpy(tok).cuda()
    ua.kv_write(pk.k[it], pk.v[it], table, gu.dev_i32(seq), gu.dev_i32(pos), kp, vp)
    R = [L - p for L, p in zip(w.seq_lens, P)]
    bad = 0
    for step in range(max(R)):
        act = [b for b in range(w.num_seqs) if step < R[b]]
        sq = np.array(act, dtype=np.int32)
        ps = np.array([P[b] + step for b in act], dtype=np.int32)
        tk = torch.from_numpy(pk.cu[sq] + ps).cuda()
        ua.kv_write(pk.k[tk], pk.v[tk], table, gu.dev_i32(sq), gu.dev_i32(ps), kp, vp)
        q = pk.q[tk].contiguous()
        d = ua.decode(q, kp, vp, table[torch.from_numpy(sq.astype(np.int64)).cuda()].contiguous(), gu.dev_i32(ps + 1),
                      max(w.seq_lens))
        bad += int((~gu.rows_equal_bits(gu.host_bits(d), full[pk.cu[sq] + ps])).sum())
    assert bad == 0, bad
    # and the caches now hold exactly the paged layout of the packed K/V (NaN elsewhere)
    assert np.array_equal(gu.host_bits(kp), pk.kp_host)
    assert np.array_equal(gu.host_bits(vp), pk.vp_host)


def test_graph_replay_with_varying_inputs(ua):
    """kv_write captured in a HIP graph, replayed with new rows and positions
    written into the captured buffers, matches eager calls each replay."""
    import torch
    P, hkv, page, d, B, maxp, N = 20, 4, 16, 128, 2, 8, 64
    g = inputs.rng(61)
    table = gu.dev_i32(g.permutation(P)[: B * maxp].reshape(B, maxp))
    kp0 = gu.dev(g.integers(0, 2 ** 16, size=(P, hkv, page, d), dtype=np.uint16))
    vp0 = gu.dev(g.integers(0, 2 ** 16, size=(P, hkv, page, d), dtype=np.uint16))
    k_new = torch.empty((N, hkv, d), dtype=torch.bfloat16, device="cuda")
    v_new = torch.empty_like(k_new)
    seq = torch.empty(N, dtype=torch.int32, device="cuda")
    pos = torch.empty(N, dtype=torch.int32, device="cuda")
    kp, vp = kp0.clone(), vp0.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s):
            ua.kv_write(k_new, v_new, table, seq, pos, kp, vp, stream=s)
    torch.cuda.synchronize()
    for rep in range(4):
        slots = g.choice(B * maxp * page, size=N, replace=False)
        k_new.copy_(gu.dev(g.integers(0, 2 ** 16, size=(N, hkv, d), dtype=np.uint16)))
        v_new.copy_(gu.dev(g.integers(0, 2 ** 16, size=(N, hkv, d), dtype=np.uint16)))
        seq.copy_(gu.dev_i32(slots // (maxp * page)))
        pos.copy_(gu.dev_i32(slots % (maxp * page)))
        kp.copy_(kp0)
        vp.copy_(vp0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ke, ve = kp0.clone(), vp0.clone()
        ua.kv_write(k_new, v_new, table, seq, pos, ke, ve)
        torch.cuda.synchronize()
        assert torch.equal(kp.view(torch.int16), ke.view(torch.int16)), rep
        assert torch.equal(vp.view(torch.int16), ve.view(torch.int16)), rep
