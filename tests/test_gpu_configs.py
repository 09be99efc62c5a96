"""The five workload configurations at full size, on the GPU.

For each configuration: the full-sequence prefill over the whole pack, then
token-wise decode of the configuration's decode set, compared with the
prefill rows bit for bit (outputs and lse; Eq. (1) at operator level,
Section 3.2), and a sample of rows compared with the fp64 definition under
the parity gate.  Inputs are seeded synthetic tensors with the shapes of the
paper's operator workloads and GSM8K rollouts (Section 6), drawn on the GPU
for the large packs.

  c1 tiny           covered by test_gpu_attention (every row, three seeds)
  c2 Qwen-style     8 x (1024 + 3072), 32/8/128: all 3072 decode steps
  c3 varlen pack    64 seqs ~U[512, 8192], 40/8/128: 4096 random tokens
                    re-run through decode in one batch; shortest sequence
                    in full against fp64
  c4 GRPO rollout   64 prompts x 8 samples, shared 1024-token prompt pages,
                    responses ~U[256, 15360]: sampled decode steps over the
                    whole response range, active batch re-permuted each step
  c5 long context   8 x 32768, 64/8/128: sampled steps of the final 1024,
                    prompt rows of prefill(31744) vs prefill(32768), and the
                    log-prob leg over a 151936-entry vocabulary
"""
import numpy as np
import pytest

import oracle
from paper_2609_35140_amd import inputs

pytestmark = pytest.mark.gpu
cfg = pytest.importorskip("config_util")


@pytest.fixture(scope="module")
def ua():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35140_amd import uattn
    uattn.lib()
    return uattn


def _free():
    import gc
    import torch
    gc.collect()
    torch.cuda.empty_cache()


def _bitwise(ua, pk, out, lse, entries, workspace=None, label=""):
    """Decode `entries` in one call; every row must equal its prefill row."""
    q, table, seqlens, maxs, tok = pk.decode_rows(entries)
    dout, dlse = ua.decode(q, pk.kp, pk.vp, table, seqlens, pk.max_seqlen, return_lse=True, workspace=workspace)
    import torch
    t = torch.from_numpy(tok).cuda()
    same = (dout.view(torch.int16) == out[t].view(torch.int16)).all(dim=-1)
    n_bad = int((~same).sum().item())
    lse_same = bool(torch.equal(dlse.view(torch.int32), lse[t].view(torch.int32)))
    print(f"{label}: {len(entries)} decode entries, {same.numel() - n_bad}/{same.numel()} rows bitwise; lse bitwise "
          f"{lse_same}", flush=True)
    assert n_bad == 0, f"{label}: {n_bad} of {same.numel()} (entry, head) rows differ from prefill"
    assert lse_same, f"{label}: lse differs from prefill"
    return dout, tok


def _oracle_rows(ua, pk, out, lse, picks, label):
    """fp64 definition at chosen (sequence, position, head) rows vs the GPU rows:
    each row is the query against keys/values 0..position of its kv head."""
    import torch
    w = pk.w
    group = w.num_q_heads // w.num_kv_heads
    scale = oracle.default_scale(w.head_dim)
    by_seq = {}
    for s, p, h in picks:
        by_seq.setdefault(int(s), []).append((int(p), int(h)))
    got, ref, lg, lref = [], [], [], []
    for s, rows in sorted(by_seq.items()):
        lo, hi = int(pk.cu[s]), int(pk.cu[s + 1])
        k64 = oracle.bf16_to_f64(cfg.host_bits(pk.k[lo:hi]))
        v64 = oracle.bf16_to_f64(cfg.host_bits(pk.v[lo:hi]))
        ti = torch.from_numpy(np.array([lo + p for p, _ in rows], dtype=np.int64)).cuda()
        q64 = oracle.bf16_to_f64(cfg.host_bits(pk.q[ti]))
        o_bits = cfg.host_bits(out[ti])
        l_gpu = lse[ti].cpu().numpy()
        for r, (p, h) in enumerate(rows):
            o, l = oracle.attention_row_fp64(q64[r, h], k64[:p + 1, h // group], v64[:p + 1, h // group], scale)
            ref.append(o)
            lref.append(l)
            got.append(oracle.bf16_to_f64(o_bits[r, h]))
            lg.append(float(l_gpu[r, h]))
        del k64, v64
    rep = oracle.parity_report(np.stack(got), np.stack(ref))
    lerr = float(np.max(np.abs(np.asarray(lg) - np.asarray(lref))))
    print(f"{label}: {len(got)} oracle rows {rep}; lse max err {lerr:.3g}", flush=True)
    assert rep["pass"], rep
    assert lerr < oracle.LSE_ABS, lerr


def test_c2_qwen_gqa_all_decode_steps(ua):
    import torch
    w = inputs.qwen_gqa()
    pk = cfg.DevicePack(w, tag=102)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    P, R, B = w.prompt_lens[0], w.response_lens[0], w.num_seqs
    ws = ua.new_workspace(ua.decode_workspace_bytes(B, pk.max_seqlen, w.num_q_heads, w.head_dim))
    bad = 0
    lse_bad = 0
    for step in range(R):  # token-by-token, all 8 sequences per step, as a rollout runs
        entries = [(s, P + step) for s in range(B)]
        q, table, seqlens, maxs, tok = pk.decode_rows(entries)
        dout, dlse = ua.decode(q, pk.kp, pk.vp, table, seqlens, pk.max_seqlen, return_lse=True, workspace=ws)
        t = torch.from_numpy(tok).cuda()
        bad += int((~(dout.view(torch.int16) == out[t].view(torch.int16)).all(dim=-1)).sum().item())
        lse_bad += int((dlse.view(torch.int32) != lse[t].view(torch.int32)).sum().item())
    rows = R * B * w.num_q_heads
    print(f"c2: {rows - bad}/{rows} decode rows bitwise equal to prefill; lse mismatches {lse_bad}", flush=True)
    assert bad == 0 and lse_bad == 0
    g = inputs.rng(50, 2)
    picks = [(int(g.integers(0, B)), int(g.integers(0, P + R)), int(g.integers(0, w.num_q_heads))) for _ in range(256)]
    _oracle_rows(ua, pk, out, lse, picks, "c2")
    del pk, out, lse
    _free()


def test_c3_varlen_pack_spot_check(ua):
    w = inputs.varlen_pack()
    pk = cfg.DevicePack(w, tag=103)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    g = inputs.rng(50, 3)
    lens = np.asarray(w.seq_lens)
    seqs = g.integers(0, w.num_seqs, size=4096)
    entries = [(int(s), int(g.integers(0, lens[s]))) for s in seqs]
    _bitwise(ua, pk, out, lse, entries, label="c3 4096 random tokens")
    picks = [(s, p, int(g.integers(0, w.num_q_heads))) for s, p in entries[:1024]]
    _oracle_rows(ua, pk, out, lse, picks, "c3 random rows")
    # the shortest sequence, every row and head, against the fp64 definition
    s = int(np.argmin(lens))
    qh, kh, vh = pk.host_sequence(s)
    o64, l64 = oracle.causal_attention_fp64(qh, kh, vh, [0, qh.shape[0]])
    lo, hi = int(pk.cu[s]), int(pk.cu[s + 1])
    got = cfg.host_bits(out[lo:hi])
    rep = oracle.parity_report((got.astype(np.uint32) << 16).view(np.float32).astype(np.float64), o64)
    print(f"c3 shortest sequence ({hi - lo} tokens x {w.num_q_heads} heads): {rep}", flush=True)
    assert rep["pass"], rep
    assert np.max(np.abs(lse[lo:hi].cpu().numpy() - l64)) < oracle.LSE_ABS
    del pk, out, lse
    _free()


def test_c4_grpo_rollout_sampled_steps(ua):
    w = inputs.grpo_rollout()
    pk = cfg.DevicePack(w, tag=104, share_prompt_pages=True)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    P = np.asarray(w.prompt_lens)
    R = np.asarray(w.response_lens)
    g = inputs.rng(50, 4)
    steps = sorted(set([0, 1, 2, 63, 64, 255, 256, 1000, int(R.max()) - 1] +
                       [int(x) for x in g.integers(0, int(R.max()), size=15)]))
    ws = ua.new_workspace(ua.decode_workspace_bytes(w.num_seqs, pk.max_seqlen, w.num_q_heads, w.head_dim))
    decoded = []
    for step in steps:
        active = np.nonzero(R > step)[0]
        active = active[g.permutation(active.size)]  # batch composition re-drawn every step
        entries = [(int(s), int(P[s]) + step) for s in active]
        _bitwise(ua, pk, out, lse, entries, workspace=ws, label=f"c4 step {step} (batch {len(entries)})")
        decoded += entries
    # oracle rows drawn from the decoded entries of a few sequences
    chosen = set(int(x) for x in g.choice(w.num_seqs, size=24, replace=False))
    cand = [(s, p) for s, p in decoded if s in chosen]
    pick_idx = g.choice(len(cand), size=min(384, len(cand)), replace=False)
    picks = [(cand[i][0], cand[i][1], int(g.integers(0, w.num_q_heads))) for i in pick_idx]
    _oracle_rows(ua, pk, out, lse, picks, "c4 decoded rows")
    del pk, out, lse, ws
    _free()


def test_c5_long_context_and_logprob(ua):
    import torch
    w = inputs.long_context()
    pk = cfg.DevicePack(w, tag=105)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    P, R, B = w.prompt_lens[0], w.response_lens[0], w.num_seqs
    g = inputs.rng(50, 5)
    steps = sorted(set([0, 1, R - 1] + [int(x) for x in g.integers(0, R, size=29)]))
    ws = ua.new_workspace(ua.decode_workspace_bytes(B, pk.max_seqlen, w.num_q_heads, w.head_dim))
    for step in steps:
        entries = [(s, P + step) for s in g.permutation(B)]
        _bitwise(ua, pk, out, lse, entries, workspace=ws, label=f"c5 step {step}")
    # prompt rows: prefill over the prompts alone equals the full prefill there
    idx = np.concatenate([np.arange(pk.cu[s], pk.cu[s] + P) for s in range(B)])
    it = torch.from_numpy(idx).cuda()
    cu_p = torch.from_numpy(inputs.cu_seqlens([P] * B)).cuda()
    pout, plse = ua.prefill(pk.q[it].contiguous(), pk.k[it].contiguous(), pk.v[it].contiguous(), cu_p, P,
                            return_lse=True)
    assert torch.equal(pout.view(torch.int16), out[it].view(torch.int16)), "prompt rows: prefill(p) != prefill(p||y)"
    assert torch.equal(plse.view(torch.int32), lse[it].view(torch.int32))
    del pout, plse, it
    picks = [(int(g.integers(0, B)), int(g.integers(0, P + R)), int(g.integers(0, w.num_q_heads))) for _ in range(256)]
    _oracle_rows(ua, pk, out, lse, picks, "c5")
    del pk, out, lse, ws
    _free()

    # log-prob leg: 8 x 1024 response rows over the vocabulary, N(0, sigma^2) logits
    rows, V = B * R, w.vocab
    logits = inputs.normal_bf16_device((rows, V), w.logit_sigma, 7, 105)
    tg = torch.from_numpy(inputs.targets(rows, V, tag=105)).cuda()
    full = ua.logprob(logits, tg)
    sample = g.choice(rows, size=64, replace=False)
    one = torch.stack([ua.logprob(logits[i:i + 1], tg[i:i + 1])[0] for i in sample])
    assert torch.equal(one.view(torch.int32), full[torch.from_numpy(sample).cuda()].view(torch.int32))
    perm = torch.from_numpy(g.permutation(rows)[: rows // 3]).cuda()
    sub = ua.logprob(logits[perm].contiguous(), tg[perm].contiguous())
    assert torch.equal(sub.view(torch.int32), full[perm].view(torch.int32))
    ratio = torch.exp(sub.double() - full[perm].double())
    assert bool((ratio == 1.0).all())
    lg_host = cfg.host_bits(logits[torch.from_numpy(sample).cuda()])
    ref = oracle.logprob_fp64(lg_host, inputs.targets(rows, V, tag=105)[sample])
    err = np.abs(full[torch.from_numpy(sample).cuda()].cpu().numpy().astype(np.float64) - ref)
    print(f"c5 logprob: single-row == batched == permuted sub-batch; oracle max err {err.max():.3g}", flush=True)
    assert err.max() < 2e-5
    del logits, full
    _free()
