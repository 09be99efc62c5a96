"""The five workload configurations at full size, on the GPU.

For each configuration: the full-sequence prefill over the whole pack, then
token-wise decode of the configuration's whole decode set, compared with the
prefill rows bit for bit (outputs and lse; Eq. (1) holds per position,
Section 4.1, and at operator level, Section 3.2), and rows compared with the
fp64 definition under the parity gate.  Inputs are seeded synthetic tensors
with the shapes of the paper's operator workloads and GSM8K rollouts
(Section 6), drawn on the GPU for the large packs.

  c1 tiny           every row of three seeds (test_gpu_attention)
  c2 Qwen-style     8 x (1024 + 3072), 32/8/128: all 3072 decode steps
                    (batch re-permuted every step), the prompt rows of a
                    prompt-only prefill, and every one of the 1,048,576
                    (token, head) rows against the fp64 definition
  c3 varlen pack    64 seqs ~U[512, 8192], 40/8/128: 4096 random tokens
                    re-run through decode in one batch; 4096 random rows and
                    the shortest sequence in full against fp64
  c4 GRPO rollout   64 prompts x 8 samples, shared 1024-token prompt pages,
                    responses ~U[256, 15360]: the whole rollout, all 15,360
                    decode steps, active batch re-permuted every step and
                    finished sequences dropped; 4096 rows against fp64
  c5 long context   8 x 32768, 64/8/128: all 1024 final decode steps
                    (batch re-permuted every step), prompt rows of
                    prefill(31744) vs prefill(32768), 4096 rows against
                    fp64, and the log-prob leg over a 151936-entry vocabulary
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from paper_2609_35140_amd import inputs

pytestmark = pytest.mark.gpu
cfg = pytest.importorskip("config_util")

# worker threads for the fp64 oracle (numpy releases the GIL in its kernels)
THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


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


def _blas_one_thread():
    from threadpoolctl import threadpool_limits
    return threadpool_limits(limits=1)


class Gate:
    """Accumulates the parity gate over many blocks of rows: every element
    within 4e-3 + 2^-8 |ref|, mean |err| over all elements <= 5e-4."""

    def __init__(self):
        self.n = 0
        self.sum_err = 0.0
        self.max_abs = 0.0
        self.n_over_bound = 0
        self.n_over_4e3 = 0
        self.nan = 0
        self.lse_max = 0.0

    def add(self, got, ref, lse_got=None, lse_ref=None):
        got = np.asarray(got, dtype=np.float64)
        ref = np.asarray(ref, dtype=np.float64)
        err = np.abs(got - ref)
        self.nan += int(np.isnan(got).sum())
        self.n += err.size
        self.sum_err += float(np.nansum(err))
        self.max_abs = max(self.max_abs, float(np.nanmax(err)) if err.size else 0.0)
        self.n_over_bound += int((~(err <= oracle.MAX_ABS + oracle.REL_BF16 * np.abs(ref))).sum())
        self.n_over_4e3 += int((err > oracle.MAX_ABS).sum())
        if lse_got is not None:
            d = np.abs(np.asarray(lse_got, dtype=np.float64) - np.asarray(lse_ref, dtype=np.float64))
            self.lse_max = max(self.lse_max, float(d.max()) if d.size else 0.0)

    def report(self):
        mean = self.sum_err / max(self.n, 1)
        return {"elements": self.n, "max_abs": self.max_abs, "mean_abs": mean, "n_over_4e-3": self.n_over_4e3,
                "n_over_bound": self.n_over_bound, "nan": self.nan, "lse_max_err": self.lse_max,
                "pass": self.n_over_bound == 0 and self.nan == 0 and mean <= oracle.MEAN_ABS
                and self.lse_max < oracle.LSE_ABS}


def _f64(bits):
    return oracle.bf16_to_f64(bits)


def _oracle_rows(pk, out, lse, picks, label):
    """fp64 definition at chosen (sequence, position, head) rows vs the GPU
    rows: each row is its query against keys/values 0..position of its kv
    head.  Sequences are handled by a pool of threads, each copying back
    its sequence's bits and widening only the kv-head prefixes it needs."""
    import torch
    w = pk.w
    group = w.num_q_heads // w.num_kv_heads
    scale = oracle.default_scale(w.head_dim)
    by_seq = {}
    for s, p, h in picks:
        by_seq.setdefault(int(s), []).append((int(p), int(h)))
    jobs = []
    for s, rows in sorted(by_seq.items()):
        lo = int(pk.cu[s])
        ti = torch.from_numpy(np.array([lo + p for p, _ in rows], dtype=np.int64)).cuda()
        top = max(p for p, _ in rows) + 1
        kb, vb = cfg.host_bits(pk.k[lo:lo + top]), cfg.host_bits(pk.v[lo:lo + top])
        qb, ob, lg = cfg.host_bits(pk.q[ti]), cfg.host_bits(out[ti]), lse[ti].cpu().numpy()
        by_kv = {}
        for r, (p, h) in enumerate(rows):
            by_kv.setdefault(h // group, []).append((r, p, h))
        for kvh, items in by_kv.items():  # one job per (sequence, kv head)
            jobs.append((items, kb, vb, kvh, qb, ob, lg))

    def run(job):
        items, kb, vb, kvh, qb, ob, lg = job
        got, ref, lgot, lref = [], [], [], []
        top = max(p for _, p, _ in items) + 1
        k64 = _f64(kb[:top, kvh])
        v64 = _f64(vb[:top, kvh])
        for r, p, h in items:
            o, l = oracle.attention_row_fp64(_f64(qb[r, h]), k64[:p + 1], v64[:p + 1], scale)
            ref.append(o)
            lref.append(l)
            got.append(_f64(ob[r, h]))
            lgot.append(float(lg[r, h]))
        return np.stack(got), np.stack(ref), np.asarray(lgot), np.asarray(lref)

    gate = Gate()
    with _blas_one_thread(), ThreadPoolExecutor(THREADS) as ex:
        for got, ref, lgot, lref in ex.map(run, jobs):
            gate.add(got, ref, lgot, lref)
    rep = gate.report()
    print(f"{label}: {len(picks)} oracle rows from {len(by_seq)} sequences: {rep}", flush=True)
    assert rep["pass"], rep
    return rep


def _random_rows(w, g, n_rows, seqs):
    """n_rows (sequence, position, head) picks spread evenly over `seqs`."""
    lens = np.asarray(w.seq_lens)
    per = n_rows // len(seqs)
    picks = []
    for s in seqs:
        for _ in range(per):
            picks.append((int(s), int(g.integers(0, lens[s])), int(g.integers(0, w.num_q_heads))))
    return picks


class Rollout:
    """Token-wise decode steps over a DevicePack, checked on the device:
    after each step the decoded rows and lse are compared bit for bit with
    the prefill rows at the same positions, the mismatch counts accumulated
    on the GPU (one host sync at the end)."""

    def __init__(self, ua, pk, out, lse, batch_max):
        import torch
        self.ua, self.pk, self.out, self.lse = ua, pk, out, lse
        w = pk.w
        self.ws = ua.new_workspace(ua.decode_workspace_bytes(batch_max, pk.max_seqlen, w.num_q_heads, w.head_dim))
        self.dout = torch.empty((batch_max, w.num_q_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
        self.dlse = torch.empty((batch_max, w.num_q_heads), dtype=torch.float32, device="cuda")
        self.bad = torch.zeros((), dtype=torch.int64, device="cuda")
        self.lse_bad = torch.zeros((), dtype=torch.int64, device="cuda")
        self.rows = 0
        self.steps = 0

    def run(self, seqs, positions):
        """seqs, positions: int64 arrays of one step's entries (a batch)."""
        import torch
        pk = self.pk
        B = len(seqs)
        tok = torch.from_numpy(pk.cu[seqs].astype(np.int64) + positions).cuda()
        q = pk.q.index_select(0, tok)
        table = pk.table_dev.index_select(0, torch.from_numpy(seqs).cuda())
        sl = torch.from_numpy((positions + 1).astype(np.int32)).cuda()
        dout, dlse = self.dout[:B], self.dlse[:B]
        self.ua.decode(q, pk.kp, pk.vp, table, sl, pk.max_seqlen, out=dout, lse=dlse, workspace=self.ws)
        same = (dout.view(torch.int16) == self.out.index_select(0, tok).view(torch.int16)).all(dim=-1)
        self.bad += (~same).sum()
        self.lse_bad += (dlse.view(torch.int32) != self.lse.index_select(0, tok).view(torch.int32)).sum()
        self.rows += B * pk.w.num_q_heads
        self.steps += 1

    def check(self, label):
        bad, lse_bad = int(self.bad.item()), int(self.lse_bad.item())
        print(f"{label}: {self.steps} decode steps, {self.rows - bad}/{self.rows} (entry, head) rows bitwise equal to "
              f"prefill; lse mismatches {lse_bad}", flush=True)
        assert bad == 0 and lse_bad == 0, (bad, lse_bad)
        return self.rows


def _prompt_rows_bitwise(ua, pk, out, lse, label):
    """Rollout prefill over the prompts alone equals the full prefill at the
    prompt rows (Eq. (1) at the prompt positions)."""
    import torch
    w = pk.w
    P = [int(x) for x in w.prompt_lens]
    idx = np.concatenate([np.arange(pk.cu[s], pk.cu[s] + P[s]) for s in range(w.num_seqs)])
    it = torch.from_numpy(idx).cuda()
    cu_p = torch.from_numpy(inputs.cu_seqlens(P)).cuda()
    pout, plse = ua.prefill(pk.q[it].contiguous(), pk.k[it].contiguous(), pk.v[it].contiguous(), cu_p, max(P),
                            return_lse=True)
    same = (pout.view(torch.int16) == out[it].view(torch.int16)).all(dim=-1)
    n_bad = int((~same).sum().item())
    lse_same = bool(torch.equal(plse.view(torch.int32), lse[it].view(torch.int32)))
    print(f"{label}: {same.numel() - n_bad}/{same.numel()} prompt rows of prefill(prompt) bitwise equal to "
          f"prefill(prompt||response); lse bitwise {lse_same}", flush=True)
    assert n_bad == 0 and lse_same
    return same.numel()


def test_c2_qwen_gqa_every_row(ua):
    import torch
    w = inputs.qwen_gqa()
    pk = cfg.DevicePack(w, tag=102)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    P, R, B = w.prompt_lens[0], w.response_lens[0], w.num_seqs
    g = inputs.rng(50, 2)
    ro = Rollout(ua, pk, out, lse, B)
    for step in range(R):  # token by token, all 8 sequences per step in a fresh order, as a rollout runs
        seqs = g.permutation(B).astype(np.int64)
        ro.run(seqs, np.full(B, P + step, dtype=np.int64))
    n_dec = ro.check("c2 decode")
    n_pr = _prompt_rows_bitwise(ua, pk, out, lse, "c2 prompts")
    assert n_dec + n_pr == w.total_tokens * w.num_q_heads == 1048576
    print(f"c2: bitwise set {n_dec + n_pr} rows = all {w.total_tokens} tokens x {w.num_q_heads} heads", flush=True)

    # every (token, head) row against the fp64 definition, one (sequence, head) causal problem at a time
    scale = oracle.default_scale(w.head_dim)
    group = w.num_q_heads // w.num_kv_heads
    gate = Gate()

    def one(job):
        qh, kh, vh, oh, lh = job
        o64, l64 = oracle.causal_attention_fp64(qh[:, None], kh[:, None], vh[:, None], [0, qh.shape[0]], scale)
        return _f64(oh), o64[:, 0], lh, l64[:, 0]

    for s in range(B):
        lo, hi = int(pk.cu[s]), int(pk.cu[s + 1])
        qb, kb, vb = pk.host_sequence(s)
        ob = cfg.host_bits(out[lo:hi])
        lb = lse[lo:hi].cpu().numpy()
        jobs = [(qb[:, h], kb[:, h // group], vb[:, h // group], ob[:, h], lb[:, h]) for h in range(w.num_q_heads)]
        with _blas_one_thread(), ThreadPoolExecutor(THREADS) as ex:
            for got, ref, lgot, lref in ex.map(one, jobs):
                gate.add(got, ref, lgot, lref)
        print(f"c2 fp64 oracle: sequence {s} done ({gate.n // w.head_dim} rows so far)", flush=True)
    rep = gate.report()
    print(f"c2 full fp64: {gate.n // w.head_dim} rows, {rep}", flush=True)
    assert gate.n == 1048576 * w.head_dim
    assert rep["pass"], rep
    del pk, out, lse, ro
    _free()


def test_c3_varlen_pack_spot_check(ua):
    import torch
    w = inputs.varlen_pack()
    pk = cfg.DevicePack(w, tag=103)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    g = inputs.rng(50, 3)
    lens = np.asarray(w.seq_lens)
    seqs = g.integers(0, w.num_seqs, size=4096).astype(np.int64)
    pos = np.array([int(g.integers(0, lens[s])) for s in seqs], dtype=np.int64)
    ro = Rollout(ua, pk, out, lse, 4096)
    ro.run(seqs, pos)
    n = ro.check("c3 4096 random tokens in one decode batch")
    assert n == 4096 * w.num_q_heads
    _oracle_rows(pk, out, lse, _random_rows(w, g, 4096, range(w.num_seqs)), "c3 random rows")
    # the shortest sequence, every row and head, against the fp64 definition
    s = int(np.argmin(lens))
    qh, kh, vh = pk.host_sequence(s)
    o64, l64 = oracle.causal_attention_fp64(qh, kh, vh, [0, qh.shape[0]])
    lo, hi = int(pk.cu[s]), int(pk.cu[s + 1])
    rep = oracle.parity_report(_f64(cfg.host_bits(out[lo:hi])), o64)
    print(f"c3 shortest sequence ({hi - lo} tokens x {w.num_q_heads} heads): {rep}", flush=True)
    assert rep["pass"], rep
    assert np.max(np.abs(lse[lo:hi].cpu().numpy() - l64)) < oracle.LSE_ABS
    del pk, out, lse, ro
    _free()


def test_c4_grpo_rollout_every_step(ua):
    import torch
    w = inputs.grpo_rollout()
    pk = cfg.DevicePack(w, tag=104, share_prompt_pages=True)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    P = np.asarray(w.prompt_lens, dtype=np.int64)
    R = np.asarray(w.response_lens, dtype=np.int64)
    g = inputs.rng(50, 4)
    ro = Rollout(ua, pk, out, lse, w.num_seqs)
    for step in range(int(R.max())):
        active = np.nonzero(R > step)[0]                # finished sequences drop out
        active = active[g.permutation(active.size)]     # batch composition re-drawn every step
        ro.run(active.astype(np.int64), P[active] + step)
        if step % 2048 == 2047:
            torch.cuda.synchronize()
            print(f"c4: {step + 1} steps issued", flush=True)
    n = ro.check("c4 whole rollout")
    assert ro.steps == int(R.max())  # the longest drawn response (responses ~ U[256, 15360])
    assert n == int(R.sum()) * w.num_q_heads
    seqs = g.choice(w.num_seqs, size=64, replace=False)
    _oracle_rows(pk, out, lse, _random_rows(w, g, 4096, seqs), "c4 random rows")
    del pk, out, lse, ro
    _free()


def test_c5_long_context_and_logprob(ua):
    import torch
    w = inputs.long_context()
    pk = cfg.DevicePack(w, tag=105)
    out, lse = ua.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, return_lse=True)
    P, R, B = w.prompt_lens[0], w.response_lens[0], w.num_seqs
    g = inputs.rng(50, 5)
    ro = Rollout(ua, pk, out, lse, B)
    for step in range(R):
        ro.run(g.permutation(B).astype(np.int64), np.full(B, P + step, dtype=np.int64))
    n = ro.check("c5 final 1024 steps")
    assert n == R * B * w.num_q_heads
    _prompt_rows_bitwise(ua, pk, out, lse, "c5 prompts")
    _oracle_rows(pk, out, lse, _random_rows(w, g, 4096, range(B)), "c5 random rows")
    del pk, out, lse, ro
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

    # the fused LM head + log-prob at the long-context step's size: 8192 response rows, hidden 8192
    # (64 q heads x 128), vocabulary 151936, weights ~ N(0, sigma^2 / H); sampled rows against the
    # oracle's reference and derived bound, and the batch-invariance of the rows
    H = w.num_q_heads * w.head_dim
    hidden = inputs.normal_bf16_device((rows, H), 1.0, 7, 1)
    lm_w = inputs.normal_bf16_device((V, H), w.logit_sigma / float(np.sqrt(H)), 7, 2)
    tg = torch.from_numpy(inputs.targets(rows, V)).cuda()
    lp = ua.lm_head_logprob(hidden, lm_w, tg)
    sample = np.sort(g.choice(rows, size=64, replace=False))
    si = torch.from_numpy(sample).cuda()
    one = ua.lm_head_logprob(hidden[si].contiguous(), lm_w, tg[si].contiguous())
    assert torch.equal(one.view(torch.int32), lp[si].view(torch.int32))
    ref, bound = oracle.lm_head_logprob_fp64(cfg.host_bits(hidden[si]), cfg.host_bits(lm_w),
                                             inputs.targets(rows, V)[sample])
    err = np.abs(lp[si].cpu().numpy().astype(np.float64) - ref)
    print(f"c5 fused LM head + logprob: 64 sampled rows of {rows}: max err {err.max():.3g}, max err/bound "
          f"{np.max(err / bound):.3f}; sub-batch bitwise equal", flush=True)
    assert np.all(err <= bound)
    del hidden, lm_w, lp
    _free()
