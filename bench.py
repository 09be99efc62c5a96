#!/usr/bin/env python3
"""Benchmark of the unified-attention hot path on one MI355X.

One step = one pass of the whole path over one batch of the Qwen-style GQA
workload (8 sequences of 1024 prompt + 3072 response tokens, 32 q / 8 kv
heads, head_dim 128, bf16 ~ N(0, 0.25), paged KV with 64-token pages):

  1. rollout prefill over the 8 prompts             (full-sequence entry point)
     and the indexed write of the prompts' K/V into the paged cache
  2. rollout decode of the 3072 response tokens,
     token by token, batch 8, against the paged cache (token-wise entry point)
  3. Q/K RMSNorm + NeoX RoPE over the 8 full trajectories, then the policy-update
     prefill over them (full-sequence entry point; it runs on the raw Q/K so
     that the bitwise comparison with the decode rows uses the same inputs)
  4. the batch-invariant LM head (hidden 4096 -> 151,936 logits, ~ N(0, 4)) of
     the 8 x 3072 response tokens, and their log-probabilities

Inputs are resident in HBM before the timed region.  Every phase is bracketed
by HIP events on the stream it runs on; the 3072 decode launches are replayed
as one HIP graph captured before timing.  After timing, the decoded
rows and the prompt-prefill rows are compared bit for bit with the policy-
update prefill rows at the same positions (the paper's Eq. (1) at operator
level).  The CPU oracle is timed on a bounded sample of the same decode work.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prefill TFLOP/s + decode KV GB/s (% of MI355X peak); prefill-vs-decode bitwise match %"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU-oracle sample")
    ap.add_argument("--cpu-row-seconds", type=float, default=2.0,
                    help="budget of each other row's CPU-oracle sample")
    ap.add_argument("--eager-decode", action="store_true", help="launch the decode steps one by one (no HIP graph)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="before timing, copy 1 GiB device to device once (the known-size dispatch that scales "
                         "the FETCH_SIZE / WRITE_SIZE counters of a profiling run)")
    return ap.parse_args()


DECODE_SOURCES = ("uattn_decode.hip", "uattn_numerics.h", "uattn_tile_io.h")
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "decode_kernel_qwen_gqa_traffic.md")


def decode_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in DECODE_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_35140_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per decode launch from the committed counter summary, or None
    when it is absent or was taken on other kernel sources."""
    try:
        with open(TRAFFIC_SUMMARY) as f:
            text = f.read()
    except OSError:
        return None
    blk = text.split("```json", 1)
    if len(blk) < 2:
        return None
    try:
        rec = json.loads(blk[1].split("```", 1)[0])
    except ValueError:
        return None
    if rec.get("source_sha256") != decode_source_digest():
        return None
    return rec


class Ev:
    """A pair of timing events on the current stream."""

    def __init__(self, torch):
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def ms(self):
        return self.a.elapsed_time(self.b)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: there is no multi-GPU path (the kernels would shard by sequence or "
              "kv head with no exchange). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_35140_amd import inputs, uattn

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = "cuda"
    torch.cuda.set_device(0)
    uattn.lib()

    w = inputs.qwen_gqa()
    B, P, R = w.num_seqs, w.prompt_lens[0], w.response_lens[0]
    L = P + R
    hq, hkv, d, page, V = w.num_q_heads, w.num_kv_heads, w.head_dim, w.page_size, w.vocab

    # ------------------------------------------------------------------ inputs
    t0 = time.time()
    host = inputs.packed_qkv(w)
    cu = host["cu_seqlens"]

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    q, k, v = to_dev(host["q"]), to_dev(host["k"]), to_dev(host["v"])
    cu_dev = torch.from_numpy(cu).to(dev)
    table, npages = inputs.paged_layout(w.seq_lens, page)
    kp = to_dev(inputs.scatter_to_pages(host["k"], cu, table, npages, page))
    vp = to_dev(inputs.scatter_to_pages(host["v"], cu, table, npages, page))
    table_dev = torch.from_numpy(table).to(dev)
    # rollout prompt pack
    pidx = torch.from_numpy(np.concatenate([np.arange(cu[b], cu[b] + P) for b in range(B)])).to(dev)
    qp, kpk, vpk = q[pidx].contiguous(), k[pidx].contiguous(), v[pidx].contiguous()
    cu_p = torch.from_numpy(inputs.cu_seqlens([P] * B)).to(dev)
    # the rollout writes the prompt's K/V into the paged cache (same bits the cache already holds)
    seq_p = torch.from_numpy(np.repeat(np.arange(B, dtype=np.int32), P)).to(dev)
    pos_p = torch.from_numpy(np.tile(np.arange(P, dtype=np.int32), B)).to(dev)
    # Q/K RMSNorm + NeoX RoPE over the full trajectories (its own buffers; the attention inputs stay raw)
    pos_full = torch.from_numpy(np.concatenate([np.arange(n, dtype=np.int32) for n in w.seq_lens])).to(dev)
    qn_w = inputs.normal_bf16_device((d,), 1.0, 90, 0)
    kn_w = inputs.normal_bf16_device((d,), 1.0, 90, 1)
    cos_sin = uattn.rope_cache(L, d, 1e6)
    q_rope, k_rope = torch.empty_like(q), torch.empty_like(k)
    # decode steps: query of token P+s of every sequence; context P+s+1
    tok = torch.from_numpy((cu[:B][None, :] + P + np.arange(R)[:, None]).astype(np.int64)).to(dev)  # [R, B]
    q_steps = q[tok.reshape(-1)].reshape(R, B, hq, d).contiguous()
    seqlens_steps = torch.from_numpy(np.repeat((P + 1 + np.arange(R, dtype=np.int32))[:, None], B, axis=1)).to(dev)
    out_steps = torch.empty_like(q_steps)
    steps = uattn.DecodeSteps(q_steps, kp, vp, table_dev, seqlens_steps, L, out_steps)
    out_prompt = torch.empty_like(qp)
    out_full = torch.empty_like(q)
    lse_full = torch.empty((q.shape[0], hq), dtype=torch.float32, device=dev)
    # policy-update backward: upstream gradient ~ N(0,1), gradient buffers and workspace
    dout = inputs.normal_bf16_device(tuple(q.shape), 1.0, 7, 3)
    dq_b, dk_b, dv_b = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    bwd_ws = torch.empty(uattn.prefill_backward_workspace_bytes(q.shape[0], hq), dtype=torch.uint8, device=dev)
    # log-prob leg: one row per response token
    rows = B * R
    # LM head: hidden states [rows, Hq*d] ~ N(0,1) and weights ~ N(0, sigma^2/H), so the
    # logits it produces are ~ N(0, logit_sigma^2); the log-prob leg reads them
    H = hq * d
    hidden = inputs.normal_bf16_device((rows, H), 1.0, 7, 1)
    lm_w = inputs.normal_bf16_device((V, H), w.logit_sigma / float(np.sqrt(H)), 7, 2)
    logits = torch.empty((rows, V), dtype=torch.bfloat16, device=dev)
    targets = torch.from_numpy(inputs.targets(rows, V)).to(dev)
    logp = torch.empty(rows, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    log(f"inputs ready in {time.time() - t0:.1f}s: T={q.shape[0]} pages={npages} logits={tuple(logits.shape)}")
    if args.calibration_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        src.fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("calibration copy: 1 GiB device to device")

    # ------------------------------------------------------------------ one step
    # The 3072 token-wise decode launches run as one HIP graph (captured once,
    # untimed), so the decode phase is not bound by host launch latency; every
    # launch in it is a full uattn_decode call on the step's resident inputs.
    graph = None
    if not args.eager_decode:
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cap):
            for s_ in range(R):
                steps.run(s_, stream=cap)
        torch.cuda.synchronize()

    def step(ev):
        ev["pre"].a.record()
        uattn.prefill(qp, kpk, vpk, cu_p, P, out=out_prompt)
        ev["pre"].b.record()
        ev["kvw"].a.record()
        uattn.kv_write(kpk, vpk, table_dev, seq_p, pos_p, kp, vp)
        ev["kvw"].b.record()
        ev["dec"].a.record()
        if graph is not None:
            graph.replay()
        else:
            for s_ in range(R):
                steps.run(s_)
        ev["dec"].b.record()
        ev["nr"].a.record()
        uattn.qk_norm_rope(q, k, pos_full, qn_w, kn_w, cos_sin, q_out=q_rope, k_out=k_rope)
        ev["nr"].b.record()
        ev["upd"].a.record()
        uattn.prefill(q, k, v, cu_dev, L, out=out_full, lse=lse_full)
        ev["upd"].b.record()
        ev["bwd"].a.record()
        uattn.prefill_backward(q, k, v, out_full, dout, lse_full, cu_dev, L, dq=dq_b, dk=dk_b, dv=dv_b,
                               workspace=bwd_ws)
        ev["bwd"].b.record()
        ev["lm"].a.record()
        uattn.lm_head(hidden, lm_w, out=logits)
        ev["lm"].b.record()
        ev["lp"].a.record()
        uattn.logprob(logits, targets, out=logp)
        ev["lp"].b.record()

    def new_events():
        return {"pre": Ev(torch), "kvw": Ev(torch), "nr": Ev(torch), "upd": Ev(torch), "lm": Ev(torch),
                "lp": Ev(torch), "dec": Ev(torch), "bwd": Ev(torch)}

    for i in range(args.warmup):
        step(new_events())
    torch.cuda.synchronize()
    evs = [new_events() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    log(f"timed {args.steps} steps in {wall:.3f}s")

    # ------------------------------------------------------------------ metrics
    K = args.steps
    pre_ms = sum(e["pre"].ms() for e in evs) / K
    upd_ms = sum(e["upd"].ms() for e in evs) / K
    bwd_ms = sum(e["bwd"].ms() for e in evs) / K
    lp_ms = sum(e["lp"].ms() for e in evs) / K
    kvw_ms = sum(e["kvw"].ms() for e in evs) / K
    nr_ms = sum(e["nr"].ms() for e in evs) / K
    lm_ms = sum(e["lm"].ms() for e in evs) / K
    dec_wall_ms = sum(e["dec"].ms() for e in evs) / K
    dec_kernel_ms = dec_wall_ms
    step_ms = wall / K * 1e3

    upd_flop = w.prefill_flop()
    pre_flop = float(B * 2.0 * d * hq * P * (P + 1))
    dec_bytes = w.decode_kv_bytes()
    lp_bytes = float(rows) * V * 2
    upd_tflops = upd_flop / (upd_ms * 1e-3) / 1e12
    # backward: five products per causal (query, key) pair (S recomputed, dP, dV, dK, dQ) = 2.5 x forward
    bwd_flop = 2.5 * upd_flop
    bwd_tflops = bwd_flop / (bwd_ms * 1e-3) / 1e12
    pre_tflops = pre_flop / (pre_ms * 1e-3) / 1e12
    dec_gbs_wall = dec_bytes / (dec_wall_ms * 1e-3) / 1e9
    lp_gbs = lp_bytes / (lp_ms * 1e-3) / 1e9
    kvw_bytes = float(B * P) * hkv * d * 2 * 2 * 2      # K and V rows read once and written once
    kvw_gbs = kvw_bytes / (kvw_ms * 1e-3) / 1e9
    nr_bytes = float(q.numel() + k.numel()) * 2 * 2    # every q and k element read once and written once
    nr_gbs = nr_bytes / (nr_ms * 1e-3) / 1e9
    lm_flop = 2.0 * rows * V * H
    lm_tflops = lm_flop / (lm_ms * 1e-3) / 1e12

    # ------------------------------------------------------------------ bitwise Eq. (1)
    full_bits = out_full.view(torch.int16)
    dec_rows = out_steps.view(torch.int16).reshape(R * B, hq, d)
    ref_rows = full_bits[tok.reshape(-1)]
    dec_eq = (dec_rows == ref_rows).all(dim=-1)                 # [(R*B), hq]
    pr_eq = (out_prompt.view(torch.int16) == full_bits[pidx]).all(dim=-1)
    n_rows = dec_eq.numel() + pr_eq.numel()
    n_match = int(dec_eq.sum().item()) + int(pr_eq.sum().item())
    bitwise_pct = 100.0 * n_match / n_rows
    # unit reuse ratio of the decoded rows' log-probs is implied by bit equality of
    # the rows; here also check the log-prob leg itself is batch invariant on a sample
    sub = ua_rows = torch.arange(0, rows, max(1, rows // 64), device=dev)
    lp_sub = uattn.logprob(logits[sub].contiguous(), targets[sub].contiguous())
    ratio_one = bool(torch.equal(lp_sub.view(torch.int32), logp[sub].view(torch.int32)))
    del ua_rows
    log(f"bitwise rows {n_match}/{n_rows}; logprob batch-invariant: {ratio_one}")
    # the backward is deterministic: a second call into fresh buffers gives the same bits
    grads2 = uattn.prefill_backward(q, k, v, out_full, dout, lse_full, cu_dev, L, workspace=bwd_ws)
    bwd_repeat = all(bool(torch.equal(a.view(torch.int16), b.view(torch.int16)))
                     for a, b in zip((dq_b, dk_b, dv_b), grads2))
    del grads2
    log(f"backward repeat bitwise equal: {bwd_repeat}")

    # ------------------------------------------------------------------ CPU oracle baseline
    cpu = None
    cpu_rows = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, host, table, npages, args.cpu_seconds)
        cpu_rows = cpu_row_baselines(w, host, table, npages, args.cpu_row_seconds)

    dec_launch_bytes = dec_bytes / R
    dec_launch_ms = dec_kernel_ms / R
    traffic = measured_traffic()
    result = {
        "metric": METRIC,
        "value": round(dec_gbs_wall, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "qwen_gqa: 8 seqs x (1024 prompt + 3072 response), 32 q / 8 kv heads, head_dim 128, "
                        "bf16 N(0,0.25), page 64; logprob 24576 rows x vocab 151936, N(0,4)",
            "global_batch": B,
            "seq_len": L,
            "parallelism": "single GPU",
            "value_is": "decode KV GB/s over the decode phase (3072 token-wise uattn_decode launches, batch 8, "
                        "replayed as one HIP graph; HIP events around the phase)",
        },
        "roofline": {
            "kernel": "decode_kernel (uattn_decode; split-KV with fused merge)",
            "bound": "hbm",
            "achieved": round(dec_launch_bytes / (dec_launch_ms * 1e-3) / 1e9, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(dec_launch_bytes / (dec_launch_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "traffic": traffic["hbm_bytes_per_launch"] if traffic else None,
            "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "traffic_over_algorithmic": round(traffic["hbm_bytes_per_launch"] / dec_launch_bytes, 4) if traffic else None,
            "bytes_per_launch": dec_launch_bytes,
            "avg_launch_ms": round(dec_launch_ms, 5),
            "avg_launch_ms_is": "decode-phase event time / 3072 launches (includes the graph's inter-launch gaps)",
        },
        "roofline_prefill": {
            "kernel": "prefill_kernel (policy-update prefill over 8 x 4096)",
            "bound": "mfma",
            "achieved": round(upd_tflops, 2),
            "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(upd_tflops / BF16_PEAK_TFLOPS, 4),
            "flop_per_launch": upd_flop,
            "avg_launch_ms": round(upd_ms, 4),
        },
        "roofline_backward": {
            "kernel": "uattn_prefill_backward (bwd_prep + bwd_dkdv + bwd_dq over 8 x 4096)",
            "bound": "mfma",
            "achieved": round(bwd_tflops, 2),
            "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(bwd_tflops / BF16_PEAK_TFLOPS, 4),
            "flop_per_call": bwd_flop,
            "flop_is": "5 products x 2*d FLOP per causal (query, key) pair per q head (2.5 x the forward)",
            "avg_call_ms": round(bwd_ms, 4),
        },
        "phases_ms": {"prompt_prefill": round(pre_ms, 4), "kv_write": round(kvw_ms, 4), "decode": round(dec_wall_ms, 3),
                      "qk_norm_rope": round(nr_ms, 4), "lm_head": round(lm_ms, 4),
                      "update_prefill": round(upd_ms, 4), "update_backward": round(bwd_ms, 4),
                      "logprob": round(lp_ms, 4)},
        "prompt_prefill_tflops": round(pre_tflops, 2),
        "logprob_gbs": round(lp_gbs, 2),
        "logprob_frac_hbm": round(lp_gbs / HBM_PEAK_GBS, 4),
        "kv_write_gbs": round(kvw_gbs, 2),
        "kv_write_frac_hbm": round(kvw_gbs / HBM_PEAK_GBS, 4),
        "qk_norm_rope_gbs": round(nr_gbs, 2),
        "qk_norm_rope_frac_hbm": round(nr_gbs / HBM_PEAK_GBS, 4),
        "lm_head_tflops": round(lm_tflops, 2),
        "lm_head_frac_mfma": round(lm_tflops / BF16_PEAK_TFLOPS, 4),
        "bitwise_match_pct": round(bitwise_pct, 4),
        "bitwise_rows": [n_match, n_rows],
        "logprob_batch_invariant": ratio_one,
        "backward_repeat_bitwise": bwd_repeat,
        "cpu_baseline": cpu,
        "cpu_baselines_other_rows": cpu_rows,
    }
    print(json.dumps(result), flush=True)


def cpu_baseline(w, host, table, npages, budget_s):
    """The fp64 oracle's token-wise decode on a bounded sample of the same
    decode steps (one BLAS thread), in algorithmic KV GB/s."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    from paper_2609_35140_amd import inputs

    B, P, R = w.num_seqs, w.prompt_lens[0], w.response_lens[0]
    cu = host["cu_seqlens"]
    kp = inputs.scatter_to_pages(host["k"], cu, table, npages, w.page_size)
    vp = inputs.scatter_to_pages(host["v"], cu, table, npages, w.page_size)
    order = inputs.rng(11, 0).permutation(R)
    done_bytes, done_steps = 0.0, 0
    per_tok = 2 * w.num_kv_heads * w.head_dim * 2
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        for s in order:
            n = P + int(s) + 1
            qrows = host["q"][cu[:B] + n - 1]
            oracle.paged_decode_fp64(qrows, kp, vp, table, [n] * B)
            done_bytes += B * n * per_tok
            done_steps += 1
            if time.perf_counter() - t0 >= budget_s:
                break
        el = time.perf_counter() - t0
    log(f"cpu oracle: {done_steps} decode steps in {el:.1f}s")
    return {"value": round(done_bytes / el / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{done_steps} of the 3072 decode steps (random order, batch 8, 32 q heads) through "
                      f"oracle.paged_decode_fp64 in {el:.1f}s on 1 thread",
            "seconds": round(el, 2)}


def cpu_row_baselines(w, host, table, npages, budget_s):
    """The fp64 oracle of every other row of the step on a bounded sample of the
    same workload (one BLAS thread each), in the unit of that row's GPU figure.
    Each row repeats its sample until `budget_s` seconds have passed."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    from paper_2609_35140_amd import inputs

    hq, hkv, d, P = w.num_q_heads, w.num_kv_heads, w.head_dim, w.prompt_lens[0]
    grp = hq // hkv
    cu = host["cu_seqlens"]

    def timed(fn):
        n, t0 = 0, time.perf_counter()
        while True:
            fn()
            n += 1
            el = time.perf_counter() - t0
            if el >= budget_s:
                return n, el

    out = {}
    with threadpool_limits(limits=1):
        # prefill: the first 1024 positions of sequence 0, the 4 q heads of kv head 0
        n = 1024
        q = host["q"][:n, :grp]
        k = host["k"][:n, :1]
        v = host["v"][:n, :1]
        flop = 4.0 * d * grp * n * (n + 1) / 2
        reps, el = timed(lambda: oracle.causal_attention_fp64(q, k, v, [0, n]))
        out["prefill"] = {"value": round(flop * reps / el / 1e12, 6), "unit": "TFLOP/s",
                          "sample": f"oracle.causal_attention_fp64, 1 x {n} tokens x {grp} q heads, x{reps}"}
        # backward: 512 positions, same heads, N(0,1) upstream gradient
        n = 512
        do = inputs.normal_bf16((n, grp, d), 1.0, 7, 3)
        flop = 2.5 * 4.0 * d * grp * n * (n + 1) / 2
        reps, el = timed(lambda: oracle.attention_backward_fp64(host["q"][:n, :grp], host["k"][:n, :1],
                                                                 host["v"][:n, :1], do, [0, n]))
        out["update_backward"] = {"value": round(flop * reps / el / 1e12, 6), "unit": "TFLOP/s",
                                  "sample": f"oracle.attention_backward_fp64, 1 x {n} tokens x {grp} q heads, x{reps}"}
        # LM head: 16 rows x a 8192-entry vocabulary slice x hidden Hq*d
        H = hq * d
        hid = inputs.normal_bf16((16, H), 1.0, 7, 4)
        wt = inputs.normal_bf16((8192, H), w.logit_sigma / float(np.sqrt(H)), 7, 5)
        reps, el = timed(lambda: oracle.logits_fp64(hid, wt))
        out["lm_head"] = {"value": round(2.0 * 16 * 8192 * H * reps / el / 1e12, 6), "unit": "TFLOP/s",
                          "sample": f"oracle.logits_fp64, 16 rows x 8192 vocab x {H}, x{reps}"}
        # log-prob: 16 rows of the full vocabulary
        lg = inputs.logits_bf16(16, w.vocab, w.logit_sigma, tag=9)
        tg = inputs.targets(16, w.vocab, tag=9)
        reps, el = timed(lambda: oracle.logprob_fp64(lg, tg))
        out["logprob"] = {"value": round(16 * w.vocab * 2 * reps / el / 1e9, 4), "unit": "GB/s",
                          "sample": f"oracle.logprob_fp64, 16 rows x {w.vocab}, x{reps}"}
        # KV write: the prompt tokens of sequence 0 into a copy of the paged cache
        kp = inputs.scatter_to_pages(host["k"], cu, table, npages, w.page_size)
        vp = inputs.scatter_to_pages(host["v"], cu, table, npages, w.page_size)
        kn, vn = host["k"][:P], host["v"][:P]
        seq = np.zeros(P, dtype=np.int32)
        pos = np.arange(P, dtype=np.int32)
        reps, el = timed(lambda: oracle.kv_write(kp, vp, kn, vn, table, seq, pos))
        out["kv_write"] = {"value": round(P * hkv * d * 2 * 2 * 2 * reps / el / 1e9, 4), "unit": "GB/s",
                           "sample": f"oracle.kv_write, {P} tokens x {hkv} kv heads, x{reps}"}
        # Q/K RMSNorm + NeoX RoPE: 256 tokens of sequence 0
        n = 256
        cs = oracle.rope_table(n, d, 1e6)
        wq = inputs.normal_bf16((d,), 1.0, 90, 0)
        wk = inputs.normal_bf16((d,), 1.0, 90, 1)
        posn = np.arange(n)
        reps, el = timed(lambda: (oracle.qk_norm_rope(host["q"][:n], posn, wq, 1e-6, cs),
                                  oracle.qk_norm_rope(host["k"][:n], posn, wk, 1e-6, cs)))
        out["qk_norm_rope"] = {"value": round(n * (hq + hkv) * d * 2 * 2 * reps / el / 1e9, 4), "unit": "GB/s",
                               "sample": f"oracle.qk_norm_rope, {n} tokens x ({hq} + {hkv}) heads, x{reps}"}
    for v in out.values():
        v.update({"cores": 1, "kind": "oracle"})
    log("cpu oracle rows: " + ", ".join(f"{k} {v['value']} {v['unit']}" for k, v in out.items()))
    return out


if __name__ == "__main__":
    main()
