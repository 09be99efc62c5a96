#!/usr/bin/env python3
"""Benchmark of the unified-attention hot path on one MI355X.

Headline workload: long context, 8 sequences of 32,768 tokens (31,744
prompt + 1,024 decoded), 64 q / 8 kv heads, head_dim 128, bf16 ~ N(0, 0.25),
paged KV with 64-token pages, log-prob over a 151,936-entry vocabulary.
One step = one pass of the whole path over that batch:

  1. rollout prefill over the 8 prompts            (full-sequence entry point)
     and the indexed write of the prompts' K/V into the paged cache
  2. rollout decode of the 1024 response tokens, token by token, batch 8,
     against the paged cache (token-wise entry point; the 1024 launches are
     replayed as one HIP graph captured before timing)
  3. Q/K RMSNorm + NeoX RoPE over the 8 full trajectories, then the
     policy-update prefill over them (full-sequence entry point) and its
     backward
  4. the batch-invariant LM head (hidden 8192 -> 151,936 logits) of the
     8 x 1024 response tokens fused with their log-probabilities, and the
     stand-alone log-probability over the same (stored) logits

Attention everywhere runs on the normalized, rotated Q/K (the rotated K is
what the paged cache holds and the decode queries are the rotated rows), so
the bitwise comparison covers the chain norm/RoPE -> attention in both
regimes.  Inputs are resident in HBM before the timed region.  Every phase
is bracketed by HIP events on the stream it runs on.  After timing, every
decoded row is compared bit for bit with the policy-update prefill row at
the same position (the paper's Eq. (1) at operator level), and the prompt
rows of the rollout prefill with the same rows of the full prefill.

Secondary figures in the same line: the Qwen-style GQA workload (8 x 4096,
32/8 heads; decode phase and prefill), the varlen training pack and the GRPO
rollout's full-pack prefill, measured streaming-read and MFMA ceilings, and
the CPU oracle timed on the host's cores.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys
import threading
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
    ap.add_argument("--workload", default="long_context", choices=["long_context", "qwen_gqa"],
                    help="headline workload (long_context is the reported one; qwen_gqa for profiling comparisons)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of each CPU-oracle sample")
    ap.add_argument("--no-secondary", action="store_true", help="skip the Qwen-style, varlen-pack and GRPO figures")
    ap.add_argument("--no-ceilings", action="store_true", help="skip the measured-ceiling microbenchmarks")
    ap.add_argument("--eager-decode", action="store_true", help="launch the decode steps one by one (no HIP graph)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="before timing, copy 1 GiB device to device once (the known-size dispatch that scales "
                         "the FETCH_SIZE / WRITE_SIZE counters of a profiling run)")
    return ap.parse_args()


DECODE_SOURCES = ("uattn_decode.hip", "uattn_numerics.h", "uattn_tile_io.h")


def decode_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in DECODE_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_35140_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per decode launch from the committed counter summary of this
    workload, or None when it is absent or was taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", f"decode_kernel_{workload}_traffic.md")
    try:
        with open(path) as f:
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
    """A pair of timing events, recorded on the current stream."""

    def __init__(self, torch):
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def ms(self):
        return self.a.elapsed_time(self.b)


def timed(torch, fn, reps):
    """Mean milliseconds of fn() over reps calls (one warm call first)."""
    fn()
    torch.cuda.synchronize()
    e = Ev(torch)
    e.a.record()
    for _ in range(reps):
        fn()
    e.b.record()
    torch.cuda.synchronize()
    return e.ms() / reps


def decode_graph(torch, steps, n):
    """The n decode launches of `steps` captured into one HIP graph."""
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cap):
        for s_ in range(n):
            steps.run(s_, stream=cap)
    torch.cuda.synchronize()
    return graph


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(prefill and decode would shard by sequence or kv head with no exchange). Run with --gpus 1.",
              file=sys.stderr)
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

    w = inputs.WORKLOADS[args.workload]()
    B, P, R = w.num_seqs, w.prompt_lens[0], w.response_lens[0]
    L = P + R
    hq, hkv, d, V = w.num_q_heads, w.num_kv_heads, w.head_dim, w.vocab

    # ------------------------------------------------------------------ inputs (device, seeded)
    t0 = time.time()
    pk = inputs.DevicePack(w, tag=205, build_pages=False)
    cu = pk.cu
    q_raw, k_raw, v = pk.q, pk.k, pk.v
    cu_dev = pk.cu_dev
    pos_full = torch.from_numpy(np.concatenate([np.arange(n, dtype=np.int32) for n in w.seq_lens])).to(dev)
    qn_w = inputs.normal_bf16_device((d,), 1.0, 90, 0)
    kn_w = inputs.normal_bf16_device((d,), 1.0, 90, 1)
    cos_sin = uattn.rope_cache(L, d, 1e6)
    # attention inputs: the normalized, rotated q and k (the timed norm/RoPE phase rewrites the same bits)
    q, k = uattn.qk_norm_rope(q_raw, k_raw, pos_full, qn_w, kn_w, cos_sin)
    kp, vp = pk.pages(k, v)
    table_dev = pk.table_dev
    # rollout prompt pack
    pidx = torch.from_numpy(np.concatenate([np.arange(cu[b], cu[b] + P) for b in range(B)])).to(dev)
    qp, kpk, vpk = q[pidx].contiguous(), k[pidx].contiguous(), v[pidx].contiguous()
    cu_p = torch.from_numpy(inputs.cu_seqlens([P] * B)).to(dev)
    seq_p = torch.from_numpy(np.repeat(np.arange(B, dtype=np.int32), P)).to(dev)
    pos_p = torch.from_numpy(np.tile(np.arange(P, dtype=np.int32), B)).to(dev)
    # decode steps: query of token P+s of every sequence; context P+s+1
    tok = torch.from_numpy((cu[:B][None, :] + P + np.arange(R)[:, None]).astype(np.int64)).to(dev)  # [R, B]
    q_steps = q[tok.reshape(-1)].reshape(R, B, hq, d).contiguous()
    seqlens_steps = torch.from_numpy(np.repeat((P + 1 + np.arange(R, dtype=np.int32))[:, None], B, axis=1)).to(dev)
    out_steps = torch.empty_like(q_steps)
    steps = uattn.DecodeSteps(q_steps, kp, vp, table_dev, seqlens_steps, L, out_steps)
    out_prompt = torch.empty_like(qp)
    out_full = torch.empty_like(q)
    lse_full = torch.empty((q.shape[0], hq), dtype=torch.float32, device=dev)
    q_rope, k_rope = torch.empty_like(q), torch.empty_like(k)
    # policy-update backward: upstream gradient ~ N(0,1), gradient buffers and workspace
    dout = inputs.normal_bf16_device(tuple(q.shape), 1.0, 7, 3)
    dq_b, dk_b, dv_b = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    bwd_ws = torch.empty(uattn.prefill_backward_workspace_bytes(q.shape[0], hq), dtype=torch.uint8, device=dev)
    # LM head + log-prob of the response tokens: hidden states [rows, Hq*d] ~ N(0,1), weights ~ N(0, sigma^2/H),
    # so the logits are ~ N(0, logit_sigma^2)
    rows = B * R
    H = hq * d
    hidden = inputs.normal_bf16_device((rows, H), 1.0, 7, 1)
    lm_w = inputs.normal_bf16_device((V, H), w.logit_sigma / float(np.sqrt(H)), 7, 2)
    logits = torch.empty((rows, V), dtype=torch.bfloat16, device=dev)
    targets = torch.from_numpy(inputs.targets(rows, V)).to(dev)
    logp = torch.empty(rows, dtype=torch.float32, device=dev)
    logp_fused = torch.empty(rows, dtype=torch.float32, device=dev)
    lmlp_ws = torch.empty(uattn.lm_head_logprob_workspace_bytes(rows, V), dtype=torch.uint8, device=dev)
    uattn.lm_head(hidden, lm_w, out=logits)  # the logits the stand-alone log-prob phase reads
    torch.cuda.synchronize()
    log(f"inputs ready in {time.time() - t0:.1f}s: {w.name} T={q.shape[0]} pages={pk.num_pages} logits={tuple(logits.shape)}")
    if args.calibration_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        src.fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("calibration copy: 1 GiB device to device")

    graph = None if args.eager_decode else decode_graph(torch, steps, R)

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
        uattn.qk_norm_rope(q_raw, k_raw, pos_full, qn_w, kn_w, cos_sin, q_out=q_rope, k_out=k_rope)
        ev["nr"].b.record()
        ev["upd"].a.record()
        uattn.prefill(q_rope, k_rope, v, cu_dev, L, out=out_full, lse=lse_full)
        ev["upd"].b.record()
        ev["bwd"].a.record()
        uattn.prefill_backward(q_rope, k_rope, v, out_full, dout, lse_full, cu_dev, L, dq=dq_b, dk=dk_b, dv=dv_b,
                               workspace=bwd_ws)
        ev["bwd"].b.record()
        ev["lm"].a.record()
        uattn.lm_head_logprob(hidden, lm_w, targets, out=logp_fused, workspace=lmlp_ws)
        ev["lm"].b.record()
        ev["lp"].a.record()
        uattn.logprob(logits, targets, out=logp)
        ev["lp"].b.record()

    names = ("pre", "kvw", "dec", "nr", "upd", "bwd", "lm", "lp")
    for _ in range(args.warmup):
        step({n: Ev(torch) for n in names})
    torch.cuda.synchronize()
    evs = [{n: Ev(torch) for n in names} for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    log(f"timed {args.steps} steps in {wall:.3f}s")

    # ------------------------------------------------------------------ metrics
    K = args.steps
    ph = {n: sum(e[n].ms() for e in evs) / K for n in names}
    step_ms = wall / K * 1e3
    upd_flop = w.prefill_flop()
    pre_flop = float(B * 2.0 * d * hq * P * (P + 1))
    dec_bytes = w.decode_kv_bytes()
    lp_bytes = float(rows) * V * 2
    bwd_flop = 2.5 * upd_flop   # five products per causal (query, key) pair: S recomputed, dP, dV, dK, dQ
    kvw_bytes = float(B * P) * hkv * d * 2 * 2 * 2      # K and V rows read once and written once
    nr_bytes = float(q.numel() + k.numel()) * 2 * 2    # every q and k element read once and written once
    lm_flop = 2.0 * rows * V * H
    tf = lambda flop, ms: flop / (ms * 1e-3) / 1e12
    gbs = lambda nbytes, ms: nbytes / (ms * 1e-3) / 1e9
    dec_gbs = gbs(dec_bytes, ph["dec"])
    upd_tflops = tf(upd_flop, ph["upd"])

    # ------------------------------------------------------------------ bitwise Eq. (1)
    full_bits = out_full.view(torch.int16)
    dec_eq = (out_steps.view(torch.int16).reshape(R * B, hq, d) == full_bits[tok.reshape(-1)]).all(dim=-1)
    n_dec, m_dec = dec_eq.numel(), int(dec_eq.sum().item())
    pr_eq = (out_prompt.view(torch.int16) == full_bits[pidx]).all(dim=-1)
    n_pr, m_pr = pr_eq.numel(), int(pr_eq.sum().item())
    rope_same = bool(torch.equal(q_rope.view(torch.int16), q.view(torch.int16))) and \
        bool(torch.equal(k_rope.view(torch.int16), k.view(torch.int16)))
    del dec_eq, pr_eq, full_bits
    sub = torch.arange(0, rows, max(1, rows // 64), device=dev)
    lp_sub = uattn.logprob(logits[sub].contiguous(), targets[sub].contiguous())
    ratio_one = bool(torch.equal(lp_sub.view(torch.int32), logp[sub].view(torch.int32)))
    lpf_sub = uattn.lm_head_logprob(hidden[sub].contiguous(), lm_w, targets[sub].contiguous())
    fused_ratio_one = bool(torch.equal(lpf_sub.view(torch.int32), logp_fused[sub].view(torch.int32)))
    fused_vs_two_call = float((logp_fused.double() - logp.double()).abs().max().item())
    lm_alone_ms = timed(torch, lambda: uattn.lm_head(hidden, lm_w, out=logits), 2)
    log(f"bitwise: decode rows {m_dec}/{n_dec}, prompt rows {m_pr}/{n_pr}; norm/RoPE repeat equal {rope_same}; "
        f"logprob batch-invariant {ratio_one}, fused {fused_ratio_one}; fused vs two-call max |d| {fused_vs_two_call:.3g}")
    grads2 = uattn.prefill_backward(q_rope, k_rope, v, out_full, dout, lse_full, cu_dev, L, workspace=bwd_ws)
    bwd_repeat = all(bool(torch.equal(a.view(torch.int16), b.view(torch.int16)))
                     for a, b in zip((dq_b, dk_b, dv_b), grads2))
    del grads2
    log(f"backward repeat bitwise equal: {bwd_repeat}")

    # host copies for the CPU oracle (a bounded sample of the same decode work)
    cpu_inputs = None
    if not args.no_cpu_baseline:
        cpu_inputs = {
            "kp": inputs.host_bits(kp), "vp": inputs.host_bits(vp), "table": pk.table,
            "q_steps": inputs.host_bits(q_steps), "P": P, "R": R, "B": B,
        }
    del pk, q_raw, k_raw, q, k, v, kp, vp, qp, kpk, vpk, q_steps, out_steps, out_prompt, out_full, lse_full
    del q_rope, k_rope, dout, dq_b, dk_b, dv_b, bwd_ws, hidden, lm_w, logits, steps, graph, lmlp_ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    dec_launch_bytes = dec_bytes / R
    dec_launch_ms = ph["dec"] / R
    traffic = measured_traffic(w.name)
    result = {
        "metric": METRIC,
        "value": round(dec_gbs, 2),
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
            "workload": (f"{w.name}: {B} seqs x {L} tokens ({P} prompt + {R} decoded), {hq} q / {hkv} kv heads, "
                         f"head_dim {d}, bf16 N(0,{w.sigma ** 2:g}), page {w.page_size}; logprob {rows} rows x vocab "
                         f"{V}, N(0,{w.logit_sigma ** 2:g})"),
            "global_batch": B,
            "seq_len": L,
            "parallelism": "single GPU",
            "value_is": (f"decode KV GB/s over the decode phase ({R} token-wise uattn_decode launches, batch {B}, "
                         f"replayed as one HIP graph; HIP events around the phase)"),
        },
        "roofline": {
            "kernel": ("uattn_decode = decode_kernel (persistent split-KV walk, partials buffered in LDS) + "
                       "decode_merge_kernel (chunk-order fold of the partials); a launch is one uattn_decode call"),
            "bound": "hbm",
            "achieved": round(gbs(dec_launch_bytes, dec_launch_ms), 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gbs(dec_launch_bytes, dec_launch_ms) / HBM_PEAK_GBS, 4),
            "traffic": traffic["hbm_bytes_per_launch"] if traffic else None,
            "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "traffic_over_algorithmic": round(traffic["hbm_bytes_per_launch"] / dec_launch_bytes, 4) if traffic else None,
            "bytes_per_launch": dec_launch_bytes,
            "avg_launch_ms": round(dec_launch_ms, 5),
            "avg_launch_ms_is": (f"decode-phase event time / {R} uattn_decode calls (both kernels and the graph's "
                                 f"inter-kernel gaps)"),
        },
        "roofline_prefill": {
            "kernel": f"prefill_kernel (policy-update prefill over {B} x {L})",
            "bound": "mfma",
            "achieved": round(upd_tflops, 2),
            "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(upd_tflops / BF16_PEAK_TFLOPS, 4),
            "flop_per_launch": upd_flop,
            "avg_launch_ms": round(ph["upd"], 4),
        },
        "roofline_backward": {
            "kernel": f"uattn_prefill_backward (bwd_prep + bwd_dkdv + bwd_dq over {B} x {L})",
            "bound": "mfma",
            "achieved": round(tf(bwd_flop, ph["bwd"]), 2),
            "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tf(bwd_flop, ph["bwd"]) / BF16_PEAK_TFLOPS, 4),
            "flop_per_call": bwd_flop,
            "flop_is": "5 products x 2*d FLOP per causal (query, key) pair per q head (2.5 x the forward)",
            "avg_call_ms": round(ph["bwd"], 4),
        },
        "phases_ms": {"prompt_prefill": round(ph["pre"], 4), "kv_write": round(ph["kvw"], 4),
                      "decode": round(ph["dec"], 3), "qk_norm_rope": round(ph["nr"], 4),
                      "lm_head_logprob_fused": round(ph["lm"], 4),
                      "update_prefill": round(ph["upd"], 4), "update_backward": round(ph["bwd"], 4),
                      "logprob": round(ph["lp"], 4)},
        "prompt_prefill_tflops": round(tf(pre_flop, ph["pre"]), 2),
        "logprob_gbs": round(gbs(lp_bytes, ph["lp"]), 2),
        "logprob_frac_hbm": round(gbs(lp_bytes, ph["lp"]) / HBM_PEAK_GBS, 4),
        "kv_write_gbs": round(gbs(kvw_bytes, ph["kvw"]), 2),
        "kv_write_frac_hbm": round(gbs(kvw_bytes, ph["kvw"]) / HBM_PEAK_GBS, 4),
        "qk_norm_rope_gbs": round(gbs(nr_bytes, ph["nr"]), 2),
        "qk_norm_rope_frac_hbm": round(gbs(nr_bytes, ph["nr"]) / HBM_PEAK_GBS, 4),
        "lm_head_logprob_fused_tflops": round(tf(lm_flop, ph["lm"]), 2),
        "lm_head_logprob_fused_frac_mfma": round(tf(lm_flop, ph["lm"]) / BF16_PEAK_TFLOPS, 4),
        "lm_head_alone_ms": round(lm_alone_ms, 4),
        "lm_head_alone_plus_logprob_ms": round(lm_alone_ms + ph["lp"], 4),
        "fused_logprob_batch_invariant": fused_ratio_one,
        "fused_vs_two_call_logprob_max_abs": fused_vs_two_call,
        "bitwise_match_pct": round(100.0 * m_dec / n_dec, 4),
        "bitwise_match_is": "decoded (token, q head) rows bit-identical to the full-sequence prefill row",
        "bitwise_decode_rows": [m_dec, n_dec],
        "bitwise_prompt_rows": [m_pr, n_pr],
        "bitwise_prompt_rows_are": "prompt-only rollout prefill rows vs the full-trajectory prefill at the same rows",
        "norm_rope_repeat_bitwise": rope_same,
        "logprob_batch_invariant": ratio_one,
        "backward_repeat_bitwise": bwd_repeat,
    }

    if not args.no_secondary:
        result["secondary"] = secondary(torch, np, inputs, uattn)
    if not args.no_ceilings:
        result["measured_ceilings"] = ceilings(result)
    if cpu_inputs is not None:
        result["cpu_baseline"] = cpu_baseline(w, cpu_inputs, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def secondary(torch, np, inputs, uattn):
    """Qwen-style GQA (decode phase and prefill), varlen-pack and GRPO-rollout
    full-pack prefill throughput, with the Qwen-style decode rows checked bit
    for bit against its prefill."""
    out = {}
    # Qwen-style GQA: 8 x (1024 + 3072), 32/8/128, page 64
    w = inputs.qwen_gqa()
    pk = inputs.DevicePack(w, tag=202)
    B, P, R = w.num_seqs, w.prompt_lens[0], w.response_lens[0]
    hq, d = w.num_q_heads, w.head_dim
    L = P + R
    tok = torch.from_numpy((pk.cu[:B][None, :] + P + np.arange(R)[:, None]).astype(np.int64)).cuda()
    q_steps = pk.q[tok.reshape(-1)].reshape(R, B, hq, d).contiguous()
    sl = torch.from_numpy(np.repeat((P + 1 + np.arange(R, dtype=np.int32))[:, None], B, axis=1)).cuda()
    out_steps = torch.empty_like(q_steps)
    steps = uattn.DecodeSteps(q_steps, pk.kp, pk.vp, pk.table_dev, sl, L, out_steps)
    graph = decode_graph(torch, steps, R)
    out_full = torch.empty_like(pk.q)
    pre_ms = timed(torch, lambda: uattn.prefill(pk.q, pk.k, pk.v, pk.cu_dev, L, out=out_full), 20)
    dec_ms = timed(torch, graph.replay, 5)
    eq = (out_steps.view(torch.int16).reshape(R * B, hq, d) == out_full.view(torch.int16)[tok.reshape(-1)]).all(-1)
    dec_bytes = w.decode_kv_bytes()
    out["qwen_gqa"] = {
        "workload": "8 seqs x (1024 prompt + 3072 decoded), 32 q / 8 kv heads, head_dim 128, bf16 N(0,0.25), page 64",
        "decode_gbs": round(dec_bytes / (dec_ms * 1e-3) / 1e9, 2),
        "decode_frac_hbm": round(dec_bytes / (dec_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "decode_launch_us": round(dec_ms / R * 1e3, 3),
        "decode_kv_set_mb": round(B * L * w.num_kv_heads * d * 2 * 2 / 1e6, 1),
        "decode_kv_set_note": "the whole KV cache fits the 256 MB Infinity Cache, so consecutive steps re-read cached pages",
        "prefill_tflops": round(w.prefill_flop() / (pre_ms * 1e-3) / 1e12, 2),
        "prefill_frac_mfma": round(w.prefill_flop() / (pre_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
        "prefill_ms": round(pre_ms, 4),
        "bitwise_decode_rows": [int(eq.sum().item()), eq.numel()],
    }
    log(f"secondary qwen_gqa: {out['qwen_gqa']}")
    del pk, q_steps, out_steps, steps, graph, out_full, eq
    torch.cuda.empty_cache()
    # full-pack prefill of the varlen training pack and of the GRPO rollout trajectories
    for name, mk, tag in (("varlen_pack", inputs.varlen_pack, 203), ("grpo_rollout", inputs.grpo_rollout, 204)):
        w = mk()
        pk = inputs.DevicePack(w, tag=tag, build_pages=False)
        o = torch.empty_like(pk.q)
        ms = timed(torch, lambda: uattn.prefill(pk.q, pk.k, pk.v, pk.cu_dev, pk.max_seqlen, out=o), 3)
        fl = w.prefill_flop()
        out[f"{name}_prefill"] = {"tokens": w.total_tokens, "flop": fl, "ms": round(ms, 3),
                                  "tflops": round(fl / (ms * 1e-3) / 1e12, 2),
                                  "frac_mfma": round(fl / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)}
        log(f"secondary {name} prefill: {out[f'{name}_prefill']}")
        del pk, o
        torch.cuda.empty_cache()
    return out


def ceilings(result):
    """Measured streaming-read and MFMA ceilings, and the headline fractions
    against them (besides the datasheet peaks)."""
    from paper_2609_35140_amd import ceilings as cl
    seq = max(cl.read_gbs(4 << 30, paged=False, nontemporal=nt) for nt in (False, True))
    paged = max(cl.read_gbs(4 << 30, block_bytes=16384, paged=True, nontemporal=nt) for nt in (False, True))
    mfma = cl.mfma_tflops()
    dec = result["roofline"]["achieved"]
    pre = result["roofline_prefill"]["achieved"]
    out = {"hbm_read_sequential_gbs": round(seq, 1), "hbm_read_paged_16kb_gbs": round(paged, 1),
           "mfma_bf16_tflops": round(mfma, 1),
           "decode_frac_of_paged_read": round(dec / paged, 4), "prefill_frac_of_measured_mfma": round(pre / mfma, 4),
           "method": "4 GiB buffer read once per launch (16-byte loads, 4 in flight per lane, XOR-folded), "
                     "contiguous or as 16 KB blocks in a random permutation, the faster of plain and non-temporal "
                     "loads; 8 independent "
                     "v_mfma_f32_16x16x32_bf16 chains per wave, 8 waves per CU, no memory traffic"}
    log(f"measured ceilings: {out}")
    return out


def cpu_model() -> str:
    try:
        txt = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in txt.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_pool(tasks, fn, threads, budget_s):
    """Run fn(task) over `tasks` on `threads` threads until the tasks or the
    time budget run out (a started task always finishes).  Returns the list
    of completed results and the elapsed seconds."""
    lock = threading.Lock()
    it = iter(tasks)
    done = []
    t0 = time.perf_counter()

    def worker():
        while True:
            if time.perf_counter() - t0 >= budget_s:
                return
            with lock:
                task = next(it, None)
            if task is None:
                return
            r = fn(task)
            with lock:
                done.append(r)

    ths = [threading.Thread(target=worker) for _ in range(threads)]
    for t in ths:
        t.start()
    for t in ths:
        t.join()
    return done, time.perf_counter() - t0


def cpu_baseline(w, ci, budget_s):
    """The CPU oracle on the host's cores, on bounded samples of the headline
    decode work: the fp64 definition (paged decode, one task per (step,
    entry)) and the fp32 tile-order emulator (one task per (entry, q head,
    8 steps)), each on all cores (one thread per core, one BLAS thread each).
    Rates are in work units of (row, key) pairs; seconds are extrapolated to
    every configuration's full prefill and decode sets by that ratio, and the
    tiny configuration is also run in full."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    from paper_2609_35140_amd import inputs

    threads = len(os.sched_getaffinity(0))
    hq, hkv, d = w.num_q_heads, w.num_kv_heads, w.head_dim
    grp = hq // hkv
    P, R, B = ci["P"], ci["R"], ci["B"]
    kp, vp, table, qs = ci["kp"], ci["vp"], ci["table"], ci["q_steps"]
    per_tok = 2 * hkv * d * 2
    g = inputs.rng(11, 0)
    scale = oracle.default_scale(d)

    # fp64 definition: decode entries of random steps
    tasks64 = [(int(s), b) for s in g.permutation(R) for b in range(B)]

    def f64(task):
        s, b = task
        n = P + s + 1
        oracle.paged_decode_fp64(qs[s, b:b + 1], kp, vp, table[b:b + 1], [n])
        return n

    with threadpool_limits(limits=1):
        done, el64 = run_pool(tasks64, f64, threads, budget_s)
    ctx64 = float(sum(done))
    gbs = ctx64 * per_tok / el64 / 1e9
    rate64 = ctx64 * hq / el64            # (row, key) pairs per second
    log(f"cpu oracle fp64: {len(done)} decode entries in {el64:.1f}s on {threads} threads ({gbs:.3f} GB/s)")

    # fp32 emulator: rows of one (entry, head) over 8 random steps at a time
    def keys_of(b, kvh, n):
        return oracle.gather_paged(kp, table[b], n, kvh), oracle.gather_paged(vp, table[b], n, kvh)

    steps8 = g.permutation(R)
    tasks32 = [(b, h, steps8[i:i + 8]) for i in range(0, R, 8) for b in range(B) for h in g.permutation(hq)[:4]]

    def f32(task):
        b, h, ss = task
        n = P + int(max(ss)) + 1
        kk, vv = keys_of(b, h // grp, n)
        oracle.tile_emulate_rows_fp32(qs[ss, b, h], kk, vv, [P + int(s) for s in ss], scale)
        return float(sum(P + int(s) + 1 for s in ss))

    with threadpool_limits(limits=1):
        done32, el32 = run_pool(tasks32, f32, threads, budget_s)
    rate32 = float(sum(done32)) / el32
    log(f"cpu emulator fp32: {len(done32)} tasks ({8 * len(done32)} rows) in {el32:.1f}s on {threads} threads")

    # work of every configuration's full sets, in (row, key) pairs
    def pairs(wl, decode_rows=None):
        pre = wl.num_q_heads * sum(L * (L + 1) / 2 for L in wl.seq_lens)
        if decode_rows is None:
            dec = wl.num_q_heads * sum(sum(range(p + 1, p + r + 1)) for p, r in zip(wl.prompt_lens, wl.response_lens))
        else:
            dec = decode_rows
        return pre, dec

    extrap = {}
    for name in ("tiny", "qwen_gqa", "varlen_pack", "grpo_rollout", "long_context"):
        wl = inputs.WORKLOADS[name]()
        if name == "varlen_pack":  # prefill only; its decode set is 4096 random tokens (mean context ~ L/2)
            pre, _ = pairs(wl)
            dec = wl.num_q_heads * 4096 * float(np.mean(wl.seq_lens)) / 2
        else:
            pre, dec = pairs(wl)
        extrap[name] = {"prefill_pairs": pre, "decode_pairs": dec,
                        "fp64_s": {"prefill": round(pre / rate64, 1), "decode": round(dec / rate64, 1)},
                        "fp32_emulator_s": {"prefill": round(pre / rate32, 1), "decode": round(dec / rate32, 1)}}
    # the tiny configuration in full, both oracles
    tw = inputs.tiny()
    t = inputs.packed_qkv(tw, seed=42)
    with threadpool_limits(limits=threads):
        a = time.perf_counter()
        oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
        tiny64 = time.perf_counter() - a
        a = time.perf_counter()
        oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"])
        tiny32 = time.perf_counter() - a
    extrap["tiny"]["measured_full_s"] = {"fp64": round(tiny64, 3), "fp32_emulator": round(tiny32, 3)}
    return {
        "value": round(gbs, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
        "cpu_model": cpu_model(),
        "sample": (f"{len(done)} decode entries (random steps of the {R}-step, batch-{B} decode, {hq} q heads, "
                   f"contexts {P + 1}..{P + R}) through oracle.paged_decode_fp64 in {el64:.1f}s, one task per thread "
                   f"on {threads} threads"),
        "seconds": round(el64, 2),
        "fp64_pairs_per_s": round(rate64, 1),
        "fp32_emulator": {"rows": 8 * len(done32), "seconds": round(el32, 2), "pairs_per_s": round(rate32, 1),
                          "sample": "rows of one (entry, q head) at 8 random decode steps per task, "
                                    "oracle.tile_emulate_rows_fp32 on the paged context"},
        "extrapolated": extrap,
        "extrapolation_is": "seconds = full-set (row, key) pairs / the sample's pairs per second; prefill sets "
                            "are every causal pair of the pack, decode sets every decoded row's context",
    }


if __name__ == "__main__":
    main()
