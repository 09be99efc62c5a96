"""Paged-decode oracle and fp32 tile-order emulator, pinned on the CPU."""
import numpy as np
import pytest

import oracle
import oracle.attention as oa
from paper_2609_35140_amd import inputs


def _paged(w, t, seed=3):
    table, npages = inputs.paged_layout(w.seq_lens, w.page_size, seed=seed, extra_pages=3)
    kp = inputs.scatter_to_pages(t["k"], t["cu_seqlens"], table, npages, w.page_size)
    vp = inputs.scatter_to_pages(t["v"], t["cu_seqlens"], table, npages, w.page_size)
    return table, kp, vp


def test_paged_decode_equals_prefill_rows():
    """Decode of entry b (query token n-1 over cached keys 0..n-1) is the
    full-sequence row n-1 (Section 3.2, operator-level agreement); unwritten
    slots hold NaN, so any stray read would show."""
    w = inputs.custom(4, 2, 32, [70, 33, 129], sigma=1.0, page_size=16)
    t = inputs.packed_qkv(w)
    table, kp, vp = _paged(w, t)
    o_full, lse_full = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    cu = t["cu_seqlens"]
    for n_rel in [1, 5, 16, 17, 33]:
        seqlens = np.array([min(n_rel, L) for L in w.seq_lens], dtype=np.int32)
        q = np.stack([t["q"][cu[b] + seqlens[b] - 1] for b in range(3)])
        o, lse = oracle.paged_decode_fp64(q, kp, vp, table, seqlens)
        assert not np.isnan(o).any()
        for b in range(3):
            tok = cu[b] + seqlens[b] - 1
            assert np.max(np.abs(o[b] - o_full[tok])) < 1e-12
            assert np.max(np.abs(lse[b] - lse_full[tok])) < 1e-12


def test_gather_paged_roundtrip():
    w = inputs.custom(2, 2, 8, [5, 40, 17], page_size=16)
    t = inputs.packed_qkv(w)
    table, kp, _ = _paged(w, t)
    cu = t["cu_seqlens"]
    for b, L in enumerate(w.seq_lens):
        for h in range(2):
            g = oracle.gather_paged(kp, table[b], L, h)
            assert np.array_equal(g, t["k"][cu[b]:cu[b] + L, h])


@pytest.mark.parametrize("seed", [1, 42, 1023])
def test_emulator_within_gate_tiny(seed):
    """Tiny workload (128 tokens, 2/1 heads, d=64, N(0,1)): the fp32 tile-order
    emulation meets the parity gate against the fp64 definition."""
    w = inputs.tiny()
    t = inputs.packed_qkv(w, seed=seed)
    o64, lse64 = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    o32, lse32 = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"])
    rep = oracle.parity_report(o32, o64)
    assert rep["pass"], rep
    assert np.max(np.abs(lse32 - lse64)) < oracle.LSE_ABS


def test_emulator_multi_chunk_within_gate():
    """Contexts spanning several 256-key chunks and a ragged tail."""
    w = inputs.custom(2, 1, 64, [600, 300], sigma=0.5)
    t = inputs.packed_qkv(w)
    o64, _ = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    o32, _ = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"])
    rep = oracle.parity_report(o32, o64)
    assert rep["pass"], rep


def test_emulator_first_token_is_v_exactly():
    w = inputs.custom(2, 1, 64, [3, 1], sigma=1.0)
    t = inputs.packed_qkv(w)
    o32, _ = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"])
    vf = oracle.bf16_to_f64(t["v"])
    for tok in [0, 3]:
        for h in range(2):
            assert np.array_equal(o32[tok, h].astype(np.float64), vf[tok, 0])


def test_emulator_single_chunk_fold_is_identity():
    """Up to 256 keys the chunked result equals the unchunked one bit for bit."""
    w = inputs.custom(2, 1, 64, [256, 100], sigma=1.0)
    t = inputs.packed_qkv(w)
    a, la = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"], chunk=256)
    b, lb = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"], chunk=1 << 20)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_emulator_partition_changes_bits_only_within_tolerance():
    """Tile width and chunk size are numerics: changing them moves results by
    rounding only (both stay within the gate)."""
    w = inputs.custom(2, 1, 64, [700], sigma=1.0)
    t = inputs.packed_qkv(w)
    o64, _ = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    for bn, ch in [(64, 256), (128, 512), (64, 64), (32, 1 << 20)]:
        o32, _ = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"], bn=bn, chunk=ch)
        assert oracle.parity_report(o32, o64)["pass"], (bn, ch)


def test_emulator_rows_mode_matches_full_mode():
    w = inputs.custom(2, 1, 64, [300, 70], sigma=1.0)
    t = inputs.packed_qkv(w)
    full, lfull = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"])
    rows = [(0, 1), (63, 0), (64, 1), (255, 0), (256, 1), (299, 0), (300, 0), (369, 1)]
    o, l = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"], rows=rows)
    for r, (tok, h) in enumerate(rows):
        assert np.array_equal(o[r], full[tok, h])
        assert l[r] == lfull[tok, h]


def test_emulator_planted_mistakes_fail_gate(monkeypatch):
    """A dropped rescale or a skipped chunk fold in the emulation fails the gate."""
    w = inputs.custom(2, 1, 64, [600], sigma=1.0)
    t = inputs.packed_qkv(w)
    o64, _ = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    real = oa._emulate_rows

    def _last_chunk_only(qh, kh, vh, qpos, c, bn, chunk, slack=oa.MAX_SLACK):
        o = np.zeros((qh.shape[0], qh.shape[1]), dtype=np.float32)
        l = np.zeros(qh.shape[0], dtype=np.float32)
        for r in range(qh.shape[0]):
            start = (qpos[r] // chunk) * chunk
            oo, ll = real(qh[r:r + 1], kh[start:], vh[start:], np.array([qpos[r] - start]), c, bn, chunk, slack)
            o[r], l[r] = oo[0], ll[0]
        return o, l
    # keep only the last chunk's partial: a dropped fold term
    monkeypatch.setattr(oa, "_emulate_rows", _last_chunk_only)
    o32, _ = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"])
    assert not oracle.parity_report(o32, o64)["pass"]


def test_parity_gate_rejects_one_ulp_bias_everywhere():
    """The mean-abs term of the gate catches a systematic one-bf16-ulp shift."""
    w = inputs.tiny()
    t = inputs.packed_qkv(w)
    o64, _ = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    o32, _ = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"])
    bits = oracle.to_bf16_bits(o32).astype(np.int32)
    shifted = oracle.bf16_to_f64((bits + 1).astype(np.uint16))
    assert not oracle.parity_report(shifted, o64)["pass"]


def test_emulator_rising_scores_move_the_reference_within_gate():
    """Keys growing along the sequence push tile maxima far above the earlier
    ones (by more than 2^8 in the exp2 domain, inside and across chunks), so
    the rescale and fold paths carry real weight; the emulation still meets
    the gate against the fp64 definition, lse included."""
    w = inputs.custom(2, 1, 64, [700, 200], sigma=0.5)
    t = inputs.ramp_keys(inputs.packed_qkv(w), 16.0)
    qf, kf = oracle.bf16_to_f64(t["q"]), oracle.bf16_to_f64(t["k"])
    c = (1.0 / 8.0) * oa.LOG2E
    s = kf[:700, 0] @ qf[699, 0]
    tmax = [s[i:i + 64].max() for i in range(0, 700, 64)]
    jumps = [(tmax[i] - max(tmax[:i])) * c for i in range(1, len(tmax))]
    assert max(jumps) > 8.0, jumps   # the stress is real
    o64, lse64 = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    o32, lse32 = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"])
    rep = oracle.parity_report(o32, o64)
    assert rep["pass"], rep
    assert np.max(np.abs(lse32 - lse64)) < oracle.LSE_ABS



@pytest.mark.parametrize("sigma,ramp", [(1.0, 0.0), (0.5, 16.0)])
def test_emulator_reference_slack_changes_bits_only_within_tolerance(sigma, ramp):
    """The slack rule (the chunk's reference maximum moves only past a rise of
    2^8) and the textbook rule (it moves on every rise, slack 0) are the same
    mathematics: both emulations meet the gate against the fp64 definition,
    lse included, and they differ from each other only within it.  With the
    ramped keys the reference moves inside chunks under both rules."""
    w = inputs.custom(2, 1, 64, [700, 130], sigma=sigma)
    t = inputs.packed_qkv(w, seed=11)
    if ramp:
        t = inputs.ramp_keys(t, ramp)
    o64, lse64 = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    outs = {}
    for slack in (0.0, oa.MAX_SLACK):
        o32, lse32 = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"], slack=slack)
        rep = oracle.parity_report(o32, o64)
        assert rep["pass"], (slack, rep)
        assert np.max(np.abs(lse32 - lse64)) < oracle.LSE_ABS
        outs[slack] = (o32, lse32)
    d = np.abs(outs[0.0][0].astype(np.float64) - outs[oa.MAX_SLACK][0].astype(np.float64))
    assert np.all(d <= 2 * (oracle.MAX_ABS + oracle.REL_BF16 * np.abs(o64)))
    assert np.max(np.abs(outs[0.0][1] - outs[oa.MAX_SLACK][1])) < 2 * oracle.LSE_ABS


def test_emulator_slack_rule_is_exact_on_one_key_rows():
    """A first tile moves the reference from -inf under any slack: a row whose
    context is a single key returns that key's V exactly either way."""
    w = inputs.custom(2, 1, 64, [1, 1, 1], sigma=1.0)
    t = inputs.packed_qkv(w, seed=2)
    for slack in (0.0, oa.MAX_SLACK, 100.0):
        o32, _ = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], t["cu_seqlens"], slack=slack)
        assert np.array_equal(o32[:, 0].astype(np.float64), oracle.bf16_to_f64(t["v"])[:, 0])


def test_emulator_one_head_rows_equal_pack_rows():
    # the per-head entry (explicit context) gives the same bits as the pack entry
    w = inputs.custom(4, 2, 64, [700, 300], sigma=1.0)
    t = inputs.packed_qkv(w, seed=5)
    cu = t["cu_seqlens"]
    rows = [(cu[0] + 699, 3), (cu[0] + 256, 3), (cu[0] + 5, 3), (cu[1] + 299, 1)]
    o_ref, l_ref = oracle.tile_emulate_fp32(t["q"], t["k"], t["v"], cu, rows=rows)
    scale = oracle.default_scale(64)
    for i, (tok, h) in enumerate(rows):
        b = 0 if tok < cu[1] else 1
        lo = int(cu[b])
        o, l = oracle.tile_emulate_rows_fp32(t["q"][tok:tok + 1, h], t["k"][lo:cu[b + 1], h // 2],
                                             t["v"][lo:cu[b + 1], h // 2], [tok - lo], scale)
        assert np.array_equal(o[0].view(np.uint32), o_ref[i].view(np.uint32))
        assert np.float32(l[0]).view(np.uint32) == np.float32(l_ref[i]).view(np.uint32)
