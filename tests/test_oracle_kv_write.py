"""Pins of the oracle's indexed KV-cache write (no GPU).

It is checked against (1) a hand-worked example with literal expected
pages, (2) the input module's independent packed-to-pages layout and the
oracle's paged reader, which must read back what was written, and (3) the
invariants that untouched slots keep their bits and that padding and
out-of-table tokens write nothing.
"""
import numpy as np

import oracle
from paper_2609_35140_amd import inputs


def test_hand_worked_example():
    # 3 physical pages of 2 slots, 1 head, d = 2; sequence 0 -> pages [2, 0], sequence 1 -> [1]
    kp = np.full((3, 1, 2, 2), 9, dtype=np.int32)
    vp = np.full((3, 1, 2, 2), 8, dtype=np.int32)
    table = np.array([[2, 0], [1, -1]])
    k_new = np.array([[[10, 11]], [[20, 21]], [[30, 31]], [[40, 41]], [[50, 51]]])
    v_new = -k_new
    seq = [0, 0, 1, 0, 1]
    pos = [0, 3, 1, -1, 2]      # token 3 is padding; token 4 falls on table entry -1
    k, v = oracle.kv_write(kp, vp, k_new, v_new, table, seq, pos)
    want_k = np.array([[[[9, 9], [20, 21]]],      # page 0: slot 1 <- seq 0 pos 3
                       [[[9, 9], [30, 31]]],      # page 1: slot 1 <- seq 1 pos 1
                       [[[10, 11], [9, 9]]]])     # page 2: slot 0 <- seq 0 pos 0
    assert np.array_equal(k, want_k)
    assert np.array_equal(v, np.where(want_k == 9, 8, -want_k))
    assert np.array_equal(kp, np.full((3, 1, 2, 2), 9))     # inputs untouched


def test_matches_independent_layout_and_reads_back():
    w = inputs.custom(4, 2, 64, [5, 37, 64, 100], sigma=1.0, page_size=16)
    t = inputs.packed_qkv(w, seed=3)
    cu = t["cu_seqlens"]
    table, npages = inputs.paged_layout(w.seq_lens, 16, seed=3, extra_pages=3)
    empty = np.full((npages, 2, 16, 64), 0x7FC0, dtype=np.uint16)
    seq = np.concatenate([np.full(L, b) for b, L in enumerate(w.seq_lens)])
    pos = np.concatenate([np.arange(L) for L in w.seq_lens])
    order = inputs.rng(5).permutation(len(pos))              # any token order gives the same state
    k, v = oracle.kv_write(empty, empty, t["k"][order], t["v"][order], table, seq[order], pos[order])
    assert np.array_equal(k, inputs.scatter_to_pages(t["k"], cu, table, npages, 16))
    assert np.array_equal(v, inputs.scatter_to_pages(t["v"], cu, table, npages, 16))
    for b, L in enumerate(w.seq_lens):
        for h in range(2):
            got = oracle.gather_paged(k, table[b], L, h)
            assert np.array_equal(got, t["k"][cu[b]:cu[b + 1], h])


def test_untouched_slots_and_skipped_tokens_keep_their_bits():
    g = inputs.rng(6)
    kp = g.integers(0, 2 ** 16, size=(6, 3, 16, 64), dtype=np.uint16)
    vp = g.integers(0, 2 ** 16, size=(6, 3, 16, 64), dtype=np.uint16)
    table = np.array([[4, 1, -1], [0, 7, 2]])
    k_new = g.integers(0, 2 ** 16, size=(5, 3, 64), dtype=np.uint16)
    v_new = g.integers(0, 2 ** 16, size=(5, 3, 64), dtype=np.uint16)
    seq = [1, 0, 0, 2, 1]
    pos = [33, 17, 40, -4, 20]   # token 2 -> table entry -1; token 3 -> no such sequence; token 4 -> page 7 >= P
    k, v = oracle.kv_write(kp, vp, k_new, v_new, table, seq, pos)
    changed = np.argwhere(np.any(k != kp, axis=-1))
    assert {tuple(x) for x in changed} <= {(2, h, 1) for h in range(3)} | {(1, h, 1) for h in range(3)}
    assert np.array_equal(k[2, :, 1], k_new[0]) and np.array_equal(v[2, :, 1], v_new[0])
    assert np.array_equal(k[1, :, 1], k_new[1]) and np.array_equal(v[1, :, 1], v_new[1])
    mask = np.ones(k.shape[:3], dtype=bool)
    mask[2, :, 1] = False
    mask[1, :, 1] = False
    assert np.array_equal(k[mask], kp[mask]) and np.array_equal(v[mask], vp[mask])
