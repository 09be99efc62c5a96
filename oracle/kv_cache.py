"""Indexed paged KV-cache write -- TEST INFRASTRUCTURE ONLY (CPU oracle).

The rollout-only operator whose post-write cache state the paper checks
exactly (Section 6 Q3 and its table of prescribed bitwise checks): new key
and value rows of a batch of tokens are copied into the paged cache at the
slot that the sequence's block table assigns to each token's position;
every other slot keeps its bits.  Written from that definition with plain
loops; shares nothing with the GPU kernel.
"""
from __future__ import annotations

import numpy as np


def kv_write(k_pages: np.ndarray, v_pages: np.ndarray, k_new: np.ndarray, v_new: np.ndarray,
             block_table: np.ndarray, seq_idx, positions):
    """Caches after the write (copies; the inputs are not modified).

    k_pages, v_pages  [P, Hkv, page, d] (any dtype, bf16 bits as uint16)
    k_new, v_new      [N, Hkv, d]
    block_table       [B, maxp] int
    seq_idx, positions  [N] int; a token with position < 0, a sequence index
                      outside [0, B), a logical page outside the table or a
                      table entry outside [0, P) is not written
    Tokens are applied in order, so with two tokens on one slot the later wins.
    """
    kp = np.array(k_pages, copy=True)
    vp = np.array(v_pages, copy=True)
    P, _, page, _ = kp.shape
    B, maxp = block_table.shape
    for n in range(len(positions)):
        pos, s = int(positions[n]), int(seq_idx[n])
        if pos < 0 or not 0 <= s < B:
            continue
        logical = pos // page
        if logical >= maxp:
            continue
        phys = int(block_table[s, logical])
        if not 0 <= phys < P:
            continue
        slot = pos % page
        kp[phys, :, slot, :] = k_new[n]
        vp[phys, :, slot, :] = v_new[n]
    return kp, vp
