"""Device-side construction of the full-size workloads for the GPU tests.

The large packs (up to 4.5 M tokens, ~37 GB of queries) are drawn on the GPU
from seeded generators (``inputs.normal_bf16_device``), laid out in the
packed varlen format and scattered into a paged cache (HND pages, unwritten
slots filled with a bf16 NaN).  Harness only: it draws and places numbers
and holds none of the attention or log-prob arithmetic.  Rows the oracle
needs are copied back to the host.
"""
from __future__ import annotations

import numpy as np

from paper_2609_35140_amd import inputs

NAN_BF16 = 0x7FC0


def _torch():
    import torch
    return torch


def host_bits(t) -> np.ndarray:
    torch = _torch()
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


class DevicePack:
    """A packed varlen batch drawn on the GPU, plus its paged KV cache.

    With ``w.shared_prompt_group > 1`` the sequences of a group carry the same
    prompt tokens, and (``share_prompt_pages``) the group's full prompt pages
    are stored once and referenced by every member's block table, as a
    serving engine's prefix cache would.
    """

    def __init__(self, w, tag: int, seed: int = inputs.BASE_SEED, share_prompt_pages: bool = True, extra_pages: int = 7):
        torch = _torch()
        self.w = w
        hq, hkv, d = w.num_q_heads, w.num_kv_heads, w.head_dim
        lens = [int(x) for x in w.seq_lens]
        P = [int(x) for x in w.prompt_lens]
        self.cu = inputs.cu_seqlens(lens)
        cu = self.cu
        T = int(cu[-1])
        self.max_seqlen = max(lens)
        sig = w.sigma
        G = int(w.shared_prompt_group)
        if G > 1:
            self.q = torch.empty((T, hq, d), dtype=torch.bfloat16, device="cuda")
            self.k = torch.empty((T, hkv, d), dtype=torch.bfloat16, device="cuda")
            self.v = torch.empty((T, hkv, d), dtype=torch.bfloat16, device="cuda")
            for grp in range(w.num_seqs // G):
                p0 = P[grp * G]
                pq = inputs.normal_bf16_device((p0, hq, d), sig, tag, 1, grp, 0, seed=seed)
                pk = inputs.normal_bf16_device((p0, hkv, d), sig, tag, 1, grp, 1, seed=seed)
                pv = inputs.normal_bf16_device((p0, hkv, d), sig, tag, 1, grp, 2, seed=seed)
                for s in range(grp * G, grp * G + G):
                    lo = int(cu[s])
                    self.q[lo:lo + p0] = pq
                    self.k[lo:lo + p0] = pk
                    self.v[lo:lo + p0] = pv
            for s in range(w.num_seqs):
                lo, hi = int(cu[s]) + P[s], int(cu[s + 1])
                if hi > lo:
                    self.q[lo:hi] = inputs.normal_bf16_device((hi - lo, hq, d), sig, tag, 2, s, 0, seed=seed)
                    self.k[lo:hi] = inputs.normal_bf16_device((hi - lo, hkv, d), sig, tag, 2, s, 1, seed=seed)
                    self.v[lo:hi] = inputs.normal_bf16_device((hi - lo, hkv, d), sig, tag, 2, s, 2, seed=seed)
        else:
            self.q = inputs.normal_bf16_device((T, hq, d), sig, tag, 0, 0, seed=seed)
            self.k = inputs.normal_bf16_device((T, hkv, d), sig, tag, 0, 1, seed=seed)
            self.v = inputs.normal_bf16_device((T, hkv, d), sig, tag, 0, 2, seed=seed)
        self.cu_dev = torch.from_numpy(cu).cuda()

        # ---- block table over a shuffled pool of physical pages
        page = int(w.page_size)
        self.page = page
        npg = [(L + page - 1) // page for L in lens]
        shared = share_prompt_pages and G > 1
        n_pp = [P[s] // page if shared else 0 for s in range(w.num_seqs)]  # shared full prompt pages
        n_group_pages = sum(n_pp[g * G] for g in range(w.num_seqs // G)) if shared else 0
        own = [npg[s] - n_pp[s] for s in range(w.num_seqs)]
        total = n_group_pages + sum(own) + extra_pages
        perm = inputs.rng(9, tag, seed=seed).permutation(total).astype(np.int32)
        maxp = max(npg)
        table = np.full((w.num_seqs, maxp), -1, dtype=np.int32)
        pos = 0
        if shared:
            for grp in range(w.num_seqs // G):
                n = n_pp[grp * G]
                pages = perm[pos:pos + n]
                pos += n
                for s in range(grp * G, grp * G + G):
                    table[s, :n] = pages
        for s in range(w.num_seqs):
            table[s, n_pp[s]:npg[s]] = perm[pos:pos + own[s]]
            pos += own[s]
        self.table = table
        self.num_pages = total
        self.table_dev = torch.from_numpy(table).cuda()

        # ---- scatter K/V into pages: token t of sequence b at position j goes
        # to page table[b, j // page], slot j % page
        seq_of = np.repeat(np.arange(w.num_seqs, dtype=np.int64), lens)
        posn = np.arange(T, dtype=np.int64) - cu[:-1].astype(np.int64)[seq_of]
        pg = torch.from_numpy(table[seq_of, posn // page].astype(np.int64)).cuda()
        sl = torch.from_numpy(posn % page).cuda()
        nan = torch.tensor(NAN_BF16, dtype=torch.int16).view(torch.bfloat16).item()
        self.kp = torch.full((total, hkv, page, d), nan, dtype=torch.bfloat16, device="cuda")
        self.vp = torch.full((total, hkv, page, d), nan, dtype=torch.bfloat16, device="cuda")
        self.kp[pg, :, sl, :] = self.k
        self.vp[pg, :, sl, :] = self.v
        del pg, sl

    def decode_rows(self, entries):
        """Decode inputs for (sequence, position) entries: the query of token
        `position` of `sequence`, context position + 1, the sequence's block
        table row.  Returns (q, table, seqlens, max_seqlen, packed token ids)."""
        torch = _torch()
        seqs = np.array([s for s, _ in entries], dtype=np.int64)
        pos = np.array([p for _, p in entries], dtype=np.int64)
        tok = self.cu[seqs].astype(np.int64) + pos
        q = self.q[torch.from_numpy(tok).cuda()].contiguous()
        table = torch.from_numpy(np.ascontiguousarray(self.table[seqs])).cuda()
        seqlens = torch.from_numpy((pos + 1).astype(np.int32)).cuda()
        return q, table, seqlens, int(pos.max()) + 1, tok

    def host_sequence(self, s: int):
        """Q, K, V bits of sequence s (for oracle rows)."""
        lo, hi = int(self.cu[s]), int(self.cu[s + 1])
        return host_bits(self.q[lo:hi]), host_bits(self.k[lo:hi]), host_bits(self.v[lo:hi])
