"""Helpers shared by the GPU tests: host<->device transfer of bf16 bit patterns
and the standard setups (packed pack, paged cache).  No attention arithmetic."""
from __future__ import annotations

import numpy as np


def torch_mod():
    import torch
    return torch


def dev(bits: np.ndarray):
    """uint16 bf16 bits -> bfloat16 CUDA tensor."""
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def dev_i32(x):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=np.int32))).cuda()


def host_bits(t) -> np.ndarray:
    torch = torch_mod()
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def host_f64(t) -> np.ndarray:
    """bf16 CUDA tensor -> exact float64 values."""
    b = host_bits(t).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def rows_equal_bits(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Per-row (last axis) strict bit equality of uint16 arrays."""
    return np.all(a == b, axis=-1)


class Pack:
    """A packed varlen batch on the GPU plus its paged cache."""

    def __init__(self, w, seed=42, tag=0, page_size=None, fill_bits=0x7FC0, extra_pages=5, table_slack=8,
                 key_ramp=None):
        from paper_2609_35140_amd import inputs
        self.w = w
        t = inputs.packed_qkv(w, seed=seed, tag=tag)
        if key_ramp is not None:
            t = inputs.ramp_keys(t, key_ramp)
        self.host = t
        self.cu = t["cu_seqlens"]
        self.q, self.k, self.v = dev(t["q"]), dev(t["k"]), dev(t["v"])
        self.cu_dev = dev_i32(self.cu)
        self.page = page_size or w.page_size
        maxp = max((L + self.page - 1) // self.page for L in w.seq_lens) + table_slack if w.seq_lens else 1
        table, npages = inputs.paged_layout(w.seq_lens, self.page, seed=seed, tag=tag, extra_pages=extra_pages,
                                            max_pages_per_seq=maxp)
        self.table = table
        self.kp_host = inputs.scatter_to_pages(t["k"], self.cu, table, npages, self.page, fill_bits)
        self.vp_host = inputs.scatter_to_pages(t["v"], self.cu, table, npages, self.page, fill_bits)
        self.kp, self.vp = dev(self.kp_host), dev(self.vp_host)
        self.table_dev = dev_i32(table)
        self.max_seqlen = max(w.seq_lens) if w.seq_lens else 0

    def decode_rows(self, entries):
        """Decode inputs for a list of (sequence, position) entries: entry i's
        query is token `position` of `sequence` with context position+1."""
        torch = torch_mod()
        seqs = np.array([s for s, _ in entries], dtype=np.int64)
        pos = np.array([p for _, p in entries], dtype=np.int64)
        tok = self.cu[seqs] + pos
        q = self.q[torch.from_numpy(tok).cuda()].contiguous()
        table = dev_i32(self.table[seqs])
        seqlens = dev_i32(pos + 1)
        return q, table, seqlens, int(pos.max()) + 1, tok
