"""Seeded synthetic workloads for the unified attention path.

This module only draws random numbers and lays them out; it holds none of
the attention or log-prob arithmetic.  Both the GPU path (through the
binding) and the CPU oracle consume what it produces, so it is the single
source of inputs for parity checks.

bf16 tensors are carried on the host as ``numpy.uint16`` bit patterns.

Workload shapes follow the five synthetic configurations of the build
(tiny, Qwen-style GQA, varlen training pack, GRPO rollout, long context),
which stand in for the paper's prefill/decode operator workloads
(Section 6, Q3) and its GSM8K rollouts (Section 6, Q1).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

BASE_SEED = 42


# --------------------------------------------------------------------------
# random streams
# --------------------------------------------------------------------------
def rng(*key: int, seed: int = BASE_SEED) -> np.random.Generator:
    """A PCG64 generator keyed by ``(seed, *key)``; identical on every host."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=tuple(int(k) for k in key))))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even) and return the bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    out = r.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(shape: Sequence[int], sigma: float, *key: int, seed: int = BASE_SEED) -> np.ndarray:
    """i.i.d. N(0, sigma^2) samples rounded to bf16, as uint16 bits."""
    g = rng(*key, seed=seed)
    x = g.standard_normal(size=tuple(shape), dtype=np.float32) * np.float32(sigma)
    return f32_to_bf16_bits(x)


# --------------------------------------------------------------------------
# workload descriptions
# --------------------------------------------------------------------------
@dataclasses.dataclass
class Workload:
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    sigma: float
    page_size: int
    prompt_lens: List[int]        # per sequence
    response_lens: List[int]      # per sequence (decoded tokens); 0 for prefill-only packs
    vocab: int = 0                # log-prob vocabulary (0: no log-prob leg)
    logit_sigma: float = 2.0
    shared_prompt_group: int = 1  # >1: groups of this many sequences share prompt tokens

    @property
    def seq_lens(self) -> List[int]:
        return [p + r for p, r in zip(self.prompt_lens, self.response_lens)]

    @property
    def num_seqs(self) -> int:
        return len(self.prompt_lens)

    @property
    def total_tokens(self) -> int:
        return int(sum(self.seq_lens))

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def prefill_flop(self) -> float:
        """Algorithmic causal FLOP: 4*d*Hq per (query, key) pair with key <= query."""
        d, hq = self.head_dim, self.num_q_heads
        return float(sum(2.0 * d * hq * L * (L + 1) for L in self.seq_lens))

    def decode_kv_bytes(self) -> float:
        """Algorithmic decode KV bytes over every response step: K and V once per kv head."""
        per_tok = 2 * self.num_kv_heads * self.head_dim * 2
        tot = 0.0
        for p, r in zip(self.prompt_lens, self.response_lens):
            # step s decodes token p+s with context p+s+1
            tot += per_tok * float(sum(range(p + 1, p + r + 1)))
        return tot


def tiny() -> Workload:
    return Workload("tiny", 2, 1, 64, 1.0, 16, [64], [64])


def qwen_gqa() -> Workload:
    return Workload("qwen_gqa", 32, 8, 128, 0.5, 64, [1024] * 8, [3072] * 8, vocab=151936)


def varlen_pack(seed: int = BASE_SEED) -> Workload:
    g = rng(3, 0, seed=seed)
    lens = [int(x) for x in g.integers(512, 8192, size=64, endpoint=True)]
    return Workload("varlen_pack", 40, 8, 128, 1.0, 64, lens, [0] * 64)


def grpo_rollout(seed: int = BASE_SEED) -> Workload:
    g = rng(4, 0, seed=seed)
    resp = [int(x) for x in g.integers(256, 15360, size=512, endpoint=True)]
    return Workload("grpo_rollout", 32, 8, 128, 0.5, 64, [1024] * 512, resp, shared_prompt_group=8)


def long_context() -> Workload:
    return Workload("long_context", 64, 8, 128, 0.5, 64, [32768 - 1024] * 8, [1024] * 8, vocab=151936)


WORKLOADS = {
    "tiny": tiny,
    "qwen_gqa": qwen_gqa,
    "varlen_pack": varlen_pack,
    "grpo_rollout": grpo_rollout,
    "long_context": long_context,
}


def custom(num_q_heads: int, num_kv_heads: int, head_dim: int, seq_lens: Sequence[int],
           sigma: float = 1.0, page_size: int = 64, prompt_lens: Optional[Sequence[int]] = None,
           name: str = "custom") -> Workload:
    seq_lens = [int(s) for s in seq_lens]
    if prompt_lens is None:
        prompt_lens = seq_lens
    prompt_lens = [int(p) for p in prompt_lens]
    resp = [s - p for s, p in zip(seq_lens, prompt_lens)]
    return Workload(name, num_q_heads, num_kv_heads, head_dim, sigma, page_size, prompt_lens, resp)


# --------------------------------------------------------------------------
# tensors
# --------------------------------------------------------------------------
def cu_seqlens(lens: Sequence[int]) -> np.ndarray:
    out = np.zeros(len(lens) + 1, dtype=np.int32)
    out[1:] = np.cumsum(np.asarray(lens, dtype=np.int64)).astype(np.int32)
    return out


def packed_qkv(w: Workload, seed: int = BASE_SEED, tag: int = 0) -> Dict[str, np.ndarray]:
    """Packed varlen Q [T,Hq,d], K/V [T,Hkv,d] as bf16 bits, plus cu_seqlens.

    Each sequence draws its own tensors from its own stream, so the values of
    a sequence do not depend on which other sequences share the pack.  With
    ``shared_prompt_group > 1`` the prompt tokens of each group are identical.
    """
    hq, hkv, d = w.num_q_heads, w.num_kv_heads, w.head_dim
    qs, ks, vs = [], [], []
    for s, (L, P) in enumerate(zip(w.seq_lens, w.prompt_lens)):
        grp = s // w.shared_prompt_group
        if w.shared_prompt_group > 1:
            pq = normal_bf16((P, hq, d), w.sigma, tag, 1, grp, 0, seed=seed)
            pk = normal_bf16((P, hkv, d), w.sigma, tag, 1, grp, 1, seed=seed)
            pv = normal_bf16((P, hkv, d), w.sigma, tag, 1, grp, 2, seed=seed)
            R = L - P
            rq = normal_bf16((R, hq, d), w.sigma, tag, 2, s, 0, seed=seed)
            rk = normal_bf16((R, hkv, d), w.sigma, tag, 2, s, 1, seed=seed)
            rv = normal_bf16((R, hkv, d), w.sigma, tag, 2, s, 2, seed=seed)
            qs.append(np.concatenate([pq, rq])); ks.append(np.concatenate([pk, rk])); vs.append(np.concatenate([pv, rv]))
        else:
            qs.append(normal_bf16((L, hq, d), w.sigma, tag, 0, s, 0, seed=seed))
            ks.append(normal_bf16((L, hkv, d), w.sigma, tag, 0, s, 1, seed=seed))
            vs.append(normal_bf16((L, hkv, d), w.sigma, tag, 0, s, 2, seed=seed))
    return {
        "q": np.ascontiguousarray(np.concatenate(qs)),
        "k": np.ascontiguousarray(np.concatenate(ks)),
        "v": np.ascontiguousarray(np.concatenate(vs)),
        "cu_seqlens": cu_seqlens(w.seq_lens),
    }


def ramp_keys(t: Dict[str, np.ndarray], growth: float) -> Dict[str, np.ndarray]:
    """The same pack with every key row of a sequence scaled by
    (1 + position / growth) and rounded back to bf16: scores then grow along
    the sequence, so an online softmax meets tile maxima far above the ones
    before them (a stress case for the rescaling path)."""
    cu = t["cu_seqlens"]
    k = bf16_bits_to_f32(t["k"]).copy()
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        f = (1.0 + np.arange(hi - lo, dtype=np.float32) / np.float32(growth)).astype(np.float32)
        k[lo:hi] *= f[:, None, None]
    out = dict(t)
    out["k"] = np.ascontiguousarray(f32_to_bf16_bits(k))
    return out


def paged_layout(seq_lens: Sequence[int], page_size: int, seed: int = BASE_SEED, tag: int = 0,
                 extra_pages: int = 0, max_pages_per_seq: Optional[int] = None) -> Tuple[np.ndarray, int]:
    """A block table [B, maxp] (int32) over a shuffled pool of physical pages.

    Logical page j of sequence b lives in physical page ``table[b, j]``; entries
    past a sequence's last page are -1.  Returns (table, num_physical_pages).
    """
    npages = [(int(L) + page_size - 1) // page_size for L in seq_lens]
    maxp = max(npages) if max_pages_per_seq is None else int(max_pages_per_seq)
    total = int(sum(npages)) + int(extra_pages)
    perm = rng(9, tag, seed=seed).permutation(total).astype(np.int32)
    table = np.full((len(seq_lens), maxp), -1, dtype=np.int32)
    pos = 0
    for b, n in enumerate(npages):
        table[b, :n] = perm[pos:pos + n]
        pos += n
    return table, total


def scatter_to_pages(x: np.ndarray, cu: np.ndarray, table: np.ndarray, num_pages: int, page_size: int,
                     fill_bits: int = 0x7FC0) -> np.ndarray:
    """Lay packed [T,H,d] rows into a paged cache [P,H,page,d] (HND).

    Slots that hold no token are filled with ``fill_bits`` (a bf16 NaN by
    default) so that any read of an unwritten slot shows up in the results.
    """
    T, H, d = x.shape
    pages = np.full((num_pages, H, page_size, d), fill_bits, dtype=np.uint16)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        for j in range(0, hi - lo, page_size):
            n = min(page_size, hi - lo - j)
            p = int(table[b, j // page_size])
            pages[p, :, :n, :] = np.transpose(x[lo + j:lo + j + n], (1, 0, 2))
    return pages


def logits_bf16(rows: int, vocab: int, sigma: float, seed: int = BASE_SEED, tag: int = 0) -> np.ndarray:
    return normal_bf16((rows, vocab), sigma, 7, tag, seed=seed)


def targets(rows: int, vocab: int, seed: int = BASE_SEED, tag: int = 0) -> np.ndarray:
    return rng(8, tag, seed=seed).integers(0, vocab, size=rows).astype(np.int32)


# --------------------------------------------------------------------------
# device-side generation (large workloads; same recipe, torch's seeded Philox)
# --------------------------------------------------------------------------
def normal_bf16_device(shape, sigma: float, *key: int, seed: int = BASE_SEED, device="cuda", chunk_elems: int = 1 << 28):
    """i.i.d. N(0, sigma^2) bf16 tensor drawn on the GPU from a generator
    seeded by (seed, *key).  Used where host generation would take minutes
    (billions of logits, multi-GB packs); the values are copied back to the
    host wherever the oracle needs them."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(rng(*key, seed=seed).integers(0, 2 ** 62)))
    out = torch.empty(tuple(shape), dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    n = flat.numel()
    for lo in range(0, n, chunk_elems):
        hi = min(n, lo + chunk_elems)
        tmp = torch.randn(hi - lo, generator=g, device=device, dtype=torch.float32)
        flat[lo:hi] = (tmp * sigma).to(torch.bfloat16)
        del tmp
    return out


NAN_BF16 = 0x7FC0


def host_bits(t) -> np.ndarray:
    """bf16 device tensor -> its bits on the host (numpy uint16)."""
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


class DevicePack:
    """A packed varlen batch drawn on the GPU, plus its paged KV cache.

    With ``w.shared_prompt_group > 1`` the sequences of a group carry the same
    prompt tokens, and (``share_prompt_pages``) the group's full prompt pages
    are stored once and referenced by every member's block table, as a
    serving engine's prefix cache would.
    """

    def __init__(self, w, tag: int, seed: int = BASE_SEED, share_prompt_pages: bool = True, extra_pages: int = 7,
                 build_pages: bool = True):
        import torch
        self.w = w
        hq, hkv, d = w.num_q_heads, w.num_kv_heads, w.head_dim
        lens = [int(x) for x in w.seq_lens]
        P = [int(x) for x in w.prompt_lens]
        self.cu = cu_seqlens(lens)
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
                pq = normal_bf16_device((p0, hq, d), sig, tag, 1, grp, 0, seed=seed)
                pk = normal_bf16_device((p0, hkv, d), sig, tag, 1, grp, 1, seed=seed)
                pv = normal_bf16_device((p0, hkv, d), sig, tag, 1, grp, 2, seed=seed)
                for s in range(grp * G, grp * G + G):
                    lo = int(cu[s])
                    self.q[lo:lo + p0] = pq
                    self.k[lo:lo + p0] = pk
                    self.v[lo:lo + p0] = pv
            for s in range(w.num_seqs):
                lo, hi = int(cu[s]) + P[s], int(cu[s + 1])
                if hi > lo:
                    self.q[lo:hi] = normal_bf16_device((hi - lo, hq, d), sig, tag, 2, s, 0, seed=seed)
                    self.k[lo:hi] = normal_bf16_device((hi - lo, hkv, d), sig, tag, 2, s, 1, seed=seed)
                    self.v[lo:hi] = normal_bf16_device((hi - lo, hkv, d), sig, tag, 2, s, 2, seed=seed)
        else:
            self.q = normal_bf16_device((T, hq, d), sig, tag, 0, 0, seed=seed)
            self.k = normal_bf16_device((T, hkv, d), sig, tag, 0, 1, seed=seed)
            self.v = normal_bf16_device((T, hkv, d), sig, tag, 0, 2, seed=seed)
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
        perm = rng(9, tag, seed=seed).permutation(total).astype(np.int32)
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

        self.kp = self.vp = None
        if build_pages:
            self.kp, self.vp = self.pages(self.k, self.v)

    def pages(self, k, v):
        """Paged copies [num_pages, Hkv, page, d] of packed k, v [T, Hkv, d]:
        token t of sequence b at position j goes to page table[b, j // page],
        slot j % page; slots no token maps to hold a bf16 NaN."""
        import torch
        w, page, T = self.w, self.page, int(self.cu[-1])
        lens = [int(x) for x in w.seq_lens]
        seq_of = np.repeat(np.arange(w.num_seqs, dtype=np.int64), lens)
        posn = np.arange(T, dtype=np.int64) - self.cu[:-1].astype(np.int64)[seq_of]
        pg = torch.from_numpy(self.table[seq_of, posn // page].astype(np.int64)).cuda()
        sl = torch.from_numpy(posn % page).cuda()
        nan = torch.tensor(NAN_BF16, dtype=torch.int16).view(torch.bfloat16).item()
        shape = (self.num_pages, w.num_kv_heads, page, w.head_dim)
        kp = torch.full(shape, nan, dtype=torch.bfloat16, device="cuda")
        vp = torch.full(shape, nan, dtype=torch.bfloat16, device="cuda")
        kp[pg, :, sl, :] = k
        vp[pg, :, sl, :] = v
        return kp, vp

    def decode_rows(self, entries):
        """Decode inputs for (sequence, position) entries: the query of token
        `position` of `sequence`, context position + 1, the sequence's block
        table row.  Returns (q, table, seqlens, max_seqlen, packed token ids)."""
        import torch
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
