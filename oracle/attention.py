"""CPU oracle for unified causal GQA attention (test infrastructure only).

This package is test infrastructure.  Only the tests, the smoke entry point
and the benchmark's CPU-baseline leg may import it; the product path never
does, and it shares no code with the HIP kernels or their binding.

Two oracles live here:

* ``causal_attention_fp64`` / ``attention_rows_fp64`` / ``paged_decode_fp64``
  -- the plain definition in float64.  Section 3.2 fixes what attention
  computes: scores Q K^T, normalized weights P = softmax(scores), output
  P V, with a causal prefix per query position (Section 3.1 holds tokens,
  positions and causal masking fixed; Section 4.1 has the full-sequence
  path process the whole trajectory under causal masking and the decode
  path read the same prefix from the KV cache).  Scores are scaled by the
  caller's ``scale`` (1/sqrt(d) by default).  The query head h reads KV
  head h // (Hq/Hkv) (grouped-query attention, contiguous groups).

* ``tile_emulate_fp32`` -- an fp32 emulation of the prescribed tile order
  that both GPU paths implement: 64-key tiles walked in ascending order,
  an online softmax whose rescaling points are the tile boundaries, P
  converted from FP32 to BF16 before the PV product (Section 3.2, first
  example of Insight 1), positional split chunks of 256 keys folded left to
  right, and one final normalization (Section 5.3, risks i-iv).  The
  normalizer l sums the same bf16-rounded weights that multiply V (the paper
  leaves what l sums open; this is the reading both GPU paths implement).  It is a
  diagnostic: the MFMA's internal summation order and the hardware exp2 are
  not reproduced, so it matches the GPU to tolerance, not bit for bit.

Inputs are bf16 bit patterns (numpy uint16) exactly as handed to the GPU.
"""
from __future__ import annotations

from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

LOG2E = 1.4426950408889634


# --------------------------------------------------------------------------
# bf16 <-> float helpers (the oracle's own)
# --------------------------------------------------------------------------
def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns as float64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    u = x32.view(np.uint32).astype(np.uint64)
    r = ((u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)) << np.uint64(16)
    y = r.astype(np.uint32).view(np.float32).copy()
    nanm = np.isnan(x32)
    if nanm.any():
        y[nanm] = np.float32(np.nan)
    return y


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    return (round_to_bf16(x).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _as_f64(x: np.ndarray) -> np.ndarray:
    return bf16_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, dtype=np.float64)


def default_scale(head_dim: int) -> float:
    return float(np.float32(1.0 / np.sqrt(head_dim)))


# --------------------------------------------------------------------------
# plain definition, float64
# --------------------------------------------------------------------------
def _one_head_causal(qh: np.ndarray, kh: np.ndarray, vh: np.ndarray, scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Causal softmax attention of one (sequence, head): rows i attend keys 0..i.

    qh [L,d], kh [L,d], vh [L,d] float64.  Returns (o [L,d], lse [L]).
    """
    L = qh.shape[0]
    s = (qh @ kh.T) * scale                        # scores (Section 3.2: Q K^T)
    s[np.triu(np.ones((L, L), dtype=bool), k=1)] = -np.inf   # key j > query i is not in the prefix
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(axis=1, keepdims=True)
    p = e / z                                      # P: normalized attention weights
    o = p @ vh                                     # P V
    lse = (m + np.log(z))[:, 0]
    return o, lse


def causal_attention_fp64(q: np.ndarray, k: np.ndarray, v: np.ndarray, cu_seqlens: Sequence[int],
                          scale: Optional[float] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Full-sequence causal GQA attention over a packed varlen batch.

    q [T,Hq,d], k/v [T,Hkv,d] (bf16 bits or float), cu_seqlens [B+1].
    Positions are sequence-relative: row i of a sequence sees its keys 0..i.
    Returns (o [T,Hq,d] float64, lse [T,Hq] float64 natural log of the sum
    of exp(scaled score)).
    """
    qf, kf, vf = _as_f64(q), _as_f64(k), _as_f64(v)
    T, hq, d = qf.shape
    hkv = kf.shape[1]
    if hq % hkv:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    g = hq // hkv
    if scale is None:
        scale = default_scale(d)
    o = np.zeros((T, hq, d), dtype=np.float64)
    lse = np.zeros((T, hq), dtype=np.float64)
    cu = [int(x) for x in cu_seqlens]
    for b in range(len(cu) - 1):
        lo, hi = cu[b], cu[b + 1]
        if hi <= lo:
            continue
        for h in range(hq):
            kvh = h // g
            oh, lh = _one_head_causal(qf[lo:hi, h], kf[lo:hi, kvh], vf[lo:hi, kvh], scale)
            o[lo:hi, h] = oh
            lse[lo:hi, h] = lh
    return o, lse


def attention_row_fp64(qrow: np.ndarray, keys: np.ndarray, vals: np.ndarray, scale: float) -> Tuple[np.ndarray, float]:
    """One query against an explicit context: qrow [d], keys/vals [n,d] (all visible)."""
    s = (keys @ qrow) * scale
    m = s.max()
    e = np.exp(s - m)
    z = e.sum()
    return (e / z) @ vals, float(m + np.log(z))


def attention_rows_fp64(q: np.ndarray, k: np.ndarray, v: np.ndarray, cu_seqlens: Sequence[int],
                        rows: Iterable[Tuple[int, int]], scale: Optional[float] = None) -> Tuple[np.ndarray, np.ndarray]:
    """The definition evaluated only at chosen (packed token index, q head) rows.

    Used to check full-size runs on a sample of outputs the oracle can
    compute one by one.
    """
    rows = list(rows)
    d = q.shape[2]
    hq, hkv = q.shape[1], k.shape[1]
    g = hq // hkv
    if scale is None:
        scale = default_scale(d)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    out = np.zeros((len(rows), d), dtype=np.float64)
    lse = np.zeros(len(rows), dtype=np.float64)
    for r, (t, h) in enumerate(rows):
        b = int(np.searchsorted(cu, t, side="right") - 1)
        lo = int(cu[b])
        qrow = _as_f64(q[t, h])
        keys = _as_f64(k[lo:t + 1, h // g])
        vals = _as_f64(v[lo:t + 1, h // g])
        out[r], lse[r] = attention_row_fp64(qrow, keys, vals, scale)
    return out, lse


def gather_paged(pages: np.ndarray, block_table_row: np.ndarray, n: int, head: int) -> np.ndarray:
    """Logical rows 0..n-1 of one sequence and kv head from an HND paged cache.

    pages [P, Hkv, page, d]; logical position j lives in physical page
    block_table_row[j // page] at slot j % page.
    """
    page = pages.shape[2]
    out = np.empty((n, pages.shape[3]), dtype=pages.dtype)
    for j0 in range(0, n, page):
        cnt = min(page, n - j0)
        out[j0:j0 + cnt] = pages[int(block_table_row[j0 // page]), head, :cnt]
    return out


def paged_decode_fp64(q: np.ndarray, k_pages: np.ndarray, v_pages: np.ndarray, block_table: np.ndarray,
                      seqlens: Sequence[int], scale: Optional[float] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Token-wise decode: entry b's query is token seqlens[b]-1 and attends the
    cached keys 0..seqlens[b]-1 (its own K/V already written).

    q [B,Hq,d]; k_pages/v_pages [P,Hkv,page,d]; block_table [B,maxp].
    Returns (o [B,Hq,d], lse [B,Hq]).
    """
    B, hq, d = q.shape
    hkv = k_pages.shape[1]
    g = hq // hkv
    if scale is None:
        scale = default_scale(d)
    o = np.zeros((B, hq, d), dtype=np.float64)
    lse = np.zeros((B, hq), dtype=np.float64)
    for b in range(B):
        n = int(seqlens[b])
        for kvh in range(hkv):
            keys = _as_f64(gather_paged(k_pages, block_table[b], n, kvh))
            vals = _as_f64(gather_paged(v_pages, block_table[b], n, kvh))
            for h in range(kvh * g, (kvh + 1) * g):
                o[b, h], lse[b, h] = attention_row_fp64(_as_f64(q[b, h]), keys, vals, scale)
    return o, lse


# --------------------------------------------------------------------------
# fp32 emulation of the prescribed tile order (diagnostic)
# --------------------------------------------------------------------------
TILE_KEYS = 64      # keys per tile (Section 3.2: the 64-key partition shared by both paths)
CHUNK_KEYS = 256    # keys per positional split chunk (multiple of the tile)
# The running maximum of a chunk is a reference that moves to a tile's maximum
# only when that exceeds it by more than MAX_SLACK in the exp2 domain (the
# prescribed rescale rule; 0 gives the textbook rule, which moves on any
# increase).  Weights then reach at most 2^MAX_SLACK.
MAX_SLACK = 8.0


def _f32(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float32)


def _emulate_rows(qh: np.ndarray, kh: np.ndarray, vh: np.ndarray, qpos: np.ndarray, c: np.float32,
                  bn: int, chunk: int, slack: float = MAX_SLACK) -> Tuple[np.ndarray, np.ndarray]:
    """Rows with query positions ``qpos`` (ascending not required) of one head.

    qh [R,d] float64 (exact bf16 values), kh/vh [>=max(qpos)+1, d] float64.
    Row with position i visits tiles 0..i//bn; tiles are grouped into chunks
    of chunk//bn tiles; each chunk starts from (m=-inf, l=0, acc=0) and its
    reference m moves to a tile's maximum t only when t*c - m*c > slack
    (alpha = exp2(m*c - t*c), else alpha = 1); chunk partials are folded left
    to right with the exact running maximum.  Returns (o float32 [R,d]
    rounded to bf16, lse float32 [R]).
    """
    R, d = qh.shape
    tiles_per_chunk = chunk // bn
    last_tile = qpos // bn
    n_chunks = last_tile // tiles_per_chunk + 1
    M = np.full(R, -np.inf, dtype=np.float32)
    Lsum = np.zeros(R, dtype=np.float32)
    A = np.zeros((R, d), dtype=np.float32)
    ninf = np.float32(-np.inf)
    for ck in range(int(n_chunks.max())):
        rows_c = np.nonzero(n_chunks > ck)[0]
        m = np.full(R, -np.inf, dtype=np.float32)
        l = np.zeros(R, dtype=np.float32)
        acc = np.zeros((R, d), dtype=np.float32)
        for t in range(ck * tiles_per_chunk, (ck + 1) * tiles_per_chunk):
            rows = rows_c[last_tile[rows_c] >= t]
            if rows.size == 0:
                break
            j0, j1 = t * bn, (t + 1) * bn
            kt = kh[j0:j1]
            vt = vh[j0:j1]
            if kt.shape[0] < bn:   # keys past the end of the context: zero rows (masked below)
                pad = bn - kt.shape[0]
                kt = np.concatenate([kt, np.zeros((pad, d))])
                vt = np.concatenate([vt, np.zeros((pad, d))])
            # scores: exact products summed, rounded once to fp32
            s = _f32(qh[rows] @ kt.T)
            keypos = np.arange(j0, j1)
            s = np.where(keypos[None, :] > qpos[rows][:, None], ninf, s).astype(np.float32)
            tmax = s.max(axis=1)
            mc_old = _f32(m[rows] * c)
            tc = _f32(tmax * c)
            with np.errstate(invalid="ignore"):
                move = _f32(tc - mc_old) > np.float32(slack)   # always from -inf
            m_new = np.where(move, tmax, m[rows]).astype(np.float32)
            mc_new = _f32(m_new * c)
            alpha = np.where(move, np.exp2(_f32(mc_old - tc)), np.float32(1.0)).astype(np.float32)
            # p = exp2(s*c - m_new*c), the product-difference evaluated as one fused op
            arg = _f32(s.astype(np.float64) * np.float64(c) - mc_new.astype(np.float64)[:, None])
            p = np.exp2(arg).astype(np.float32)
            pb = round_to_bf16(p).astype(np.float64)        # FP32 -> BF16 before PV
            # l sums the same bf16 weights that multiply V (one product, rounded once)
            rowsum = _f32(pb.sum(axis=1))
            l[rows] = _f32(_f32(alpha * l[rows]) + rowsum)
            pv = _f32(pb @ vt)
            acc[rows] = _f32(_f32(alpha[:, None] * acc[rows]) + pv)
            m[rows] = m_new
        # fold chunk ck into the running (M, L, A), left to right
        if ck == 0:
            M[rows_c], Lsum[rows_c], A[rows_c] = m[rows_c], l[rows_c], acc[rows_c]
        else:
            Mn = np.maximum(M[rows_c], m[rows_c])
            MCn = _f32(Mn * c)
            a = np.exp2(_f32(_f32(M[rows_c] * c) - MCn)).astype(np.float32)
            b = np.exp2(_f32(_f32(m[rows_c] * c) - MCn)).astype(np.float32)
            Lsum[rows_c] = _f32(_f32(a * Lsum[rows_c]) + _f32(b * l[rows_c]))
            A[rows_c] = _f32(_f32(a[:, None] * A[rows_c]) + _f32(b[:, None] * acc[rows_c]))
            M[rows_c] = Mn
    o = round_to_bf16(_f32(A / Lsum[:, None]))
    lse = _f32(_f32(_f32(M * c) + _f32(np.log2(Lsum))) * np.float32(np.log(2.0)))
    return o, lse


def tile_emulate_fp32(q: np.ndarray, k: np.ndarray, v: np.ndarray, cu_seqlens: Sequence[int],
                      scale: Optional[float] = None, bn: int = TILE_KEYS, chunk: int = CHUNK_KEYS,
                      rows: Optional[Iterable[Tuple[int, int]]] = None,
                      slack: float = MAX_SLACK) -> Tuple[np.ndarray, np.ndarray]:
    """fp32 emulation of the prescribed tile order over a packed batch.

    With ``rows`` None every (token, head) row is produced, shapes as in
    ``causal_attention_fp64`` (o is float32 holding bf16-representable
    values).  With ``rows`` given, returns (o [R,d], lse [R]) for those rows.
    """
    qf, kf, vf = _as_f64(q), _as_f64(k), _as_f64(v)
    T, hq, d = qf.shape
    hkv = kf.shape[1]
    g = hq // hkv
    if scale is None:
        scale = default_scale(d)
    c = np.float32(np.float64(np.float32(scale)) * LOG2E)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    if rows is None:
        o = np.zeros((T, hq, d), dtype=np.float32)
        lse = np.zeros((T, hq), dtype=np.float32)
        for b in range(len(cu) - 1):
            lo, hi = int(cu[b]), int(cu[b + 1])
            if hi <= lo:
                continue
            qpos = np.arange(hi - lo)
            for h in range(hq):
                oh, lh = _emulate_rows(qf[lo:hi, h], kf[lo:hi, h // g], vf[lo:hi, h // g], qpos, c, bn, chunk,
                                       slack)
                o[lo:hi, h], lse[lo:hi, h] = oh, lh
        return o, lse
    rows = list(rows)
    o = np.zeros((len(rows), d), dtype=np.float32)
    lse = np.zeros(len(rows), dtype=np.float32)
    for r, (t, h) in enumerate(rows):
        b = int(np.searchsorted(cu, t, side="right") - 1)
        lo = int(cu[b])
        oo, ll = _emulate_rows(qf[t:t + 1, h], kf[lo:t + 1, h // g], vf[lo:t + 1, h // g],
                               np.array([t - lo]), c, bn, chunk, slack)
        o[r], lse[r] = oo[0], ll[0]
    return o, lse


def tile_emulate_rows_fp32(qrows: np.ndarray, keys: np.ndarray, vals: np.ndarray, qpos: Sequence[int],
                           scale: float, bn: int = TILE_KEYS, chunk: int = CHUNK_KEYS,
                           slack: float = MAX_SLACK) -> Tuple[np.ndarray, np.ndarray]:
    """The fp32 tile-order emulation for rows of ONE head against an explicit
    context (the emulator's counterpart of ``attention_row_fp64``).

    qrows [R,d] (bf16 bits or float), keys/vals [n,d] with n > max(qpos):
    row r attends keys 0..qpos[r].  Returns (o [R,d] float32 holding bf16
    values, lse [R] float32), exactly what ``tile_emulate_fp32`` gives for
    the same rows.
    """
    qpos = np.asarray(qpos, dtype=np.int64)
    c = np.float32(np.float64(np.float32(scale)) * LOG2E)
    return _emulate_rows(_as_f64(qrows), _as_f64(keys), _as_f64(vals), qpos, c, bn, chunk, slack)


# --------------------------------------------------------------------------
# the parity gate
# --------------------------------------------------------------------------
MAX_ABS = 4e-3
MEAN_ABS = 5e-4
REL_BF16 = 2.0 ** -8
# lse: the normalizer is the sum of the bf16-rounded weights.  bf16 has an
# 8-bit significand, so round-to-nearest leaves each weight within 2^-8
# (relative) of its fp32 value and |log L' - log L| <= -log(1 - 2^-8)
# = 3.91e-3; fp32 rounding of the sum, of M*c and of the logarithm adds
# about 1e-5.  (With the textbook rescale rule the largest weight is exactly
# 1 and the bound is rarely approached; with the slack rule it can be.)
LSE_ABS = 4.0e-3


def parity_report(o_test: np.ndarray, o_ref64: np.ndarray) -> dict:
    """Compare a bf16-valued result with the fp64 definition.

    Gate: mean |err| <= 5e-4 and, per element, |err| <= 4e-3 + 2^-8 |ref|
    (the literal 4e-3 plus one bf16 unit of the reference's magnitude, since
    bf16 cannot hold values above 1 to within 4e-3).  The literal max-abs
    figure and the count of elements above 4e-3 are reported alongside, as
    is the count where even the correctly rounded reference exceeds 4e-3.
    """
    t = np.asarray(o_test, dtype=np.float64)
    r = np.asarray(o_ref64, dtype=np.float64)
    err = np.abs(t - r)
    bound = MAX_ABS + REL_BF16 * np.abs(r)
    floor = np.abs(round_to_bf16(r.astype(np.float32)).astype(np.float64) - r)
    n = err.size
    return {
        "n": int(n),
        "max_abs": float(err.max()) if n else 0.0,
        "mean_abs": float(err.mean()) if n else 0.0,
        "n_over_4e-3": int((err > MAX_ABS).sum()),
        "n_rounding_floor_over_4e-3": int((floor > MAX_ABS).sum()),
        "n_over_bound": int((err > bound).sum()),
        "nan": int(np.isnan(t).sum()),
        "pass": bool(n == 0 or ((err <= bound).all() and err.mean() <= MEAN_ABS and not np.isnan(t).any())),
    }
