"""Python binding for libuattn.so (argument marshalling only).

Every function here checks shapes/dtypes, takes device pointers from torch
tensors and calls the C ABI declared in ``include/uattn.h`` on the current
torch stream.  All arithmetic runs in the HIP kernels; there is no CPU or
PyTorch fallback -- if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("UATTN_LIB") or os.path.join(_PKG, "libuattn.so")

UATTN_OK = 0
TILE_KEYS = 64
CHUNK_KEYS = 256

_lib = None


class UattnError(RuntimeError):
    pass


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise UattnError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_35140_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    c_i32, c_i64, c_f, c_p, c_sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
    lib.uattn_abi_version.restype = c_i32
    lib.uattn_abi_version.argtypes = []
    lib.uattn_status_string.restype = ctypes.c_char_p
    lib.uattn_status_string.argtypes = [c_i32]
    lib.uattn_prefill.restype = c_i32
    lib.uattn_prefill.argtypes = [c_p, c_p, c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_f, c_p, c_p, c_p]
    lib.uattn_decode_workspace_bytes.restype = c_sz
    lib.uattn_decode_workspace_bytes.argtypes = [c_i32, c_i32, c_i32, c_i32]
    lib.uattn_decode.restype = c_i32
    lib.uattn_decode.argtypes = [c_p, c_p, c_p, c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_f,
                                 c_p, c_p, c_p, c_sz, c_p]
    lib.uattn_decode_scratch_limit.restype = c_sz
    lib.uattn_decode_scratch_limit.argtypes = []
    lib.uattn_decode_noalloc.restype = c_i32
    lib.uattn_decode_noalloc.argtypes = [c_p, c_p, c_p, c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32,
                                         c_i32, c_f, c_p, c_p, c_p]
    lib.uattn_logprob.restype = c_i32
    lib.uattn_logprob.argtypes = [c_p, c_i64, c_p, c_i32, c_i32, c_f, c_p, c_p]
    lib.uattn_qk_norm_rope.restype = c_i32
    lib.uattn_qk_norm_rope.argtypes = [c_p, c_p, c_p, c_p, c_p, c_f, c_p, c_i32, c_i32, c_i32, c_i32, c_i32, c_p, c_p,
                                       c_p]
    lib.uattn_rope_cache.restype = c_i32
    lib.uattn_rope_cache.argtypes = [c_p, c_i32, c_i32, ctypes.c_double, c_p]
    lib.uattn_lm_head.restype = c_i32
    lib.uattn_lm_head.argtypes = [c_p, c_i64, c_p, c_i64, c_i32, c_i32, c_i32, c_p, c_i64, c_p]
    lib.uattn_lm_head_logprob_workspace_bytes.restype = c_sz
    lib.uattn_lm_head_logprob_workspace_bytes.argtypes = [c_i32, c_i32]
    lib.uattn_lm_head_logprob.restype = c_i32
    lib.uattn_lm_head_logprob.argtypes = [c_p, c_i64, c_p, c_i64, c_p, c_i32, c_i32, c_i32, c_f, c_p, c_p, c_i64, c_p,
                                          c_sz, c_p]
    lib.uattn_prefill_backward_workspace_bytes.restype = c_sz
    lib.uattn_prefill_backward_workspace_bytes.argtypes = [c_i32, c_i32]
    lib.uattn_prefill_backward.restype = c_i32
    lib.uattn_prefill_backward.argtypes = [c_p, c_p, c_p, c_p, c_p, c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_i32,
                                           c_i32, c_f, c_p, c_p, c_p, c_p, c_sz, c_p]
    lib.uattn_kv_write.restype = c_i32
    lib.uattn_kv_write.argtypes = [c_p, c_p, c_i64, c_p, c_p, c_p, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32,
                                   c_p, c_p, c_p]
    _lib = lib
    return lib


def lib():
    """The loaded ctypes library (raises if it is not built)."""
    return _load()


def abi_version() -> int:
    return int(_load().uattn_abi_version())


def status_string(code: int) -> str:
    return _load().uattn_status_string(int(code)).decode()


def _check(code: int):
    if code != UATTN_OK:
        raise UattnError(status_string(code))


def _stream(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def _bf16_cuda(t, name):
    import torch
    _need(t.is_cuda, f"{name} must be a GPU tensor")
    _need(t.dtype == torch.bfloat16, f"{name} must be bfloat16")
    _need(t.is_contiguous(), f"{name} must be contiguous")


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)


def prefill(q, k, v, cu_seqlens, max_seqlen: int, softmax_scale: Optional[float] = None, out=None,
            return_lse: bool = False, lse=None, stream=None):
    """Full-sequence causal attention (uattn_prefill).

    q [T,Hq,d], k/v [T,Hkv,d] bf16 CUDA; cu_seqlens int32 CUDA [B+1].
    Returns out [T,Hq,d] (and lse [T,Hq] fp32 if requested).
    """
    import torch
    for name, t in (("q", q), ("k", k), ("v", v)):
        _bf16_cuda(t, name)
    _need(q.dim() == 3 and k.dim() == 3 and v.dim() == 3, "q/k/v must be [T, H, d]")
    T, hq, d = q.shape
    _need(k.shape == v.shape and k.shape[0] == T and k.shape[2] == d, "k/v shape mismatch")
    _need(cu_seqlens.dtype == torch.int32 and cu_seqlens.is_cuda and cu_seqlens.is_contiguous(),
          "cu_seqlens must be contiguous int32 on the GPU")
    if softmax_scale is None:
        softmax_scale = default_scale(d)
    if out is None:
        out = torch.empty_like(q)
    else:
        _bf16_cuda(out, "out")
        _need(out.shape == q.shape, "out shape")
    if return_lse and lse is None:
        lse = torch.empty((T, hq), dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse.dtype == torch.float32 and lse.is_contiguous() and lse.shape == (T, hq), "lse must be [T,Hq] fp32")
    _check(_load().uattn_prefill(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens), cu_seqlens.numel() - 1, T,
                                 int(max_seqlen), hq, k.shape[1], d, float(softmax_scale), _ptr(out), _ptr(lse),
                                 _stream(stream)))
    return (out, lse) if lse is not None else out


def prefill_backward_workspace_bytes(total_tokens: int, num_q_heads: int) -> int:
    return int(_load().uattn_prefill_backward_workspace_bytes(int(total_tokens), int(num_q_heads)))


def prefill_backward(q, k, v, out, dout, lse, cu_seqlens, max_seqlen: int, softmax_scale: Optional[float] = None,
                     dq=None, dk=None, dv=None, workspace=None, stream=None):
    """Gradients of the full-sequence attention (uattn_prefill_backward).

    q, k, v, cu_seqlens, max_seqlen, softmax_scale as for prefill; out and lse
    are prefill's outputs for them; dout [T,Hq,d] bf16 is the upstream
    gradient.  Returns (dq [T,Hq,d], dk [T,Hkv,d], dv [T,Hkv,d]) bf16.
    """
    import torch
    for name, t in (("q", q), ("k", k), ("v", v), ("out", out), ("dout", dout)):
        _bf16_cuda(t, name)
    _need(q.dim() == 3 and k.dim() == 3 and v.dim() == 3, "q/k/v must be [T, H, d]")
    T, hq, d = q.shape
    hkv = k.shape[1]
    _need(k.shape == v.shape and k.shape[0] == T and k.shape[2] == d, "k/v shape mismatch")
    _need(out.shape == q.shape and dout.shape == q.shape, "out/dout must match q")
    _need(lse.dtype == torch.float32 and lse.is_cuda and lse.is_contiguous() and tuple(lse.shape) == (T, hq),
          "lse must be [T,Hq] fp32 on the GPU")
    _need(cu_seqlens.dtype == torch.int32 and cu_seqlens.is_cuda and cu_seqlens.is_contiguous(),
          "cu_seqlens must be contiguous int32 on the GPU")
    if softmax_scale is None:
        softmax_scale = default_scale(d)
    outs = []
    for name, t, like in (("dq", dq, q), ("dk", dk, k), ("dv", dv, v)):
        if t is None:
            t = torch.empty_like(like)
        else:
            _bf16_cuda(t, name)
            _need(t.shape == like.shape, f"{name} shape")
        outs.append(t)
    need = prefill_backward_workspace_bytes(T, hq)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)  # no initial contents needed
    _check(_load().uattn_prefill_backward(
        _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse), _ptr(cu_seqlens), cu_seqlens.numel() - 1, T,
        int(max_seqlen), hq, hkv, d, float(softmax_scale), _ptr(outs[0]), _ptr(outs[1]), _ptr(outs[2]),
        _ptr(workspace), workspace.numel() * workspace.element_size() if workspace is not None else 0,
        _stream(stream)))
    return tuple(outs)


def decode_workspace_bytes(batch: int, max_seqlen: int, num_q_heads: int, head_dim: int) -> int:
    return int(_load().uattn_decode_workspace_bytes(batch, max_seqlen, num_q_heads, head_dim))


def new_workspace(nbytes: int, device="cuda"):
    """A zero-filled decode workspace (the counters it holds must start at zero).

    The returned tensor carries the extent of its known-zero prefix as an
    attribute of the tensor object itself, so the binding never re-zeroes it
    needlessly and never trusts a stale record: a different tensor (even one
    at the same device address) starts with no such record.
    """
    import torch
    t = torch.zeros(int(nbytes), dtype=torch.uint8, device=device)
    t._uattn_zero_prefix = int(nbytes)
    return t


def counter_bytes(batch: int, num_q_heads: int) -> int:
    """Size of the counter region at the start of a decode workspace."""
    return (4 * batch * num_q_heads + 255) // 256 * 256


def _partials_start(ws_bytes: int, batch: int, max_seqlen: int, num_q_heads: int, head_dim: int) -> int:
    """Byte offset where a call's fp32 partials begin (they sit at the end of
    the workspace; the counters at its start)."""
    nslot = ((max_seqlen + CHUNK_KEYS - 1) // CHUNK_KEYS + 1) // 2 * 2   # chunks rounded up to even
    acc = (4 * batch * num_q_heads * nslot * head_dim + 255) // 256 * 256
    ml = (4 * batch * num_q_heads * nslot * 2 + 255) // 256 * 256
    return (ws_bytes & ~15) - acc - ml


def _prepare_workspace(workspace, batch: int, max_seqlen: int, num_q_heads: int, head_dim: int):
    """Make the counter region of ``workspace`` zero before a call, as uattn.h
    requires, and record what the call leaves zero.

    The record lives on the tensor object (``_uattn_zero_prefix``), never in
    a table keyed by address: a workspace tensor this binding has not seen
    before (or a different view of the same memory) is zeroed on first use,
    whatever an earlier tensor at that address held.  After the call the
    counters are zero again (the kernel resets them), while the partial
    region at the end of the buffer holds data.
    """
    nbytes = workspace.numel() * workspace.element_size()
    c = min(counter_bytes(batch, num_q_heads), nbytes)
    known = getattr(workspace, "_uattn_zero_prefix", 0)
    if known < c:
        workspace.view(-1)[: c // workspace.element_size()].zero_()
        known = c
    workspace._uattn_zero_prefix = max(c, min(known, _partials_start(nbytes, batch, max_seqlen, num_q_heads,
                                                                        head_dim)))


def decode(q, k_pages, v_pages, block_table, seqlens, max_seqlen: int, softmax_scale: Optional[float] = None,
           out=None, return_lse: bool = False, lse=None, workspace=None, stream=None):
    """Token-wise paged decode (uattn_decode).

    q [B,Hq,d]; k_pages/v_pages [P,Hkv,page,d] bf16 CUDA; block_table [B,maxp]
    int32; seqlens [B] int32 (context length including the current token).
    ``workspace`` is a zero-filled uint8 CUDA tensor (``new_workspace``); a
    fresh one is allocated when not given.
    """
    import torch
    for name, t in (("q", q), ("k_pages", k_pages), ("v_pages", v_pages)):
        _bf16_cuda(t, name)
    _need(q.dim() == 3 and k_pages.dim() == 4 and v_pages.shape == k_pages.shape, "shapes: q [B,Hq,d], pages [P,Hkv,page,d]")
    B, hq, d = q.shape
    _, hkv, page, d2 = k_pages.shape
    _need(d2 == d, "head_dim mismatch")
    for name, t in (("block_table", block_table), ("seqlens", seqlens)):
        _need(t.dtype == torch.int32 and t.is_cuda and t.is_contiguous(), f"{name} must be contiguous int32 on the GPU")
    _need(block_table.dim() == 2 and block_table.shape[0] == B and seqlens.shape == (B,), "block_table/seqlens shape")
    if softmax_scale is None:
        softmax_scale = default_scale(d)
    if out is None:
        out = torch.empty_like(q)
    else:
        _bf16_cuda(out, "out")
        _need(out.shape == q.shape, "out shape")
    if return_lse and lse is None:
        lse = torch.empty((B, hq), dtype=torch.float32, device=q.device)
    need = decode_workspace_bytes(B, int(max_seqlen), hq, d) if B > 0 else 0
    if workspace is None and need > 0:
        workspace = new_workspace(need, q.device)
    if workspace is not None and need > 0:
        _need(workspace.is_cuda and workspace.is_contiguous(), "workspace must be a contiguous GPU tensor")
        _prepare_workspace(workspace, B, int(max_seqlen), hq, d)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_load().uattn_decode(_ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(block_table), _ptr(seqlens), B,
                                block_table.shape[1], page, k_pages.shape[0], int(max_seqlen), hq, hkv, d, float(softmax_scale),
                                _ptr(out), _ptr(lse), _ptr(workspace), ws_bytes, _stream(stream)))
    return (out, lse) if lse is not None else out


def decode_scratch_limit() -> int:
    """Bytes of the library's static decode scratch array (uattn_decode_noalloc)."""
    return int(_load().uattn_decode_scratch_limit())


def decode_noalloc(q, k_pages, v_pages, block_table, seqlens, max_seqlen: int, softmax_scale: Optional[float] = None,
                   out=None, return_lse: bool = False, lse=None, stream=None):
    """uattn_decode_noalloc: the token-wise decode with the library's static
    scratch array as its workspace (the call itself allocates nothing; pass
    ``out``/``lse`` to keep this binding from allocating them).  Arguments and
    results as for :func:`decode`."""
    import torch
    for name, t in (("q", q), ("k_pages", k_pages), ("v_pages", v_pages)):
        _bf16_cuda(t, name)
    _need(q.dim() == 3 and k_pages.dim() == 4 and v_pages.shape == k_pages.shape, "shapes: q [B,Hq,d], pages [P,Hkv,page,d]")
    B, hq, d = q.shape
    _, hkv, page, d2 = k_pages.shape
    _need(d2 == d, "head_dim mismatch")
    for name, t in (("block_table", block_table), ("seqlens", seqlens)):
        _need(t.dtype == torch.int32 and t.is_cuda and t.is_contiguous(), f"{name} must be contiguous int32 on the GPU")
    _need(block_table.dim() == 2 and block_table.shape[0] == B and seqlens.shape == (B,), "block_table/seqlens shape")
    if softmax_scale is None:
        softmax_scale = default_scale(d)
    if out is None:
        out = torch.empty_like(q)
    else:
        _bf16_cuda(out, "out")
        _need(out.shape == q.shape, "out shape")
    if return_lse and lse is None:
        lse = torch.empty((B, hq), dtype=torch.float32, device=q.device)
    if lse is not None:
        _need(lse.dtype == torch.float32 and lse.is_contiguous() and tuple(lse.shape) == (B, hq), "lse must be [B,Hq] fp32")
    _check(_load().uattn_decode_noalloc(_ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(block_table), _ptr(seqlens), B,
                                        block_table.shape[1], page, k_pages.shape[0], int(max_seqlen), hq, hkv, d,
                                        float(softmax_scale), _ptr(out), _ptr(lse), _stream(stream)))
    return (out, lse) if lse is not None else out


def logprob(logits, targets, inv_temperature: float = 1.0, out=None, stream=None):
    """Per-token log-probability (uattn_logprob). logits [T,V] bf16 (row stride may exceed V)."""
    import torch
    _need(logits.is_cuda and logits.dtype == torch.bfloat16 and logits.dim() == 2, "logits must be [T,V] bf16 on the GPU")
    _need(logits.stride(1) == 1, "logits rows must be contiguous")
    T, V = logits.shape
    _need(targets.dtype == torch.int32 and targets.is_cuda and targets.shape == (T,) and targets.is_contiguous(),
          "targets must be [T] int32 on the GPU")
    if out is None:
        out = torch.empty(T, dtype=torch.float32, device=logits.device)
    _check(_load().uattn_logprob(_ptr(logits), logits.stride(0), _ptr(targets), T, V, float(inv_temperature),
                                 _ptr(out), _stream(stream)))
    return out


def kv_write(k_new, v_new, block_table, seq_idx, positions, k_pages, v_pages, stream=None):
    """Write new K/V token rows into the paged cache in place (uattn_kv_write).

      k_new, v_new   [N, Hkv, d] bf16 (token rows may be strided: stride(0) elements apart)
      block_table    [B, maxp] int32; seq_idx, positions [N] int32 (position < 0: padding)
      k_pages, v_pages  [P, Hkv, page, d] bf16, updated in place
    """
    import torch
    for name, t in (("k_pages", k_pages), ("v_pages", v_pages)):
        _bf16_cuda(t, name)
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        _need(t.is_cuda and t.dtype == torch.bfloat16, f"{name} must be a bfloat16 GPU tensor")
    _need(k_new.dim() == 3 and v_new.shape == k_new.shape, "k_new/v_new must be [N,Hkv,d]")
    N, hkv, d = k_new.shape
    _need(k_new.stride(2) == 1 and k_new.stride(1) == d and v_new.stride() == k_new.stride(),
          "k_new/v_new: heads and d must be contiguous, both with the same token stride")
    P, hkv2, page, d2 = k_pages.shape
    _need(hkv2 == hkv and d2 == d and v_pages.shape == k_pages.shape and k_pages.is_contiguous()
          and v_pages.is_contiguous(), "page shapes")
    for name, t in (("block_table", block_table), ("seq_idx", seq_idx), ("positions", positions)):
        _need(t.dtype == torch.int32 and t.is_cuda and t.is_contiguous(), f"{name} must be int32 on the GPU")
    _need(block_table.dim() == 2 and seq_idx.shape == (N,) and positions.shape == (N,), "index shapes")
    B, maxp = block_table.shape
    _check(_load().uattn_kv_write(_ptr(k_new), _ptr(v_new), k_new.stride(0), _ptr(block_table), _ptr(seq_idx),
                                  _ptr(positions), N, B, maxp, page, P, hkv, d, _ptr(k_pages), _ptr(v_pages),
                                  _stream(stream)))
    return k_pages, v_pages


def rope_cache(max_position: int, head_dim: int, theta: float, out=None, stream=None):
    """The NeoX rotary table [max_position, head_dim/2, 2] fp32 (uattn_rope_cache)."""
    import torch
    if out is None:
        out = torch.empty((max_position, head_dim // 2, 2), dtype=torch.float32, device="cuda")
    _need(out.dtype == torch.float32 and out.is_cuda and out.is_contiguous()
          and tuple(out.shape) == (max_position, head_dim // 2, 2), "out must be [max_position, head_dim/2, 2] fp32")
    _check(_load().uattn_rope_cache(_ptr(out), max_position, head_dim, float(theta), _stream(stream)))
    return out


def qk_norm_rope(q, k, positions, q_weight, k_weight, cos_sin, eps: float = 1e-6, q_out=None, k_out=None,
                 stream=None):
    """RMSNorm of every q and k head row, then NeoX rotary embedding (uattn_qk_norm_rope).

      q [T, Hq, d], k [T, Hkv, d] bf16; positions [T] int32; q_weight, k_weight [d] bf16;
      cos_sin [max_position, d/2, 2] fp32.  Outputs may be q and k themselves (in place).
    """
    import torch
    for name, t in (("q", q), ("k", k), ("q_weight", q_weight), ("k_weight", k_weight)):
        _bf16_cuda(t, name)
    _need(q.dim() == 3 and k.dim() == 3 and q.shape[0] == k.shape[0] and q.shape[2] == k.shape[2], "q/k shapes")
    T, hq, d = q.shape
    hkv = k.shape[1]
    _need(q_weight.shape == (d,) and k_weight.shape == (d,), "weights must be [d]")
    _need(positions.dtype == torch.int32 and positions.is_cuda and positions.shape == (T,) and positions.is_contiguous(),
          "positions must be [T] int32 on the GPU")
    _need(cos_sin.dtype == torch.float32 and cos_sin.is_cuda and cos_sin.is_contiguous() and cos_sin.dim() == 3
          and cos_sin.shape[1:] == (d // 2, 2), "cos_sin must be [max_position, d/2, 2] fp32")
    if q_out is None:
        q_out = torch.empty_like(q)
    if k_out is None:
        k_out = torch.empty_like(k)
    _need(q_out.shape == q.shape and k_out.shape == k.shape, "output shapes")
    _check(_load().uattn_qk_norm_rope(_ptr(q), _ptr(k), _ptr(positions), _ptr(q_weight), _ptr(k_weight), float(eps),
                                      _ptr(cos_sin), cos_sin.shape[0], T, hq, hkv, d, _ptr(q_out), _ptr(k_out),
                                      _stream(stream)))
    return q_out, k_out


def lm_head(hidden, weight, out=None, stream=None):
    """Batch-invariant logits = bf16(hidden . weight^T) (uattn_lm_head).

      hidden [T, H] bf16, weight [V, H] bf16 (rows may be strided); out [T, V] bf16 (row stride a multiple of 8).
    """
    import torch
    for name, t in (("hidden", hidden), ("weight", weight)):
        _need(t.is_cuda and t.dtype == torch.bfloat16 and t.dim() == 2 and t.stride(1) == 1,
              f"{name} must be a 2-D bfloat16 GPU tensor with contiguous rows")
    T, H = hidden.shape
    V, H2 = weight.shape
    _need(H2 == H, "hidden and weight widths differ")
    if out is None:
        stride = (V + 7) // 8 * 8
        out = torch.empty((T, stride), dtype=torch.bfloat16, device=hidden.device)[:, :V]
    _need(out.dtype == torch.bfloat16 and out.is_cuda and out.shape == (T, V) and out.stride(1) == 1, "out shape")
    _check(_load().uattn_lm_head(_ptr(hidden), hidden.stride(0), _ptr(weight), weight.stride(0), T, V, H, _ptr(out),
                                 out.stride(0), _stream(stream)))
    return out


def lm_head_logprob_workspace_bytes(num_rows: int, vocab: int) -> int:
    return int(_load().uattn_lm_head_logprob_workspace_bytes(int(num_rows), int(vocab)))


def lm_head_logprob(hidden, weight, targets, inv_temperature: float = 1.0, out=None, logits=None, workspace=None,
                    stream=None):
    """LM head fused with the token log-probability (uattn_lm_head_logprob).

      hidden [T, H], weight [V, H] bf16 (rows may be strided); targets [T] int32.
      Returns logp [T] fp32.  ``logits`` ([T, V] bf16, row stride a multiple
      of 8), when given, also receives the logits.
    """
    import torch
    for name, t in (("hidden", hidden), ("weight", weight)):
        _need(t.is_cuda and t.dtype == torch.bfloat16 and t.dim() == 2 and t.stride(1) == 1,
              f"{name} must be a 2-D bfloat16 GPU tensor with contiguous rows")
    T, H = hidden.shape
    V, H2 = weight.shape
    _need(H2 == H, "hidden and weight widths differ")
    _need(targets.dtype == torch.int32 and targets.is_cuda and targets.shape == (T,) and targets.is_contiguous(),
          "targets must be [T] int32 on the GPU")
    if out is None:
        out = torch.empty(T, dtype=torch.float32, device=hidden.device)
    _need(out.dtype == torch.float32 and out.is_cuda and out.shape == (T,) and out.is_contiguous(), "out must be [T] fp32")
    if logits is not None:
        _need(logits.dtype == torch.bfloat16 and logits.is_cuda and logits.shape == (T, V) and logits.stride(1) == 1,
              "logits must be [T, V] bf16 with contiguous rows")
    need = lm_head_logprob_workspace_bytes(T, V)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=hidden.device)  # no initial contents needed
    _check(_load().uattn_lm_head_logprob(_ptr(hidden), hidden.stride(0), _ptr(weight), weight.stride(0), _ptr(targets),
                                         T, V, H, float(inv_temperature), _ptr(out), _ptr(logits),
                                         logits.stride(0) if logits is not None else 0, _ptr(workspace),
                                         workspace.numel() * workspace.element_size(), _stream(stream)))
    return out


def raw_call(name: str, *args) -> int:
    """Call a C entry point with raw arguments (for error-path tests)."""
    return int(getattr(_load(), name)(*args))


class DecodeSteps:
    """Argument lists for a run of uattn_decode calls over fixed buffers.

    A rollout loop calls decode once per generated token on the same cache,
    block table and workspace; only the query, length and output slices
    change.  This marshals every call's arguments once, so the loop pays one
    ctypes call per step.

      q_steps        [S, B, Hq, d] bf16   (step i uses q_steps[i])
      seqlens_steps  [S, B] int32
      out_steps      [S, B, Hq, d] bf16
    """

    def __init__(self, q_steps, k_pages, v_pages, block_table, seqlens_steps, max_seqlen: int, out_steps,
                 workspace=None, softmax_scale: Optional[float] = None, stream=None):
        import torch
        for name, t in (("q_steps", q_steps), ("k_pages", k_pages), ("v_pages", v_pages), ("out_steps", out_steps)):
            _bf16_cuda(t, name)
        _need(q_steps.dim() == 4 and out_steps.shape == q_steps.shape, "q_steps/out_steps must be [S,B,Hq,d]")
        S, B, hq, d = q_steps.shape
        _, hkv, page, d2 = k_pages.shape
        _need(d2 == d and v_pages.shape == k_pages.shape, "page shapes")
        _need(seqlens_steps.dtype == torch.int32 and seqlens_steps.shape == (S, B) and seqlens_steps.is_contiguous(),
              "seqlens_steps must be [S,B] int32")
        _need(block_table.dtype == torch.int32 and block_table.is_contiguous() and block_table.shape[0] == B,
              "block_table must be [B,maxp] int32")
        if softmax_scale is None:
            softmax_scale = default_scale(d)
        need = decode_workspace_bytes(B, int(max_seqlen), hq, d)
        if workspace is None and need > 0:
            workspace = new_workspace(need, q_steps.device)
        if workspace is not None and need > 0:
            _need(workspace.is_cuda and workspace.is_contiguous(), "workspace must be a contiguous GPU tensor")
            _prepare_workspace(workspace, B, int(max_seqlen), hq, d)
        self.workspace = workspace
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        st = _stream(stream)
        qstride = B * hq * d * 2
        lstride = B * 4
        self._fn = _load().uattn_decode
        self.args = [
            (q_steps.data_ptr() + i * qstride, _ptr(k_pages), _ptr(v_pages), _ptr(block_table),
             seqlens_steps.data_ptr() + i * lstride, B, block_table.shape[1], page, k_pages.shape[0], int(max_seqlen),
             hq, hkv, d, float(softmax_scale), out_steps.data_ptr() + i * qstride, None, _ptr(workspace), ws_bytes, st)
            for i in range(S)
        ]
        self._keep = (q_steps, k_pages, v_pages, block_table, seqlens_steps, out_steps)

    def __len__(self):
        return len(self.args)

    def run(self, i: int, stream=None):
        """Launch step i (on ``stream`` if given, else the stream fixed at construction)."""
        a = self.args[i]
        if stream is not None:
            a = a[:-1] + (_stream(stream),)
        code = self._fn(*a)
        if code != UATTN_OK:
            raise UattnError(status_string(code))
