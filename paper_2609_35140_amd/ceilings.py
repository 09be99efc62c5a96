"""Binding of libuattn_ceilings.so: measured ceilings for the roofline
fractions (streaming HBM read over a contiguous buffer or over 16 KB blocks
in a page-table order, and bf16 MFMA throughput).  Argument marshalling and
HIP-event timing only; the work runs in the library's kernels."""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libuattn_ceilings.so")
MFMA_FLOP = 16 * 16 * 32 * 2      # one v_mfma_f32_16x16x32_bf16
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_35140_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        c_i32, c_i64, c_p = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        lib.uattn_ceiling_read.restype = c_i32
        lib.uattn_ceiling_read.argtypes = [c_p, c_p, c_i64, c_i64, c_i32, c_p, c_p]
        lib.uattn_ceiling_read_grid.restype = c_i32
        lib.uattn_ceiling_read_grid.argtypes = []
        lib.uattn_ceiling_mfma.restype = c_i32
        lib.uattn_ceiling_mfma.argtypes = [c_i32, c_i32, c_p, c_p]
        _lib = lib
    return _lib


def lib():
    return _load()


def _time(fn, reps):
    import torch
    fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def read(src, block_table=None, block_bytes: int = 16384, checksum=None, nontemporal: bool = False):
    """Launch one streaming read of `src` (a uint8/any CUDA tensor) in blocks of
    `block_bytes`, in the order of `block_table` (int32 CUDA, or None for the
    identity order).  Returns the checksum tensor [grid] uint32 (as int32)."""
    import torch
    lib = _load()
    nbytes = src.numel() * src.element_size()
    nblocks = nbytes // block_bytes if block_table is None else block_table.numel()
    if checksum is None:
        checksum = torch.empty(lib.uattn_ceiling_read_grid(), dtype=torch.int32, device=src.device)
    code = lib.uattn_ceiling_read(src.data_ptr(), None if block_table is None else block_table.data_ptr(), nblocks,
                                  block_bytes, 1 if nontemporal else 0, checksum.data_ptr(),
                                  torch.cuda.current_stream().cuda_stream)
    if code != 0:
        raise RuntimeError(f"uattn_ceiling_read failed with code {code}")
    return checksum


def read_gbs(nbytes: int = 4 << 30, block_bytes: int = 16384, paged: bool = False, reps: int = 10, seed: int = 0,
             nontemporal: bool = False):
    """Measured streaming-read GB/s over a buffer of `nbytes` (well above the
    256 MB Infinity Cache), contiguous or in a random block order."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    src.view(torch.int32).fill_(0x5A5A5A5A)
    table = None
    if paged:
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        table = torch.randperm(nbytes // block_bytes, generator=g, device="cuda").to(torch.int32)
    ck = torch.empty(_load().uattn_ceiling_read_grid(), dtype=torch.int32, device="cuda")
    ms = _time(lambda: read(src, table, block_bytes, ck, nontemporal), reps)
    del src, table
    torch.cuda.empty_cache()
    return nbytes / (ms * 1e-3) / 1e9


def mfma_tflops(waves: int = 0, iters: int = 4000, reps: int = 5):
    """Measured dense bf16 MFMA TFLOP/s (v_mfma_f32_16x16x32_bf16, 8 independent
    accumulators per wave, 8 waves per CU: two per SIMD)."""
    import torch
    lib = _load()
    if waves <= 0:
        waves = 8 * torch.cuda.get_device_properties(0).multi_processor_count
    waves = (waves + 3) // 4 * 4
    out = torch.empty(waves, dtype=torch.float32, device="cuda")

    def fn():
        code = lib.uattn_ceiling_mfma(waves, iters, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
        if code != 0:
            raise RuntimeError(f"uattn_ceiling_mfma failed with code {code}")

    ms = _time(fn, reps)
    return waves * iters * 8 * MFMA_FLOP / (ms * 1e-3) / 1e12
