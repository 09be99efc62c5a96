// Global -> LDS staging of one 64-key K/V tile, and the LDS layout it produces.
//
// Tiles move with the gfx950 direct-to-LDS loads (global_load_lds_dwordx4):
// each lane names a 16-byte global piece and the hardware deposits the 64
// pieces of one instruction contiguously in LDS, so no registers stage the
// data and no LDS store instructions are issued.  Because the LDS destination
// of a lane is fixed by its lane index, bank spreading uses an XOR swizzle of
// the 16-byte pieces within each row (chosen per read pattern, see below)
// rather than row padding: the lane that owns LDS piece p of row r fetches
// logical piece p ^ f(r) of that row.
//
// Rows whose position holds no key (past the context) are fetched from a
// zero block in device memory, so the tile always holds zeros there and no
// out-of-range address is ever formed.
//
// Work split: each wave of the workgroup fills an equal run of consecutive
// rows (16 rows with 4 waves, 8 with 8) of K and of V, so a wave's rows are
// one strided run in global memory (consecutive tokens of a packed batch, or
// consecutive slots of one cache page: pages hold >= 16 keys).
#pragma once

#include "uattn_numerics.h"

namespace uattn {

// 256 zero bytes; the source of every tile row past the context.
__device__ __attribute__((aligned(256))) uint4 g_zero_rows[16];

// Issue the loads of this wave's RPW rows of K and V into `stage`
// (RPW = 64 / number of waves; rows RPW*wave .. RPW*wave + RPW-1).
//   kbase/vbase : element pointers of tile row RPW*wave (unused when nvalid <= 0)
//   row_stride  : elements between consecutive rows
//   nvalid      : rows RPW*wave + r with r < nvalid hold keys; the rest are zero-filled
template <int D, int RPW>
struct TileLoads {
  static constexpr int kInstr = RPW * TileLayout<D>::kPieces / 64;  // 1 KB instructions per wave per matrix
  static constexpr int kPerTile = 2 * kInstr;                        // K and V
};

template <int D, int RPW>
__device__ __forceinline__ void load_tile_rows(__bf16* stage, const __bf16* kbase, const __bf16* vbase,
                                               int64_t row_stride, int nvalid, int wave, int lane) {
  using TL = TileLayout<D>;
  constexpr int kInstr = RPW * TL::kPieces / 64;  // 1 KB instructions per wave per matrix
  static_assert(kInstr >= 1 && RPW * TL::kPieces == 64 * kInstr, "tile split");
  const __bf16* zero = reinterpret_cast<const __bf16*>(g_zero_rows) + 8 * (lane & 15);
#pragma unroll
  for (int i = 0; i < kInstr; ++i) {
    const int slot = (wave * kInstr + i) * 64 + lane;  // 16-byte piece index in the tile
    const int row = slot / TL::kPieces, piece = slot % TL::kPieces;
    const int r = row - RPW * wave;
    const bool ok = r < nvalid;
    const __bf16* ks = ok ? kbase + r * row_stride + 8 * (piece ^ TL::k_swz(row)) : zero;
    const __bf16* vs = ok ? vbase + r * row_stride + 8 * (piece ^ TL::v_swz(row)) : zero;
    __bf16* kd = stage + (wave * kInstr + i) * 64 * 8;
    __bf16* vd = kd + TL::kTileElems;
    __builtin_amdgcn_global_load_lds(ks, (__attribute__((address_space(3))) void*)kd, 16, 0, 0);
    __builtin_amdgcn_global_load_lds(vs, (__attribute__((address_space(3))) void*)vd, 16, 0, 0);
  }
}

// ---------------------------------------------------------------------------
// Explicitly scheduled variant.  The compiler's wait-count pass cannot tell an
// LDS read from an earlier direct-to-LDS load that writes other LDS bytes, so
// with the builtin loads it drains every outstanding load before the first
// transposing LDS read of a tile, and a plain __syncthreads() drains them too
// (its workgroup release fence).  Both defeat loads kept in flight across
// tiles.  The loads below are issued from inline assembly, which that pass
// does not track; the caller then owns every vmcnt wait before reading what
// they wrote, and synchronises the workgroup with lds_barrier / wait_barrier.
// The compiler allocates nothing in M0 in the kernels that use these.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// LDS byte address of a generic pointer into LDS: the shared aperture is
// 4 GB aligned, so it is the low 32 bits of the flat address (no address
// space cast, whose null check the compiler may mishandle).
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}
// 16 bytes per lane from `src` to LDS at m0 + 16*lane (m0 wave-uniform).
__device__ __forceinline__ void dma_b128(const void* src, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds_wave_base)
               : "memory", "m0");
}
// The same from a wave-uniform base plus a per-lane 32-bit byte offset (the
// instruction's scalar-base form: no 64-bit address arithmetic per lane).
__device__ __forceinline__ void dma_b128_based(const void* sbase, uint32_t voffset, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voffset), "s"(sbase), "s"(lds_wave_base)
               : "memory", "m0");
}
// 4 bytes per lane from `src` to LDS at m0 + 4*lane.
__device__ __forceinline__ void dma_b32(const void* src, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(src), "s"(lds_wave_base)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Workgroup barrier that orders LDS only (no wait on global memory).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
// Wait until at most n vector-memory operations of this wave are outstanding,
// then barrier: every wave's loads issued before its last n have landed.
template <int n>
__device__ __forceinline__ void wait_barrier() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" : : "n"(n) : "memory");
}
template <int n>
__device__ __forceinline__ void wait_vmem_asm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(n) : "memory");
}
// wait_barrier for the tile ring: all but the `pending` most recently issued
// tiles (per_tile operations each) have landed, in every wave.
template <int per_tile>
__device__ __forceinline__ void wait_tiles_barrier(int pending) {
  switch (pending) {
    case 0: wait_barrier<0>(); break;
    case 1: wait_barrier<per_tile>(); break;
    case 2: wait_barrier<2 * per_tile>(); break;
    default: wait_barrier<3 * per_tile>(); break;
  }
}

// load_tile_rows with the untracked loads (same rows, pieces and swizzle).
template <int D, int RPW>
__device__ __forceinline__ void load_tile_rows_async(__bf16* stage, const __bf16* kbase, const __bf16* vbase,
                                                     int64_t row_stride, int nvalid, int wave, int lane) {
  using TL = TileLayout<D>;
  constexpr int kInstr = RPW * TL::kPieces / 64;
  static_assert(kInstr >= 1 && RPW * TL::kPieces == 64 * kInstr, "tile split");
  const __bf16* zero = reinterpret_cast<const __bf16*>(g_zero_rows) + 8 * (lane & 15);
  const uint32_t kd0 = __builtin_amdgcn_readfirstlane(lds_addr(stage + wave * kInstr * 64 * 8));
  if (nvalid >= RPW) {
    // every row of this wave is in the sequence: uniform bases, per-lane
    // byte offsets that do not change from tile to tile
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      const int slot = (wave * kInstr + i) * 64 + lane;
      const int row = slot / TL::kPieces, piece = slot % TL::kPieces;
      const int r = row - RPW * wave;
      const uint32_t ko = static_cast<uint32_t>((r * row_stride + 8 * (piece ^ TL::k_swz(row))) * 2);
      const uint32_t vo = static_cast<uint32_t>((r * row_stride + 8 * (piece ^ TL::v_swz(row))) * 2);
      dma_b128_based(kbase, ko, kd0 + i * 64 * 16);
      dma_b128_based(vbase, vo, kd0 + i * 64 * 16 + TL::kTileElems * 2);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < kInstr; ++i) {
    const int slot = (wave * kInstr + i) * 64 + lane;
    const int row = slot / TL::kPieces, piece = slot % TL::kPieces;
    const int r = row - RPW * wave;
    const bool ok = r < nvalid;
    const __bf16* ks = ok ? kbase + r * row_stride + 8 * (piece ^ TL::k_swz(row)) : zero;
    const __bf16* vs = ok ? vbase + r * row_stride + 8 * (piece ^ TL::v_swz(row)) : zero;
    dma_b128(ks, kd0 + i * 64 * 16);
    dma_b128(vs, kd0 + i * 64 * 16 + TL::kTileElems * 2);
  }
}

// Wait until at most `n` of this wave's vector-memory operations are still
// outstanding (they complete in issue order, so every earlier load has landed).
template <int n>
__device__ __forceinline__ void wait_vmem_below() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | 0x0F70);
}
// Wait until all but the loads of the `pending` most recently issued tiles
// have landed, where one tile costs `per_tile` operations (pending < 4).
template <int per_tile>
__device__ __forceinline__ void wait_tiles_pending(int pending) {
  switch (pending) {
    case 0: wait_vmem_below<0>(); break;
    case 1: wait_vmem_below<per_tile>(); break;
    case 2: wait_vmem_below<2 * per_tile>(); break;
    default: wait_vmem_below<3 * per_tile>(); break;
  }
}
__device__ __forceinline__ void wait_tile_loads() { wait_vmem_below<0>(); }

}  // namespace uattn
