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
