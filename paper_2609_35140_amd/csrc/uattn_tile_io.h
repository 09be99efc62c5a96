// Global -> register -> LDS staging of one 64-key K/V tile.
//
// 256 threads cooperate.  Thread t owns a (key group, d group) unit: KPU
// consecutive keys times 8 consecutive d values.  Consecutive threads take
// consecutive 16-byte pieces of the same key row, so every global load is a
// contiguous run per row.  K and V go to LDS key-major, as they are in memory
// (the PV product transposes V on its LDS read).  Rows whose position holds no
// key (past the context) are written as zeros, never read from memory.
#pragma once

#include "uattn_numerics.h"

namespace uattn {

template <int D>
struct TileIO {
  static constexpr int kCPR = D / 8;              // 16-byte pieces per row
  static constexpr int kKPU = (64 * kCPR) / 256;  // keys per thread unit (4 for d=128, 2 for d=64)
  static_assert(kKPU == 2 || kKPU == 4, "unsupported head_dim");

  u32x4 k[kKPU];
  u32x4 v[kKPU];

  __device__ __forceinline__ static int key_group(int tid) { return tid / kCPR; }
  __device__ __forceinline__ static int d_group(int tid) { return tid % kCPR; }
  // First tile row this thread loads (rows first_row .. first_row + kKPU - 1).
  __device__ __forceinline__ static int first_row(int tid) { return key_group(tid) * kKPU; }

  // Rows first_row .. first_row + kKPU - 1: row i (< nvalid) is read at element
  // offset off0 + i * row_stride of the K (and V) array; rows >= nvalid are zeros.
  __device__ __forceinline__ void load(const __bf16* kbase, const __bf16* vbase, int64_t off0, int64_t row_stride,
                                       int nvalid, int tid) {
    const int64_t o = off0 + 8 * d_group(tid);
#pragma unroll
    for (int i = 0; i < kKPU; ++i) {
      if (i < nvalid) {
        k[i] = *reinterpret_cast<const u32x4*>(kbase + o + i * row_stride);
        v[i] = *reinterpret_cast<const u32x4*>(vbase + o + i * row_stride);
      } else {
        k[i] = u32x4{0u, 0u, 0u, 0u};
        v[i] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }

  __device__ __forceinline__ void store(__bf16* stage, int tid) const {
    const int dg = d_group(tid), r0 = first_row(tid);
    __bf16* ks = stage;
    __bf16* vs = stage + Lds<D>::kKElems;
#pragma unroll
    for (int i = 0; i < kKPU; ++i) {
      *reinterpret_cast<u32x4*>(ks + (r0 + i) * Lds<D>::kKStride + 8 * dg) = k[i];
      *reinterpret_cast<u32x4*>(vs + (r0 + i) * Lds<D>::kVStride + 8 * dg) = v[i];
    }
  }
};

}  // namespace uattn
