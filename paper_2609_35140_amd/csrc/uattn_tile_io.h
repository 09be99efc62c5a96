// Global -> register -> LDS staging of one 64-key K/V tile.
//
// 256 threads cooperate.  Thread t owns a (key group, d group) unit: KPU
// consecutive keys times 8 consecutive d values.  Consecutive threads take
// consecutive 16-byte pieces of the same key row, so every global load is a
// contiguous run per row.  K goes to LDS as is ([key][d]); V goes to LDS
// transposed ([d][key]) so that the PV product can read 8 consecutive keys
// of one d with a single 16-byte LDS read.  Rows whose position holds no key
// (past the context) are written as zeros, never read from memory.
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

  // offs[i] = element offset of row first_row+i in the K (and V) array, or -1.
  __device__ __forceinline__ void load(const __bf16* kbase, const __bf16* vbase, const int64_t (&offs)[kKPU], int tid) {
    const int dg = d_group(tid);
#pragma unroll
    for (int i = 0; i < kKPU; ++i) {
      if (offs[i] >= 0) {
        k[i] = *reinterpret_cast<const u32x4*>(kbase + offs[i] + 8 * dg);
        v[i] = *reinterpret_cast<const u32x4*>(vbase + offs[i] + 8 * dg);
      } else {
        k[i] = u32x4{0u, 0u, 0u, 0u};
        v[i] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }

  __device__ __forceinline__ void store(__bf16* stage, int tid) const {
    const int dg = d_group(tid), r0 = first_row(tid);
    __bf16* ks = stage;
    __bf16* vt = stage + Lds<D>::kKElems;
#pragma unroll
    for (int i = 0; i < kKPU; ++i)
      *reinterpret_cast<u32x4*>(ks + (r0 + i) * Lds<D>::kKStride + 8 * dg) = k[i];
    // transpose: for each of the 8 d values, the kKPU keys are contiguous in V^T
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int word = e >> 1, sh = (e & 1) * 16;
      uint32_t lo01 = ((v[0][word] >> sh) & 0xFFFFu) | (((v[1][word] >> sh) & 0xFFFFu) << 16);
      __bf16* dst = vt + (8 * dg + e) * Lds<D>::kVStride + r0;
      if constexpr (kKPU == 4) {
        uint32_t lo23 = ((v[2][word] >> sh) & 0xFFFFu) | (((v[3][word] >> sh) & 0xFFFFu) << 16);
        *reinterpret_cast<u32x2*>(dst) = u32x2{lo01, lo23};
      } else {
        *reinterpret_cast<uint32_t*>(dst) = lo01;
      }
    }
  }
};

}  // namespace uattn
