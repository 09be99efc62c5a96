// Microbenchmarks for the measured ceilings (declared in uattn_ceilings.h).
#include <hip/hip_runtime.h>

#include "../../include/uattn_ceilings.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;  // 16-byte loads in flight per lane before they are consumed

int read_grid() {
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) cus = n;
  }
  return cus * 8;  // eight 4-wave workgroups per CU
}

// Workgroup w reads blocks w, w + grid, ...; a block is read as consecutive
// 4 KB rounds (256 lanes x 16 bytes), kUnroll rounds issued before use.
// NT: the loads carry the non-temporal hint.
template <bool NT>
__global__ __launch_bounds__(kThreads) void read_kernel(const u32x4* __restrict__ src,
                                                       const int32_t* __restrict__ table, int64_t nblocks,
                                                       int64_t pieces_per_block, uint32_t* __restrict__ checksum) {
  u32x4 acc = {0u, 0u, 0u, 0u};
  const int tid = threadIdx.x;
  for (int64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const int64_t blk = table != nullptr ? static_cast<int64_t>(table[b]) : b;
    const u32x4* p = src + blk * pieces_per_block + tid;
    for (int64_t r = 0; r < pieces_per_block; r += kThreads * kUnroll) {
      u32x4 v[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        if constexpr (NT)
          v[u] = __builtin_nontemporal_load(p + r + u * kThreads);
        else
          v[u] = p[r + u * kThreads];
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) acc ^= v[u];
    }
  }
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x ^= __shfl_xor(x, m);
  __shared__ uint32_t part[kThreads / 64];
  if ((tid & 63) == 0) part[tid >> 6] = x;
  __syncthreads();
  if (tid == 0) checksum[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

// The eight accumulators are named registers of one inline-assembly block,
// so the compiler can neither merge nor rotate them: eight independent
// dependency chains per wave, each MFMA reading its own previous result.
__global__ __launch_bounds__(kThreads) void mfma_kernel(int32_t waves, int32_t iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = static_cast<__bf16>(static_cast<float>((lane + e) & 7) * 0.125f);
    b[e] = static_cast<__bf16>(static_cast<float>((lane * 3 + e) & 7) * 0.0625f);
  }
  f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0, c4 = c0, c5 = c0, c6 = c0, c7 = c0;
  for (int it = 0; it < iters; ++it) {
    asm volatile(
        "v_mfma_f32_16x16x32_bf16 %0, %8, %9, %0\n\t"
        "v_mfma_f32_16x16x32_bf16 %1, %8, %9, %1\n\t"
        "v_mfma_f32_16x16x32_bf16 %2, %8, %9, %2\n\t"
        "v_mfma_f32_16x16x32_bf16 %3, %8, %9, %3\n\t"
        "v_mfma_f32_16x16x32_bf16 %4, %8, %9, %4\n\t"
        "v_mfma_f32_16x16x32_bf16 %5, %8, %9, %5\n\t"
        "v_mfma_f32_16x16x32_bf16 %6, %8, %9, %6\n\t"
        "v_mfma_f32_16x16x32_bf16 %7, %8, %9, %7"
        : "+v"(c0), "+v"(c1), "+v"(c2), "+v"(c3), "+v"(c4), "+v"(c5), "+v"(c6), "+v"(c7)
        : "v"(a), "v"(b));
  }
  // wait states before vector instructions read the last results
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  const f32x4 c = ((c0 + c1) + (c2 + c3)) + ((c4 + c5) + (c6 + c7));
  const float s = (c[0] + c[1]) + (c[2] + c[3]);
  if (lane == 0 && wave < waves) out[wave] = s;
}

}  // namespace

extern "C" {

int32_t uattn_ceiling_read_grid(void) { return read_grid(); }

int32_t uattn_ceiling_read(const void* src, const int32_t* block_table, int64_t num_blocks, int64_t block_bytes,
                           int32_t flags, uint32_t* checksum, void* stream) {
  if (num_blocks < 0 || block_bytes <= 0 || (flags & ~1) != 0 || (block_bytes % (kThreads * kUnroll * 16)) != 0) return 1;
  if (num_blocks == 0) return 0;
  if (src == nullptr || checksum == nullptr || (reinterpret_cast<uintptr_t>(src) & 15u) != 0) return 1;
  if (flags & 1)
    hipLaunchKernelGGL(read_kernel<true>, dim3(read_grid()), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                       static_cast<const u32x4*>(src), block_table, num_blocks, block_bytes / 16, checksum);
  else
    hipLaunchKernelGGL(read_kernel<false>, dim3(read_grid()), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                       static_cast<const u32x4*>(src), block_table, num_blocks, block_bytes / 16, checksum);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

int32_t uattn_ceiling_mfma(int32_t waves, int32_t iters, float* out, void* stream) {
  if (waves <= 0 || iters <= 0 || out == nullptr) return 1;
  const int blocks = (waves + kThreads / 64 - 1) / (kThreads / 64);
  hipLaunchKernelGGL(mfma_kernel, dim3(blocks), dim3(kThreads), 0, static_cast<hipStream_t>(stream), waves, iters,
                     out);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

}  // extern "C"
