// Per-token log-probability: logp = x[y] - logsumexp(x), x = logits * inv_temperature.
//
// One workgroup (256 threads) per row.  Thread t streams the row's 16-byte
// vectors t, t+256, t+512, ... keeping an online (max, sum) pair; the 256
// pairs are then combined by a fixed butterfly inside each wave and a fixed
// pairing of the four waves.  The reduction structure depends only on vocab,
// never on the number of rows or a row's position, so a row's result is
// bit-identical in any batch (the precondition for reusing rollout
// log-probabilities with ratio exactly 1).
//
// The temperature is folded into the exponent: with k = inv_temperature *
// log2(e) and m the row max of the raw logits (inv_temperature > 0),
//   sum = sum_v exp2(fma(logit_v, k, -m*k)),
//   logp = (logit_y - m) * inv_temperature - log2(sum) * ln(2).
#include "uattn_internal.h"
#include "uattn_numerics.h"

#pragma clang fp contract(off)

namespace uattn {
namespace {

constexpr int kThreads = 256;

struct MaxSum {
  float m, s;
};

// Factor that moves a sum kept relative to max `from` to max `to` (to >= from).
__device__ __forceinline__ float rebase(float from, float to, float k) {
  return from == neg_inf() ? 0.f : hw_exp2(from * k - to * k);
}

__device__ __forceinline__ MaxSum combine(MaxSum a, MaxSum b, float k) {
  MaxSum r;
  r.m = fmaxf(a.m, b.m);
  r.s = a.s * rebase(a.m, r.m, k) + b.s * rebase(b.m, r.m, k);
  return r;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__global__ __launch_bounds__(kThreads) void logprob_kernel(const uint16_t* __restrict__ logits, int64_t stride,
                                                           const int32_t* __restrict__ targets, int vocab, float it,
                                                           float k, float* __restrict__ logp) {
  const int row = blockIdx.x, tid = threadIdx.x;
  const uint16_t* x = logits + static_cast<int64_t>(row) * stride;
  MaxSum acc{neg_inf(), 0.f};
  const int nvec = vocab / 8;
  for (int i = tid; i < nvec; i += kThreads) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(x + 8 * static_cast<int64_t>(i));
    float f[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f[2 * j] = bf16_lo(w[j]);
      f[2 * j + 1] = bf16_hi(w[j]);
    }
    const float mx = fmaxf(fmaxf(fmaxf(f[0], f[1]), fmaxf(f[2], f[3])), fmaxf(fmaxf(f[4], f[5]), fmaxf(f[6], f[7])));
    const float m_new = fmaxf(acc.m, mx);
    const float mk = m_new * k;
    float e[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) e[j] = hw_exp2(__builtin_fmaf(f[j], k, -mk));
    const float sum8 = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
    acc.s = acc.s * rebase(acc.m, m_new, k) + sum8;
    acc.m = m_new;
  }
  for (int i = 8 * nvec + tid; i < vocab; i += kThreads) {
    const float f = __uint_as_float(static_cast<uint32_t>(x[i]) << 16);
    const float m_new = fmaxf(acc.m, f);
    acc.s = acc.s * rebase(acc.m, m_new, k) + hw_exp2(__builtin_fmaf(f, k, -(m_new * k)));
    acc.m = m_new;
  }
  // wave butterfly (combine is commutative, so every lane ends with the same pair)
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    MaxSum o{__shfl_xor(acc.m, off, 64), __shfl_xor(acc.s, off, 64)};
    acc = combine(acc, o, k);
  }
  __shared__ MaxSum part[kThreads / 64];
  if ((tid & 63) == 0) part[tid >> 6] = acc;
  __syncthreads();
  if (tid == 0) {
    const MaxSum r = combine(combine(part[0], part[1], k), combine(part[2], part[3], k), k);
    const int y = targets[row];
    if (y < 0 || y >= vocab) {
      logp[row] = __builtin_nanf("");
    } else {
      const float xy = __uint_as_float(static_cast<uint32_t>(x[y]) << 16);
      logp[row] = (xy - r.m) * it - hw_log2(r.s) * 0.69314718055994530942f;
    }
  }
}

}  // namespace

hipError_t launch_logprob(const LogprobLaunch& a, hipStream_t stream) {
  const float k = static_cast<float>(static_cast<double>(a.inv_temperature) * 1.4426950408889634);
  hipLaunchKernelGGL(logprob_kernel, dim3(a.num_rows), dim3(kThreads), 0, stream,
                     static_cast<const uint16_t*>(a.logits), a.row_stride, a.targets, a.vocab, a.inv_temperature, k,
                     a.logp);
  return hipGetLastError();
}

}  // namespace uattn
