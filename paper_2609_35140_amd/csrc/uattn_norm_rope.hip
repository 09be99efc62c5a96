// Q/K RMSNorm + NeoX rotary embedding (one pass), and its rotary table.
//
// A workgroup takes one token's head rows; one row of head_dim bf16 is
// handled by head_dim/8 lanes, 16 bytes (8 elements) each.  The sum of squares
// is summed by each lane over its 8 elements in order, then across the row's
// lanes by an xor butterfly, so every lane of the row holds the same total
// computed in one fixed order.  NeoX pairs element i with i + head_dim/2,
// which lives in the lane head_dim/16 positions away; the two exchange their
// normalized values with one xor shuffle.  Nothing depends on how many rows
// there are or where a row sits, so the full-sequence and token-wise regimes
// produce identical rows.
#include <math.h>

#include "uattn_internal.h"
#include "uattn_numerics.h"

namespace uattn {
namespace {

struct NormRopeParams {
  const __bf16* q;
  const __bf16* k;
  const int32_t* positions;
  const __bf16* qw;
  const __bf16* kw;
  const float* cos_sin;
  __bf16* q_out;
  __bf16* k_out;
  float eps;
  int32_t max_position, num_tokens, hq, hkv;
};

// One workgroup per token: its Hq + Hkv head rows, 256 / (head_dim/8) rows
// per pass (the token's position and rotary row are workgroup-uniform).
template <int D>
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(NormRopeParams p) {
  constexpr int LPR = D / 8;          // lanes per row
  constexpr int RPP = 256 / LPR;      // rows per pass of the workgroup
  constexpr int HALF = LPR / 2;       // lane distance of a NeoX pair
  const int tid = threadIdx.x;
  const int j = tid % LPR;            // 16-byte piece of the row
  const int rows = p.hq + p.hkv;
  const bool first = j < HALF;
  const int i0 = 8 * (first ? j : j - HALF);  // rotary index of element 0 of this lane
  for (int64_t t = blockIdx.x; t < p.num_tokens; t += gridDim.x) {
    const int32_t pos = p.positions[t];
    const bool pos_ok = pos >= 0 && pos < p.max_position;
    float cs[16];
    if (pos_ok) {
      const float4* cp = reinterpret_cast<const float4*>(p.cos_sin + (static_cast<int64_t>(pos) * (D / 2) + i0) * 2);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float4 v4 = cp[u];
        cs[4 * u] = v4.x;
        cs[4 * u + 1] = v4.y;
        cs[4 * u + 2] = v4.z;
        cs[4 * u + 3] = v4.w;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 16; ++u) cs[u] = __builtin_nanf("");
    }
    for (int r0 = 0; r0 < rows; r0 += RPP) {
      const int r = r0 + tid / LPR;
      const bool on = r < rows;
      const bool is_q = r < p.hq;
      const int h = is_q ? r : r - p.hq;
      const __bf16* src = is_q ? p.q + (t * p.hq + h) * D : p.k + (t * p.hkv + h) * D;
      __bf16* dst = is_q ? p.q_out + (t * p.hq + h) * D : p.k_out + (t * p.hkv + h) * D;
      const __bf16* wsrc = is_q ? p.qw : p.kw;
      bf16x8 xv = {}, wv = {};
      if (on) {
        xv = *reinterpret_cast<const bf16x8*>(src + 8 * j);
        wv = *reinterpret_cast<const bf16x8*>(wsrc + 8 * j);
      }
      float x[8];
      float ss = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x[e] = static_cast<float>(xv[e]);
        ss = ss + x[e] * x[e];
      }
#pragma unroll
      for (int m = LPR / 2; m >= 1; m >>= 1) ss = ss + __shfl_xor(ss, m, 64);
      const float r_inv = 1.0f / __builtin_sqrtf(ss / static_cast<float>(D) + p.eps);
      bf16x8 yv;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float n = static_cast<float>(to_bf16(x[e] * r_inv));
        yv[e] = to_bf16(static_cast<float>(wv[e]) * n);
      }
      // the partner lane's normalized values (element i +/- head_dim/2)
      uint4 yu, pu;
      __builtin_memcpy(&yu, &yv, 16);
      pu.x = __shfl_xor(yu.x, HALF, 64);
      pu.y = __shfl_xor(yu.y, HALF, 64);
      pu.z = __shfl_xor(yu.z, HALF, 64);
      pu.w = __shfl_xor(yu.w, HALF, 64);
      bf16x8 pv;
      __builtin_memcpy(&pv, &pu, 16);
      bf16x8 ov;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float c = cs[2 * e], s = cs[2 * e + 1];
        const float y = static_cast<float>(yv[e]), z = static_cast<float>(pv[e]);
        ov[e] = first ? to_bf16(y * c - z * s) : to_bf16(y * c + z * s);
      }
      if (on) *reinterpret_cast<bf16x8*>(dst + 8 * j) = ov;
    }
  }
}

__global__ __launch_bounds__(256) void rope_cache_kernel(float* cos_sin, int32_t max_position, int32_t d, double theta) {
  const int64_t n = static_cast<int64_t>(max_position) * (d / 2);
  for (int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; idx < n;
       idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t pos = idx / (d / 2);
    const int i = static_cast<int>(idx % (d / 2));
    const double inv_freq = pow(theta, -2.0 * i / d);
    const double ang = static_cast<double>(pos) * inv_freq;
    cos_sin[2 * idx] = static_cast<float>(cos(ang));
    cos_sin[2 * idx + 1] = static_cast<float>(sin(ang));
  }
}

}  // namespace

hipError_t launch_qk_norm_rope(const NormRopeLaunch& a, hipStream_t stream) {
  NormRopeParams p;
  p.q = static_cast<const __bf16*>(a.q);
  p.k = static_cast<const __bf16*>(a.k);
  p.positions = a.positions;
  p.qw = static_cast<const __bf16*>(a.q_weight);
  p.kw = static_cast<const __bf16*>(a.k_weight);
  p.cos_sin = a.cos_sin;
  p.q_out = static_cast<__bf16*>(a.q_out);
  p.k_out = static_cast<__bf16*>(a.k_out);
  p.eps = a.eps;
  p.max_position = a.max_position;
  p.num_tokens = a.num_tokens;
  p.hq = a.num_q_heads;
  p.hkv = a.num_kv_heads;
  const dim3 grid(static_cast<unsigned>(a.num_tokens));  // one workgroup per token
  const dim3 block(256);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(qk_norm_rope_kernel<128>, grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL(qk_norm_rope_kernel<64>, grid, block, 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_rope_cache(float* cos_sin, int32_t max_position, int32_t head_dim, double theta, hipStream_t stream) {
  const int64_t n = static_cast<int64_t>(max_position) * (head_dim / 2);
  const int64_t want = (n + 255) / 256;
  const int64_t cap = static_cast<int64_t>(device_cus()) * 16;
  hipLaunchKernelGGL(rope_cache_kernel, dim3(static_cast<unsigned>(want < cap ? want : cap)), dim3(256), 0, stream,
                     cos_sin, max_position, head_dim, theta);
  return hipGetLastError();
}

}  // namespace uattn
