// The per-tile arithmetic shared by every attention kernel in libuattn.
//
// Both entry points (full-sequence prefill and token-wise decode) compute
// each output row through exactly these functions, in the same order, with
// the same instructions.  That is what makes them agree bit for bit: the
// paper names the quantities that must not differ between the two paths
// (Section 3.2: the KV tile boundaries, which fix the online-softmax
// rescaling, the FP32->BF16 conversion of the attention weights and the PV
// accumulation order; Section 5.3: reduction orders of QK^T, PV, softmax and
// normalization, placement of scale and mask, the exact exp/reciprocal
// instructions and subnormal handling, and the order of rescale, update and
// normalize).  Here each of those is pinned:
//
//   * keys are walked in 64-key tiles aligned to the sequence start, in
//     ascending order; a row at position i visits tiles 0 .. i/64 and never a
//     tile that holds no visible key;
//   * tiles are grouped into positional chunks of 256 keys; each chunk starts
//     from (m = -inf, l = 0, acc = 0) and chunk results are folded left to
//     right, whether or not the caller's schedule runs chunks in parallel;
//   * scores S^T = K Q^T and the output O^T = V^T P^T are products on
//     v_mfma_f32_32x32x16_bf16, with queries in the N (column) slots, d and
//     keys consumed in fixed ascending 16-wide K steps starting from zero
//     (scores) or from the rescaled accumulator (output);
//   * the mask is a select to -inf (keys after the query), never a bias;
//   * softmax runs on raw scores with the scale folded into the exponent:
//     p = exp2(fma(s, c, -m*c)) with c = fp32(scale * log2(e)) computed once
//     on the host; alpha = exp2(m_old*c - m_new*c); the hardware v_exp_f32;
//   * l accumulates the fp32 p (in-lane pairwise tree, then the partner
//     half-wave), acc is rescaled by alpha BEFORE the PV product accumulates
//     into it, p is rounded to bf16 (nearest-even) only for the PV product;
//   * no data-dependent skip of any multiply (alpha == 1 included);
//     subnormals are preserved (the kernels' default fp32 denormal mode);
//   * the result is bf16_rne(A / L) with IEEE division.
//
// Floating-point contraction is disabled for everything in this header so
// that the compiler cannot fuse a multiply-add in one kernel and not in the
// other; the only fused operations are the explicit fmaf calls.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace uattn {

constexpr int kTileKeys = 64;
constexpr int kChunkKeys = 256;
constexpr int kTilesPerChunk = kChunkKeys / kTileKeys;
constexpr int kQCols = 32;  // query columns per MFMA (N of 32x32x16)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// LDS row strides (elements).  K tile: [64 keys][D + 8]; V tile: [64 keys][kVStride].
// Both tiles are stored key-major as they come from memory.  The K pad keeps
// 16-lane groups of 128-bit reads on distinct banks; the V stride keeps the
// 32-lane groups of transposing 64-bit reads (see pv_tile) on distinct banks.
template <int D> struct Lds {
  static constexpr int kKStride = D + 8;
  static constexpr int kVStride = D == 128 ? 160 : 96;
  static constexpr int kKElems = kTileKeys * kKStride;
  static constexpr int kVElems = kTileKeys * kVStride;
  static constexpr int kStageElems = kKElems + kVElems;
};

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

__device__ __forceinline__ float hw_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float hw_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ __bf16 to_bf16(float x) { return static_cast<__bf16>(x); }

// ---------------------------------------------------------------------------
// Register <-> key maps of the score tile.
//
// The 32x32 MFMA result holds, in lane half h = lane / 32, register r, the row
// 8*(r/4) + 4*h + r%4 of the 32-row block.  Rows are keys; which key each
// A-operand row carries is chosen so that, after the in-lane regrouping of
// p into the PV operand, every 8 consecutive K slots of the PV product are 8
// consecutive keys (two transposing reads of the V tile, 4 keys each).
// ---------------------------------------------------------------------------
__device__ __forceinline__ constexpr int score_key(int blk, int r, int h) {
  return 32 * blk + 16 * ((r >> 2) >> 1) + 8 * h + 4 * ((r >> 2) & 1) + (r & 3);
}
// Key carried by A-operand row `row` (0..31) of score block `blk`.
__device__ __forceinline__ constexpr int arow_key(int blk, int row) {
  return score_key(blk, ((row >> 3) << 2) | (row & 3), (row >> 2) & 1);
}

// ---------------------------------------------------------------------------
// Scores: s[blk] = K_blk Q^T over d, ascending 16-wide steps from zero.
//   ks_lds : K tile in LDS, [64][Lds<D>::kKStride]
//   qf     : this lane's Q^T operand, qf[step] = q[col][16*step + 8*h .. +7]
// ---------------------------------------------------------------------------
template <int D>
__device__ __forceinline__ void qk_scores(const __bf16* ks_lds, const bf16x8 (&qf)[D / 16], f32x16 (&s)[2], int lane) {
  const int h = lane >> 5, row = lane & 31;
#pragma unroll
  for (int blk = 0; blk < 2; ++blk) {
    const __bf16* krow = ks_lds + arow_key(blk, row) * Lds<D>::kKStride + 8 * h;
    f32x16 acc = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < D / 16; ++st) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + 16 * st);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[st], acc, 0, 0, 0);
    }
    s[blk] = acc;
  }
}

// Select -inf for keys after the query: key position key_base + key > qpos.
__device__ __forceinline__ void mask_scores(f32x16 (&s)[2], int key_base, int qpos, int lane) {
  const int h = lane >> 5;
#pragma unroll
  for (int blk = 0; blk < 2; ++blk)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      s[blk][r] = (key_base + score_key(blk, r, h) > qpos) ? neg_inf() : s[blk][r];
}

// Cross-half partner value (lane ^ 32).
__device__ __forceinline__ float partner(float x) {
  return __shfl_xor(x, 32, 64);
}

// ---------------------------------------------------------------------------
// Online-softmax step for one tile.  In: raw scores s (masked).  Out: s holds
// p = exp2(fma(s, c, -m_new*c)); m, l updated; returns alpha.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float softmax_tile(f32x16 (&s)[2], float& m, float& l, float c) {
  // tile max (exact, order-free)
  float t[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) t[r] = fmaxf(s[0][r], s[1][r]);
#pragma unroll
  for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
    for (int r = 0; r < w; ++r) t[r] = fmaxf(t[r], t[r + w]);
  float tmax = fmaxf(t[0], partner(t[0]));
  const float m_new = fmaxf(m, tmax);
  const float mc_old = m * c;
  const float mc_new = m_new * c;
  const float alpha = hw_exp2(mc_old - mc_new);
#pragma unroll
  for (int blk = 0; blk < 2; ++blk)
#pragma unroll
    for (int r = 0; r < 16; ++r) s[blk][r] = hw_exp2(__builtin_fmaf(s[blk][r], c, -mc_new));
  // row sum: pairwise tree over (blk0 r, blk1 r), then r halves, then partner
  float u[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) u[r] = s[0][r] + s[1][r];
#pragma unroll
  for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
    for (int r = 0; r < w; ++r) u[r] = u[r] + u[r + w];
  const float rs = u[0] + partner(u[0]);
  l = alpha * l + rs;
  m = m_new;
  return alpha;
}

// p (fp32, score layout) -> bf16 PV B-operand: step st, element e holds the
// key 16*st + 8*h + e.
__device__ __forceinline__ void pack_p(const f32x16 (&p)[2], bf16x8 (&pb)[4]) {
#pragma unroll
  for (int st = 0; st < 4; ++st)
#pragma unroll
    for (int e = 0; e < 8; ++e) pb[st][e] = to_bf16(p[st >> 1][4 * (2 * (st & 1) + (e >> 2)) + (e & 3)]);
}

// acc[db] (O^T block db0+db: rows d, cols queries) <- alpha*acc + V^T_db P^T.
//   vs_lds : V tile in LDS, key-major [64][Lds<D>::kVStride]
// The A operand (row d, K slots = keys 16*st + 8*h + e) is gathered with the
// transposing 64-bit LDS read: within each 16-lane group, lane 4a+b receives
// element b of the 4-element rows addressed by lanes a, a+4, a+8, a+12.  So
// source lane s addresses key (base + s/4) at column (group's d base + 4*(s%4)),
// and lane i of the group receives column d base + i for four consecutive keys.
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ s16x4 lds_read_tr16(const __bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
}
template <int D, int NDB>
__device__ __forceinline__ void pv_tile(const __bf16* vs_lds, const bf16x8 (&pb)[4], f32x16 (&acc)[NDB], float alpha,
                                        int db0, int lane) {
  const int g = lane >> 4, s = lane & 15;
  const int h = g >> 1;
  const int key0 = 8 * h + (s >> 2);
  const int col0 = 16 * (g & 1) + 4 * (s & 3);
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = alpha * acc[db][r];
    const __bf16* vb = vs_lds + key0 * Lds<D>::kVStride + 32 * (db0 + db) + col0;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const s16x4 lo = lds_read_tr16(vb + (16 * st) * Lds<D>::kVStride);
      const s16x4 hi = lds_read_tr16(vb + (16 * st + 4) * Lds<D>::kVStride);
      const s16x4 w[2] = {lo, hi};
      bf16x8 a;
      __builtin_memcpy(&a, w, sizeof(a));
      acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[st], acc[db], 0, 0, 0);
    }
  }
}

// ---------------------------------------------------------------------------
// Left fold of chunk partials: (M, L, A) <- (M, L, A) (+) (m, l, acc).
// The first chunk is taken as is (no arithmetic).
// ---------------------------------------------------------------------------
struct FoldScale {
  float a, b, m_new;
};
__device__ __forceinline__ FoldScale fold_scale(float M, float m, float c) {
  FoldScale f;
  f.m_new = fmaxf(M, m);
  const float mc_new = f.m_new * c;
  f.a = hw_exp2(M * c - mc_new);
  f.b = hw_exp2(m * c - mc_new);
  return f;
}
__device__ __forceinline__ float fold_val(const FoldScale& f, float X, float x) { return f.a * X + f.b * x; }

// Final normalization and the optional log-sum-exp (natural log, scaled scores).
__device__ __forceinline__ __bf16 finalize_val(float A, float L) { return to_bf16(A / L); }
__device__ __forceinline__ float finalize_lse(float M, float L, float c) {
  return (M * c + hw_log2(L)) * 0.69314718055994530942f;
}

}  // namespace uattn
