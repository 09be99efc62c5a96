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
//     v_mfma_f32_16x16x32_bf16, with queries in the N (column) slots, d and
//     keys consumed in fixed ascending 32-wide K steps starting from zero
//     (scores) or from the rescaled accumulator (output);
//   * the mask is a select to -inf (keys after the query), never a bias;
//   * softmax runs on raw scores with the scale folded into the exponent:
//     p = exp2(fma(s, c, -m*c)) with c = fp32(scale * log2(e)) computed once
//     on the host; the hardware v_exp_f32;
//   * the running maximum m of a chunk is a reference that moves to a tile's
//     maximum t only when t*c - m*c > kMaxSlack (8; always when m = -inf),
//     with alpha = exp2(m_old*c - t*c); otherwise m stays and alpha is 1, so
//     weights may reach 2^8 (within fp32 and bf16 range, and every weight
//     still carries one bf16 rounding of relative size <= 2^-9);
//   * p is rounded to bf16 (nearest-even) for the PV product, and l is the
//     sum of the same bf16 p, accumulated by that product (an extra all-ones
//     row block); acc and l are rescaled by alpha BEFORE the product
//     accumulates into them;
//   * the alpha multiplies are skipped only when alpha is exactly 1 in every
//     lane of the wave (x * 1 == x, so the bits do not depend on which rows
//     share a wave); no other data-dependent skip; subnormals are preserved
//     (the kernels' default fp32 denormal mode);
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
constexpr int kQCols = 16;   // query columns per MFMA (N of 16x16x32)
constexpr int kKeyBlocks = kTileKeys / 16;  // 16-key M blocks of a score tile
constexpr int kMaxGroup = 2 * kQCols;       // q heads per kv head the decode kernel serves

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

// LDS layout of one pipeline stage: a K tile then a V tile, each [64 keys][D]
// key-major as in memory, with the 16-byte pieces of every row permuted by an
// XOR swizzle so that the two read patterns below hit distinct banks.
template <int D>
struct TileLayout {
  static constexpr int kPieces = D / 8;                  // 16-byte pieces per row
  static constexpr int kTileElems = kTileKeys * D;       // one K or V tile
  static constexpr int kStageElems = 2 * kTileElems;     // K tile then V tile
  static constexpr int kInstrPerWave = kPieces / 4;      // 1 KB instructions per wave per matrix

  // K is read as 16 consecutive rows at one logical piece (16-lane groups of
  // 128-bit reads): spread those rows over 16 distinct bank groups.
  __device__ __forceinline__ static int k_swz(int row) { return D == 128 ? (row & 15) : ((row >> 1) & 7); }
  // V is read by the transposing 64-bit read: 8 consecutive rows x 2 logical
  // pieces (x 2 halves) per 32-lane group.
  __device__ __forceinline__ static int v_swz(int row) { return D == 128 ? 2 * (row & 7) : 2 * ((row >> 1) & 3); }

  // Element offsets inside a stage of (row, d) for K and V.
  __device__ __forceinline__ static int k_off(int row, int d) {
    return row * D + 8 * ((d >> 3) ^ k_swz(row)) + (d & 7);
  }
  __device__ __forceinline__ static int v_off(int row, int d) {
    return kTileElems + row * D + 8 * ((d >> 3) ^ v_swz(row)) + (d & 7);
  }
};

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// The maximum used for every running max and block max: IEEE 754-2019
// maximum (NaN propagates, -0 < +0), one v_maximum3_f32 per three operands.
// The C library maximum would give the same values for the finite and -inf
// operands compared here, but the compiler must then canonicalize each MFMA
// result it reads (an extra v_max_f32 x, x per score).
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ float hw_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// The same v_exp_f32 for a value that inline asm reads.  A VALU instruction
// that reads a transcendental result needs one wait state after it; the
// compiler adds it only between instructions it generated itself, not before
// an asm operand, so the asm here carries its own.
__device__ __forceinline__ float hw_exp2_for_asm(float x) {
  float r;
  asm("v_exp_f32 %0, %1\n\ts_nop 0" : "=v"(r) : "v"(x));
  return r;
}
__device__ __forceinline__ float hw_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ __bf16 to_bf16(float x) { return static_cast<__bf16>(x); }

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Layout of a score tile.  For one group of 16 queries (an N block), lane
// L = 16*g + col holds query column `col` and, in s[kb][j], the score of key
// 16*kb + 4*g + j of the 64-key tile (the 16x16 MFMA result layout: lane L,
// register j holds row 4*(L/16) + j, column L%16).  The four lane groups g
// of one column together hold its 64 keys.
// ---------------------------------------------------------------------------
__device__ __forceinline__ constexpr int score_key(int kb, int j, int g) { return 16 * kb + 4 * g + j; }

// ---------------------------------------------------------------------------
// Scores: s[nb][kb] = K_kb Q_nb^T over d in ascending 32-wide steps from zero.
//   stage  : LDS stage holding the K tile (TileLayout)
//   qf     : this lane's Q^T operands, qf[nb][step] = q[col of nb][32*step + 8*g .. +7]
// ---------------------------------------------------------------------------
template <int D, int NB>
__device__ __forceinline__ void qk_scores(const __bf16* stage, const bf16x8 (&qf)[NB][D / 32], f32x4 (&s)[NB][4],
                                          int lane) {
  using TL = TileLayout<D>;
  const int g = lane >> 4, row = lane & 15;
  const int swz = TL::k_swz(row);  // equals k_swz(16*kb + row) for every kb
#pragma unroll
  for (int kb = 0; kb < kKeyBlocks; ++kb) {
    const __bf16* krow = stage + (16 * kb + row) * D;
    bf16x8 a[D / 32];
#pragma unroll
    for (int st = 0; st < D / 32; ++st) a[st] = *reinterpret_cast<const bf16x8*>(krow + 8 * ((4 * st + g) ^ swz));
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < D / 32; ++st) acc = mfma16(a[st], qf[nb][st], acc);
      s[nb][kb] = acc;
    }
  }
}

// Select -inf for keys after the query: key position key_base + key > qpos,
// i.e. 16*kb + j > qpos - key_base - 4*g, one bound per lane compared with
// constants.
__device__ __forceinline__ void mask_scores(f32x4 (&s)[4], int key_base, int qpos, int lane) {
  const int bound = qpos - key_base - 4 * (lane >> 4);
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int j = 0; j < 4; ++j) s[kb][j] = (score_key(kb, j, 0) > bound) ? neg_inf() : s[kb][j];
}

// Cross-group reductions with the gfx950 lane-swap instructions.  With both
// operands equal, permlane32_swap returns (lanes 0-31 copied to both halves,
// lanes 32-63 copied to both halves) and permlane16_swap does the same for
// the 16-lane halves of each 32-lane half, so combining the two results gives
// every lane the reduction of itself and its lane^32 (lane^16) partner, with
// the operands in the same order in every lane.
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// ---------------------------------------------------------------------------
// Online-softmax step of one query column for one tile, in three pieces that
// every kernel composes in the same order:
//   tile_max      the column maximum of the (masked) raw scores of the tile,
//                 in every lane of the column;
//   advance_max   the reference after the tile (moves to the tile maximum
//                 only past the slack) and its alpha;
//   tile_weights  s <- p = exp2(fma(s, c, -m_new*c)).
// The row sum l is accumulated by the PV product (pv_tile), from the same
// bf16 p that weights V.
//
// The slack keeps the reference (and with it every accumulator) in place for
// all but the rare tile whose scores rise more than 2^8 above it in the exp2
// domain, so the multiplies by alpha -- a quarter of the vector work of a
// tile -- are almost always skipped; the decode walks the same tiles in the
// same order through the same function, so both paths keep the same
// reference.  The fold of chunk partials (fold_scale below) keeps the exact
// running maximum.
// ---------------------------------------------------------------------------
constexpr float kMaxSlack = 8.0f;
__device__ __forceinline__ float tile_max(const f32x4 (&s)[4]) {
  float t[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) t[j] = vmax(vmax(s[0][j], s[1][j]), vmax(s[2][j], s[3][j]));
  float tmax = vmax(vmax(t[0], t[1]), vmax(t[2], t[3]));
  tmax = max_xor16(tmax);
  return max_xor32(tmax);
}
// m <- the reference after a tile whose maximum is tmax; returns alpha.
__device__ __forceinline__ float advance_max(float& m, float tmax, float c) {
  const float mc_old = m * c;
  const float tc = tmax * c;
  const bool move = tc - mc_old > kMaxSlack;  // -inf reference: +inf > slack
  const float alpha = move ? hw_exp2(mc_old - tc) : 1.0f;
  m = move ? tmax : m;
  return alpha;
}
__device__ __forceinline__ void tile_weights(f32x4 (&s)[4], float m_new, float c) {
  const float mc_new = m_new * c;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int j = 0; j < 4; ++j) s[kb][j] = hw_exp2(__builtin_fmaf(s[kb][j], c, -mc_new));
}
// The whole step: m <- the new reference, s <- p; returns alpha.
__device__ __forceinline__ float softmax_tile(f32x4 (&s)[4], float& m, float c) {
  const float alpha = advance_max(m, tile_max(s), c);
  tile_weights(s, m, c);
  return alpha;
}

// True when some lane of the wave has an alpha other than 1 (the multiplies
// by alpha are then issued for every lane; x * 1 == x in the others).
template <int NB>
__device__ __forceinline__ bool any_rescale(const float (&alpha)[NB]) {
  bool r = false;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) r = r || alpha[nb] != 1.0f;
  return __builtin_amdgcn_ballot_w64(r) != 0;
}
// acc <- alpha * acc, lsum <- alpha * lsum for the wave's query columns,
// skipped when every alpha is 1.
template <int NB, int NDB>
__device__ __forceinline__ void rescale_acc(f32x4 (&acc)[NB][NDB], f32x4 (&lsum)[NB], const float (&alpha)[NB]) {
  if (!any_rescale<NB>(alpha)) return;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int j = 0; j < 4; ++j) lsum[nb][j] = alpha[nb] * lsum[nb][j];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[nb][db][j] = alpha[nb] * acc[nb][db][j];
  }
}

// p (fp32, score layout) -> bf16 PV B operand.  Step st covers keys
// 32*st .. 32*st+31; in lane group g, element e holds key
// 32*st + 16*(e/4) + 4*g + e%4, i.e. s[2*st + e/4][e%4].
__device__ __forceinline__ void pack_p(const f32x4 (&p)[4], bf16x8 (&pb)[2]) {
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int e = 0; e < 8; ++e) pb[st][e] = to_bf16(p[2 * st + (e >> 2)][e & 3]);
}

// Transposing 64-bit LDS read (16-bit elements): within each 16-lane group,
// lane 4a+b receives element b of the 4-element rows addressed by lanes a,
// a+4, a+8, a+12.
__device__ __forceinline__ s16x4 lds_read_tr16(const __bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
}

// acc[nb][db] (O^T block: rows d = 16*(db0+db) + 4*g + j, column = query of nb)
//   <- alpha[nb] * acc + V^T_db P_nb^T, K steps st = 0, 1 in order (the
//   multiplies by alpha through rescale_acc, all before the first product);
// lsum[nb] <- alpha[nb] * lsum + 1^T P_nb^T: the same product with an all-ones
// operand in place of V^T, so every register of lsum holds the column's
// running sum of the bf16 weights (l).
//   vtile  : LDS V tile, [64 keys][D] with the TileLayout V swizzle
// The V^T operand of step st for d block db (lane i of group g: row d = 16*db + i,
// keys 32*st + 16*h + 4*g + k for the two halves h) comes from two transposing
// reads whose source lane s addresses key (32*st + 16*h + 4*g + s/4), column
// 16*db + 4*(s%4).
//
// kFirst: the first tile of a chunk, where acc and lsum are zero and alpha is
// zero (the running maximum starts at -inf), so alpha * acc is +0 and the
// products start from a zero accumulator instead: the same bits for finite
// scores, without the multiplies.
template <int D, int NB, int NDB, bool kFirst = false>
__device__ __forceinline__ void pv_tile(const __bf16* vtile, const bf16x8 (&pb)[NB][2], f32x4 (&acc)[NB][NDB],
                                        f32x4 (&lsum)[NB], const float (&alpha)[NB], int db0, int lane) {
  using TL = TileLayout<D>;
  const int g = lane >> 4, src = lane & 15;
  const int key = 4 * g + (src >> 2);       // + 32*st + 16*half; the swizzle depends on key bits below 16
  const int swz = TL::v_swz(key);
  const int sub = src & 3;                  // 4-column group inside the 16-wide d block
  const __bf16* vrow = vtile + key * D + 4 * (sub & 1);
  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = static_cast<__bf16>(1.0f);
  if constexpr (!kFirst) rescale_acc<NB, NDB>(acc, lsum, alpha);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if constexpr (kFirst) lsum[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 2; ++st) lsum[nb] = mfma16(ones, pb[nb][st], lsum[nb]);
  }
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    const int piece = (2 * (db0 + db) + (sub >> 1)) ^ swz;
    bf16x8 a[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const s16x4 lo = lds_read_tr16(vrow + (32 * st) * D + 8 * piece);
      const s16x4 hi = lds_read_tr16(vrow + (32 * st + 16) * D + 8 * piece);
      const s16x4 w[2] = {lo, hi};
      __builtin_memcpy(&a[st], w, sizeof(bf16x8));
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if constexpr (kFirst) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 2; ++st) acc[nb][db] = mfma16(a[st], pb[nb][st], acc[nb][db]);
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
  f.m_new = vmax(M, m);
  const float mc_new = f.m_new * c;
  f.a = hw_exp2_for_asm(M * c - mc_new);  // read by fold_val_tied's asm
  f.b = hw_exp2(m * c - mc_new);
  return f;
}
// a*X + b*x with one rounding for the sum: fma(a, X, b*x)
__device__ __forceinline__ float fold_val(const FoldScale& f, float X, float x) {
  return __builtin_fmaf(f.a, X, f.b * x);
}
// The same operation with the result in X's register.  Written as the three-operand
// v_fma_f32 so that the sum lands in X's register: from fmaf the compiler
// picks the two-operand form, whose result shares the product's register,
// and then copies every folded value back (two moves per element of a
// prefill fold).
__device__ __forceinline__ float fold_val_tied(const FoldScale& f, float X, float x) {
  const float bx = f.b * x;
  float r;
  // operands: %0 = r (tied to X, %2), %1 = a, %3 = b*x
  asm("v_fma_f32 %0, %1, %0, %3" : "=v"(r) : "v"(f.a), "0"(X), "v"(bx));
  return r;
}

// Final normalization and the optional log-sum-exp (natural log, scaled scores).
__device__ __forceinline__ __bf16 finalize_val(float A, float L) { return to_bf16(A / L); }
__device__ __forceinline__ float finalize_lse(float M, float L, float c) {
  return (M * c + hw_log2(L)) * 0.69314718055994530942f;
}

}  // namespace uattn
