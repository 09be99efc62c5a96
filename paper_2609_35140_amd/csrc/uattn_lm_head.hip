// Batch-invariant LM head: logits = bf16(hidden . weight^T).
//
// Each MFMA computes a 16 (vocab) x 16 (token) block of logits^T = W H^T, so
// a lane's four results are four consecutive vocab entries of one token (one
// 8-byte store).  Workgroup = 8 waves = 256 vocab rows x 256 tokens; wave
// (wm, wn) owns 64 vocab x 128 tokens (4 x 8 blocks), so each 16-byte LDS
// operand read feeds 4 or 8 MFMAs.  K (the hidden dimension) is walked in
// 64-wide chunks through a two-stage LDS ring filled by direct-to-LDS loads
// (16-byte pieces XOR-swizzled by row, so the 16-lane operand reads hit
// distinct banks), and every accumulator steps K in ascending 32-wide MFMA
// steps from zero: a row's logits never depend on the batch, its size or the
// row's place in a tile.
//
// Workgroup order: the hardware deals consecutive ids to the 8 XCDs in turn;
// id -> (vocab tile, token tile) keeps one vocab tile's weights (2 MB for
// hidden 4096) on one XCD while all token tiles pass, so they stay in that
// XCD's L2 and the hidden rows stream from the shared cache.
//
// Fused log-probability epilogue (uattn_lm_head_logprob): instead of (or as
// well as) storing the bf16 logits, the workgroup reduces each token's 256
// logits of its vocab tile to a partial (max, sum of exp) pair and picks out
// the target's logit when the target lies in the tile; a second kernel folds
// each token's partials in ascending vocab-tile order.  Every reduction has
// a structure fixed by vocab positions alone (lane, wave and tile order), so
// a token's result does not depend on the batch or its place in it.
#include "uattn_internal.h"
#include "uattn_numerics.h"
#include "uattn_tile_io.h"

namespace uattn {
namespace {

constexpr int kKC = 64;       // hidden elements per chunk
constexpr int kLmXcds = 8;

struct LmHeadParams {
  const __bf16* h;
  const __bf16* w;
  __bf16* out;          // logits, or nullptr (fused log-prob without stored logits)
  int64_t hs, ws, os;
  int32_t T, V, K, n_vt, n_tt;
  // fused log-prob epilogue
  const int32_t* targets;
  float* part_m;        // [n_vt][T] tile max of the raw bf16 logits
  float* part_s;        // [n_vt][T] sum over the tile of exp2(fma(x, k, -m*k))
  float* y_logit;       // [T] the target's raw bf16 logit
  float k;              // inv_temperature * log2(e)
};

// VT vocab rows x TT tokens per workgroup, WM x WN waves (wave tile
// VT/WM x TT/WN), a ring of STAGES chunks.
template <int VT, int TT, int WM, int WN, int STAGES>
struct LmCfg {
  static constexpr int NW = WM * WN;       // waves per workgroup
  static constexpr int BI = VT / WM / 16;   // 16-row vocab blocks per wave
  static constexpr int BJ = TT / WN / 16;   // 16-column token blocks per wave
  static constexpr int kAInstr = VT * kKC * 2 / 1024 / NW;  // 1 KB direct-to-LDS loads per wave per chunk
  static constexpr int kBInstr = TT * kKC * 2 / 1024 / NW;
  static_assert(kAInstr * 1024 * NW == VT * kKC * 2 && kBInstr * 1024 * NW == TT * kKC * 2, "chunk split");
  static constexpr int kChunkOps = kAInstr + kBInstr;
  struct Smem {
    __bf16 a[STAGES][VT * kKC];   // weight rows, 128 bytes each, pieces swizzled
    __bf16 b[STAGES][TT * kKC];   // hidden rows
  };
};

template <int VT, int TT, int WM, int WN, int STAGES, bool kLogprob>
__global__ __launch_bounds__(WM * WN * 64, 1) void lm_head_kernel(LmHeadParams p) {
  using C = LmCfg<VT, TT, WM, WN, STAGES>;
  constexpr int BI = C::BI, BJ = C::BJ;
  __shared__ __attribute__((aligned(1024))) typename C::Smem sm;
  const int pid = blockIdx.x;
  const int xcd = pid % kLmXcds, kk = pid / kLmXcds;
  const int vt = xcd + kLmXcds * (kk / p.n_tt);
  const int tt = kk % p.n_tt;
  if (vt >= p.n_vt) return;
  const int v0 = vt * VT, t0 = tt * TT;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WM, wn = wave / WM;
  const __bf16* zero = reinterpret_cast<const __bf16*>(g_zero_rows) + 8 * (lane & 15);

  // chunk c (hidden elements 64c .. 64c+63) of this workgroup's rows into stage c % STAGES
  auto issue_chunk = [&](int c) {
    const int k0 = c * kKC;
    __bf16* a = &sm.a[c % STAGES][0];
    __bf16* b = &sm.b[c % STAGES][0];
#pragma unroll
    for (int i = 0; i < C::kAInstr; ++i) {
      const int slot = (wave * C::kAInstr + i) * 64 + lane;
      const int row = slot >> 3, lp = (slot & 7) ^ (row & 7);
      const __bf16* src = (v0 + row < p.V) ? p.w + static_cast<int64_t>(v0 + row) * p.ws + k0 + 8 * lp : zero;
      dma_b128(src, __builtin_amdgcn_readfirstlane(lds_addr(a + (wave * C::kAInstr + i) * 512)));
    }
#pragma unroll
    for (int i = 0; i < C::kBInstr; ++i) {
      const int slot = (wave * C::kBInstr + i) * 64 + lane;
      const int row = slot >> 3, lp = (slot & 7) ^ (row & 7);
      const __bf16* src = (t0 + row < p.T) ? p.h + static_cast<int64_t>(t0 + row) * p.hs + k0 + 8 * lp : zero;
      dma_b128(src, __builtin_amdgcn_readfirstlane(lds_addr(b + (wave * C::kBInstr + i) * 512)));
    }
  };

  f32x4 acc[BI][BJ];
#pragma unroll
  for (int i = 0; i < BI; ++i)
#pragma unroll
    for (int j = 0; j < BJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = p.K / kKC;
#pragma unroll
  for (int c = 0; c < STAGES - 1; ++c)
    if (c < nk) issue_chunk(c);
  const int r16 = lane & 15, g = lane >> 4;
  // the fused epilogue's targets, read before the K loop so that their round trip hides behind it
  int ytgt[kLogprob ? BJ : 1];
  if constexpr (kLogprob) {
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const int t = t0 + (TT / WN) * wn + 16 * j + r16;
      ytgt[j] = t < p.T ? p.targets[t] : -1;
    }
  }
#pragma unroll 1
  for (int c = 0; c < nk; ++c) {
    // chunk c has landed once only the chunks issued after it may still load;
    // after the barrier every wave is also done with chunk c-1, whose stage
    // takes chunk c + STAGES - 1
    wait_tiles_barrier<C::kChunkOps>(min(STAGES - 2, nk - 1 - c));
    if (c + STAGES - 1 < nk) issue_chunk(c + STAGES - 1);
    const __bf16* a = &sm.a[c % STAGES][0];
    const __bf16* b = &sm.b[c % STAGES][0];
#pragma unroll
    for (int s = 0; s < kKC / 32; ++s) {
      const int lp = 4 * s + g;
      bf16x8 av[BI], bv[BJ];
#pragma unroll
      for (int i = 0; i < BI; ++i) {
        const int row = (VT / WM) * wm + 16 * i + r16;
        av[i] = *reinterpret_cast<const bf16x8*>(a + row * kKC + 8 * (lp ^ (row & 7)));
      }
#pragma unroll
      for (int j = 0; j < BJ; ++j) {
        const int row = (TT / WN) * wn + 16 * j + r16;
        bv[j] = *reinterpret_cast<const bf16x8*>(b + row * kKC + 8 * (lp ^ (row & 7)));
      }
#pragma unroll
      for (int i = 0; i < BI; ++i)
#pragma unroll
        for (int j = 0; j < BJ; ++j) acc[i][j] = mfma16(av[i], bv[j], acc[i][j]);
    }
  }

  // lane: token 16j + r16 of the wave's columns, vocab 16i + 4g .. +3 of its rows
  if (p.out != nullptr) {
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const int t = t0 + (TT / WN) * wn + 16 * j + r16;
      if (t >= p.T) continue;
      __bf16* orow = p.out + static_cast<int64_t>(t) * p.os;
#pragma unroll
      for (int i = 0; i < BI; ++i) {
        const int v = v0 + (VT / WM) * wm + 16 * i + 4 * g;
        bf16x4 o;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) o[jj] = to_bf16(acc[i][j][jj]);
        if (v + 3 < p.V) {
          *reinterpret_cast<bf16x4*>(orow + v) = o;
        } else {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            if (v + jj < p.V) orow[v + jj] = o[jj];
        }
      }
    }
  }
  if constexpr (kLogprob) {
    static_assert(VT == 256 && WM == 4 && TT <= 256, "reduction layout: four waves of 64 vocab entries");
    // the K loop's LDS is free once every wave is past its last chunk
    lds_barrier();
    float* red = reinterpret_cast<float*>(&sm);   // [WM][TT] per-wave maxima, then per-wave sums
    const float k = p.k;
    // x = the stored bf16 logit (raw; the temperature sits in k), -inf past the vocabulary
    float x[BJ][BI][4];
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const int tl = (TT / WN) * wn + 16 * j + r16;
      const int t = t0 + tl;
      const int y = ytgt[j];
#pragma unroll
      for (int i = 0; i < BI; ++i) {
        const int v = v0 + (VT / WM) * wm + 16 * i + 4 * g;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const float xv = static_cast<float>(to_bf16(acc[i][j][jj]));
          x[j][i][jj] = (v + jj < p.V) ? xv : neg_inf();
          if (v + jj == y) p.y_logit[t] = xv;
        }
      }
      // the wave's maximum over its 64 entries of this token (max is exact: any order)
      float mx = neg_inf();
#pragma unroll
      for (int i = 0; i < BI; ++i) mx = vmax(vmax(mx, vmax(x[j][i][0], x[j][i][1])), vmax(x[j][i][2], x[j][i][3]));
      mx = max_xor32(max_xor16(mx));
      if (g == 0) red[wm * TT + tl] = mx;
    }
    lds_barrier();
    float m_tile[BJ];
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const int tl = (TT / WN) * wn + 16 * j + r16;
      m_tile[j] = vmax(vmax(red[tl], red[TT + tl]), vmax(red[2 * TT + tl], red[3 * TT + tl]));
    }
    lds_barrier();
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const int tl = (TT / WN) * wn + 16 * j + r16;
      const float mk = m_tile[j] * k;
      // fixed order: the four values of a block in pairs, then the blocks in pairs
      float sb[BI];
#pragma unroll
      for (int i = 0; i < BI; ++i) {
        float e[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) e[jj] = hw_exp2(__builtin_fmaf(x[j][i][jj], k, -mk));
        sb[i] = (e[0] + e[1]) + (e[2] + e[3]);
      }
      float sum = (sb[0] + sb[1]) + (sb[2] + sb[3]);
      // the four lane groups of the column: the same pairs in every lane
      sum = sum + __shfl_xor(sum, 16, 64);
      sum = sum + __shfl_xor(sum, 32, 64);
      if (g == 0) red[wm * TT + tl] = sum;
    }
    lds_barrier();
    if (tid < TT) {
      const int t = t0 + tid;
      if (t < p.T) {
        const float s4 = (red[tid] + red[TT + tid]) + (red[2 * TT + tid] + red[3 * TT + tid]);
        p.part_s[static_cast<int64_t>(vt) * p.T + t] = s4;
      }
    }
    // the tile maxima (the same value in every wave): lanes g == 0 of the waves wm == 0 write them
    if (wm == 0 && g == 0) {
#pragma unroll
      for (int j = 0; j < BJ; ++j) {
        const int t = t0 + (TT / WN) * wn + 16 * j + r16;
        if (t < p.T) p.part_m[static_cast<int64_t>(vt) * p.T + t] = m_tile[j];
      }
    }
  }
}

// Fold of a token's vocab-tile partials in ascending tile order, then
//   logp = (x_y - M) * inv_temperature - log2(S) * ln 2
// (S is the sum of exp2((x - M) * inv_temperature * log2 e)).  The partials
// are loaded kFoldBatch tiles at a time ahead of their fold, so the fold's
// sequential chain does not wait for one memory round trip per tile.
constexpr int kFoldBatch = 16;
__global__ __launch_bounds__(256) void logprob_fold_kernel(const float* __restrict__ part_m,
                                                           const float* __restrict__ part_s,
                                                           const float* __restrict__ y_logit,
                                                           const int32_t* __restrict__ targets, int32_t T, int32_t V,
                                                           int32_t n_vt, float it, float k, float* __restrict__ logp) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  const int y = targets[t];
  const float xy = (y >= 0 && y < V) ? y_logit[t] : 0.f;
  float M = 0.f, S = 0.f;
  for (int v0 = 0; v0 < n_vt; v0 += kFoldBatch) {
    float bm[kFoldBatch], bs[kFoldBatch];
#pragma unroll
    for (int i = 0; i < kFoldBatch; ++i) {
      const int64_t vt = min(v0 + i, n_vt - 1);
      bm[i] = part_m[vt * T + t];
      bs[i] = part_s[vt * T + t];
    }
#pragma unroll
    for (int i = 0; i < kFoldBatch; ++i) {
      const int vt = v0 + i;
      if (vt >= n_vt) break;
      if (vt == 0) {
        M = bm[i];
        S = bs[i];
      } else {
        const float mn = vmax(M, bm[i]);
        const float mk = mn * k;
        S = S * hw_exp2(M * k - mk) + bs[i] * hw_exp2(bm[i] * k - mk);
        M = mn;
      }
    }
  }
  logp[t] = (y < 0 || y >= V) ? __builtin_nanf("") : (xy - M) * it - hw_log2(S) * 0.69314718055994530942f;
}

template <int VT, int TT, int WM, int WN, int STAGES, bool kLogprob>
hipError_t launch_cfg(LmHeadParams p, hipStream_t stream) {
  p.n_vt = (p.V + VT - 1) / VT;
  p.n_tt = (p.T + TT - 1) / TT;
  const int64_t nblocks = static_cast<int64_t>((p.n_vt + kLmXcds - 1) / kLmXcds) * kLmXcds * p.n_tt;
  if (nblocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((lm_head_kernel<VT, TT, WM, WN, STAGES, kLogprob>), dim3(static_cast<unsigned>(nblocks)),
                     dim3(WM * WN * 64), 0, stream, p);
  return hipGetLastError();
}

constexpr int kVocabTile = 256;

}  // namespace

hipError_t launch_lm_head(const LmHeadLaunch& a, hipStream_t stream) {
  LmHeadParams p;
  p.h = static_cast<const __bf16*>(a.hidden);
  p.w = static_cast<const __bf16*>(a.weight);
  p.out = static_cast<__bf16*>(a.logits);
  p.hs = a.hidden_stride;
  p.ws = a.weight_stride;
  p.os = a.logits_stride;
  p.T = a.num_rows;
  p.V = a.vocab;
  p.K = a.hidden_dim;
  p.targets = nullptr;
  p.part_m = p.part_s = p.y_logit = nullptr;
  p.k = 0.f;
  return launch_cfg<kVocabTile, 256, 4, 2, 2, false>(p, stream);
}

size_t lm_head_logprob_ws_bytes(int64_t num_rows, int64_t vocab) {
  const int64_t n_vt = (vocab + kVocabTile - 1) / kVocabTile;
  return static_cast<size_t>((2 * n_vt + 1) * num_rows) * sizeof(float);
}

hipError_t launch_lm_head_logprob(const LmHeadLaunch& a, const int32_t* targets, float inv_temperature, float* logp,
                                  void* workspace, hipStream_t stream) {
  LmHeadParams p;
  p.h = static_cast<const __bf16*>(a.hidden);
  p.w = static_cast<const __bf16*>(a.weight);
  p.out = static_cast<__bf16*>(a.logits);
  p.hs = a.hidden_stride;
  p.ws = a.weight_stride;
  p.os = a.logits_stride;
  p.T = a.num_rows;
  p.V = a.vocab;
  p.K = a.hidden_dim;
  const int64_t n_vt = (a.vocab + kVocabTile - 1) / kVocabTile;
  float* ws = static_cast<float*>(workspace);
  p.targets = targets;
  p.part_m = ws;
  p.part_s = ws + n_vt * a.num_rows;
  p.y_logit = ws + 2 * n_vt * a.num_rows;
  p.k = static_cast<float>(static_cast<double>(inv_temperature) * 1.4426950408889634);
  hipError_t e = launch_cfg<kVocabTile, 256, 4, 2, 2, true>(p, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(logprob_fold_kernel, dim3((a.num_rows + 255) / 256), dim3(256), 0, stream, p.part_m, p.part_s,
                     p.y_logit, targets, a.num_rows, a.vocab, static_cast<int32_t>(n_vt), inv_temperature, p.k, logp);
  return hipGetLastError();
}

}  // namespace uattn
