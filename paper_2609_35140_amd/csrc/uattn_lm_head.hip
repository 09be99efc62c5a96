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
  __bf16* out;
  int64_t hs, ws, os;
  int32_t T, V, K, n_vt, n_tt;
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

template <int VT, int TT, int WM, int WN, int STAGES>
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


template <int VT, int TT, int WM, int WN, int STAGES>
hipError_t launch_cfg(LmHeadParams p, hipStream_t stream) {
  p.n_vt = (p.V + VT - 1) / VT;
  p.n_tt = (p.T + TT - 1) / TT;
  const int64_t nblocks = static_cast<int64_t>((p.n_vt + kLmXcds - 1) / kLmXcds) * kLmXcds * p.n_tt;
  if (nblocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((lm_head_kernel<VT, TT, WM, WN, STAGES>), dim3(static_cast<unsigned>(nblocks)),
                     dim3(WM * WN * 64), 0, stream, p);
  return hipGetLastError();
}

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
  return launch_cfg<256, 256, 4, 2, 2>(p, stream);
}

}  // namespace uattn
