// Full-sequence entry point: causal GQA attention over a packed varlen batch.
//
// Workgroup = 8 waves = 256 consecutive query rows of one q head of one
// sequence; wave w owns rows q0 .. q0+31 (q0 = tile*256 + 32*w), two 16-column
// MFMA blocks, one row per column.  Two waves share each SIMD.  All waves
// stream the same K/V tiles through a two-stage LDS ring filled by
// direct-to-LDS loads; a wave stops at its own diagonal tile (q0 / 64), so no
// row ever sees a tile without a visible key.  Every row's arithmetic is the
// shared per-tile sequence in uattn_numerics.h, chunk-folded every 4 tiles,
// exactly as the decode path folds its positional split.
//
// Grid: one dimension; see the workgroup-id mapping below (query tiles counted
// from the END of each sequence, so the longest work is dispatched first, and
// the q heads sharing a kv head kept on one XCD).
#include <type_traits>
#include "uattn_internal.h"
#include "uattn_numerics.h"
#include "uattn_tile_io.h"

namespace uattn {
namespace {

#ifndef UATTN_PREFILL_WAVES
#define UATTN_PREFILL_WAVES 8
#endif
constexpr int kWaves = UATTN_PREFILL_WAVES;
#ifndef UATTN_PREFILL_NB
#define UATTN_PREFILL_NB 2
#endif
constexpr int kNB = UATTN_PREFILL_NB;        // 16-column MFMA blocks (query groups) per wave
constexpr int kWaveRows = kNB * kQCols;
constexpr int kWgRows = kWaves * kWaveRows;
#ifndef UATTN_PREFILL_STAGES
#define UATTN_PREFILL_STAGES 2
#endif
constexpr int kStages = UATTN_PREFILL_STAGES;  // LDS ring: tiles are issued kStages-1 ahead

struct PrefillParams {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const int32_t* cu;
  __bf16* out;
  float* lse;
  int hq, hkv, group, total;
  int num_seqs, ngroups;  // work groups = (query tile from the end, sequence, kv head)
  float c;
};

// Hardware dispatch hands consecutive workgroup ids to the 8 XCDs in turn, and
// each XCD has its own L2.  Workgroup id -> (work group, q head in group) so
// that the G q heads of one (tile, sequence, kv head), which read the same K/V
// tiles, run back to back on the same XCD, while work groups are spread over
// XCDs in descending-cost order (query tiles counted from the end first).
constexpr int kXcds = 8;

template <int D>
__global__ __launch_bounds__(kWaves * 64, 8 / kWaves) void prefill_kernel(PrefillParams p) {
  constexpr int NDB = D / 16;  // 16-wide d blocks of the output
  using TL = TileLayout<D>;
  __shared__ __attribute__((aligned(1024))) __bf16 lds[kStages * TL::kStageElems];

  const int pid = blockIdx.x;
  const int k = pid / kXcds, gi = k % p.group;
  const int wgroup = (k / p.group) * kXcds + pid % kXcds;
  if (wgroup >= p.ngroups) return;
  const int per_tile = p.num_seqs * p.hkv;
  const int zrev = wgroup / per_tile;
  const int seq = (wgroup % per_tile) / p.hkv;
  const int kvh = wgroup % p.hkv;
  const int head = kvh * p.group + gi;
  // clamp the (trusted) offsets so that a malformed table cannot index outside the tensors
  const int lo = min(max(p.cu[seq], 0), p.total);
  const int L = max(min(p.cu[seq + 1], p.total) - lo, 0);
  const int nqt = (L + kWgRows - 1) / kWgRows;
  const int qt = nqt - 1 - zrev;
  if (qt < 0) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int g = lane >> 4, col = lane & 15;
  const int q0 = qt * kWgRows + wave * kWaveRows;
  const bool wave_on = q0 < L;
  const int last_q0 = min(qt * kWgRows + kWgRows - kWaveRows, ((L - 1) / kWaveRows) * kWaveRows);
  const int wg_last_tile = last_q0 / kTileKeys;
  const int my_last_tile = q0 / kTileKeys;

  // this lane's Q^T operands: query q0 + 16*nb + col, d = 32*step + 8*g .. +7
  bf16x8 qf[kNB][D / 32];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const int qp = q0 + kQCols * nb + col;
    if (wave_on && qp < L) {
      const __bf16* qrow = p.q + (static_cast<int64_t>(lo + qp) * p.hq + head) * D + 8 * g;
#pragma unroll
      for (int st = 0; st < D / 32; ++st) qf[nb][st] = *reinterpret_cast<const bf16x8*>(qrow + 32 * st);
    } else {
#pragma unroll
      for (int st = 0; st < D / 32; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[nb][st][e] = static_cast<__bf16>(0.0f);
    }
  }

  constexpr int RPW = kTileKeys / kWaves;
  const int64_t row_stride = static_cast<int64_t>(p.hkv) * D;
  auto issue_tile = [&](int t) {  // this wave's rows of tile t into stage t % kStages
    const int pos = t * kTileKeys + RPW * wave;
    const int64_t off = (static_cast<int64_t>(lo + pos) * p.hkv + kvh) * D;
    load_tile_rows_async<D, RPW>(lds + (t % kStages) * TL::kStageElems, p.k + off, p.v + off, row_stride, L - pos,
                                 wave, lane);
  };

  f32x4 acc[kNB][NDB], A[kNB][NDB], lsum[kNB];
  float m[kNB], M[kNB], Ls[kNB];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
      A[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    m[nb] = neg_inf();
    lsum[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    M[nb] = neg_inf();
    Ls[nb] = 0.f;
  }
  const float c = p.c;

#pragma unroll
  for (int t = 0; t < kStages - 1; ++t)
    if (t <= wg_last_tile) issue_tile(t);
  // The Q^T operands have landed (and with them the first tiles).  Said with
  // the compiler's own wait, so that it knows: otherwise it keeps the Q loads
  // pending through the loop (it cannot see the waits written in assembly)
  // and waits on the vector-memory count before each tile's first product,
  // which then also waits for the next tile's loads.
  wait_vmem_below<0>();
  // tile t, in stage SI = t % kStages, at position POS = t % 4 of its chunk
  auto tile_step = [&](int t, auto stage_const, auto pos_const) {
    constexpr int SI = decltype(stage_const)::value;
    constexpr int POS = decltype(pos_const)::value;
    __bf16* stage = lds + SI * TL::kStageElems;
    // this wave's rows of tile t are in LDS once only the later tiles' loads
    // remain; after the barrier every wave's rows are, and every wave is done
    // with tile t-1
    wait_tiles_barrier<TileLoads<D, RPW>::kPerTile>(min(kStages - 2, wg_last_tile - t));
    if (t + kStages - 1 <= wg_last_tile) issue_tile(t + kStages - 1);
    if (wave_on && t <= my_last_tile) {
      f32x4 s[kNB][4];
      qk_scores<D, kNB>(stage, qf, s, lane);
      float alpha[kNB];
      bf16x8 pb[kNB][2];
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) {
        if (t == my_last_tile) mask_scores(s[nb], t * kTileKeys, q0 + kQCols * nb + col, lane);
        alpha[nb] = softmax_tile(s[nb], m[nb], c);
        pack_p(s[nb], pb[nb]);
      }
      // a chunk's first tile starts its accumulators afresh (pv_tile kFirst)
      pv_tile<D, kNB, NDB, POS == 0>(stage + TL::kTileElems, pb, acc, lsum, alpha, 0, lane);
      if (t == my_last_tile || POS == kTilesPerChunk - 1) {
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) {
          if (t < kTilesPerChunk) {
            M[nb] = m[nb];
            Ls[nb] = lsum[nb][0];
#pragma unroll
            for (int db = 0; db < NDB; ++db) A[nb][db] = acc[nb][db];
          } else {
            const FoldScale f = fold_scale(M[nb], m[nb], c);
            Ls[nb] = fold_val(f, Ls[nb], lsum[nb][0]);
#pragma unroll
            for (int db = 0; db < NDB; ++db)
#pragma unroll
              for (int j = 0; j < 4; ++j) A[nb][db][j] = fold_val_tied(f, A[nb][db][j], acc[nb][db][j]);
            M[nb] = f.m_new;
          }
          m[nb] = neg_inf();  // acc and lsum restart at the next chunk's first tile
        }
      }
    }
  };
  // The tile loop is unrolled by a chunk (4 tiles, two rounds of the stage
  // ring), so that every LDS address of a stage is a constant offset from one
  // base and a tile's place in its chunk is known at compile time.
  static_assert(kStages == 2 && kTilesPerChunk == 4, "unrolled by a chunk of two stage rounds");
  for (int t = 0; t <= wg_last_tile; t += 4) {
    tile_step(t, std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{});
    if (t + 1 <= wg_last_tile) tile_step(t + 1, std::integral_constant<int, 1>{}, std::integral_constant<int, 1>{});
    if (t + 2 <= wg_last_tile) tile_step(t + 2, std::integral_constant<int, 0>{}, std::integral_constant<int, 2>{});
    if (t + 3 <= wg_last_tile) tile_step(t + 3, std::integral_constant<int, 1>{}, std::integral_constant<int, 3>{});
  }

#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const int qp = q0 + kQCols * nb + col;
    if (wave_on && qp < L) {
      __bf16* orow = p.out + (static_cast<int64_t>(lo + qp) * p.hq + head) * D + 4 * g;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = finalize_val(A[nb][db][j], Ls[nb]);
        *reinterpret_cast<bf16x4*>(orow + 16 * db) = w;
      }
      if (p.lse != nullptr && g == 0) p.lse[static_cast<int64_t>(lo + qp) * p.hq + head] = finalize_lse(M[nb], Ls[nb], c);
    }
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillLaunch& a, hipStream_t stream) {
  PrefillParams p;
  p.q = static_cast<const __bf16*>(a.q);
  p.k = static_cast<const __bf16*>(a.k);
  p.v = static_cast<const __bf16*>(a.v);
  p.cu = a.cu_seqlens;
  p.out = static_cast<__bf16*>(a.out);
  p.lse = a.lse;
  p.hq = a.num_q_heads;
  p.hkv = a.num_kv_heads;
  p.group = a.num_q_heads / a.num_kv_heads;
  p.total = a.total_tokens;
  p.c = a.c;
  p.num_seqs = a.num_seqs;
  const int64_t ntiles = (a.max_seqlen + kWgRows - 1) / kWgRows;
  const int64_t ngroups = ntiles * a.num_seqs * a.num_kv_heads;
  const int64_t nblocks = (ngroups + kXcds - 1) / kXcds * kXcds * p.group;
  if (nblocks > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  p.ngroups = static_cast<int>(ngroups);
  const dim3 grid(static_cast<unsigned>(nblocks));
  const dim3 block(kWaves * 64);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(prefill_kernel<128>, grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL(prefill_kernel<64>, grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace uattn
