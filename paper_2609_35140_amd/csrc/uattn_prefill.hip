// Full-sequence entry point: causal GQA attention over a packed varlen batch.
//
// Workgroup = 4 waves = 128 consecutive query rows of one q head of one
// sequence; wave w owns rows q0 .. q0+31 (q0 = tile*128 + 32*w), one row per
// MFMA column.  All four waves stream the same K/V tiles through a double-
// buffered LDS stage; a wave stops at its own diagonal tile (q0 / 64), so no
// row ever sees a tile without a visible key.  Every row's arithmetic is the
// shared per-tile sequence in uattn_numerics.h, chunk-folded every 4 tiles,
// exactly as the decode path folds its positional split.
//
// Grid: x = q head, y = sequence, z = query tile counted from the END of the
// sequence (z = 0 is the last, most expensive tile), so the longest work is
// dispatched first.
#include "uattn_internal.h"
#include "uattn_numerics.h"
#include "uattn_tile_io.h"

namespace uattn {
namespace {

constexpr int kWaveRows = 32;
constexpr int kWgRows = 128;

struct PrefillParams {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const int32_t* cu;
  __bf16* out;
  float* lse;
  int hq, hkv, group, total;
  float c;
};

template <int D>
__global__ __launch_bounds__(256, 2) void prefill_kernel(PrefillParams p) {
  constexpr int NDB = D / 32;
  __shared__ __attribute__((aligned(16))) __bf16 lds[2 * Lds<D>::kStageElems];

  const int head = blockIdx.x, seq = blockIdx.y;
  // clamp the (trusted) offsets so that a malformed table cannot index outside the tensors
  const int lo = min(max(p.cu[seq], 0), p.total);
  const int L = max(min(p.cu[seq + 1], p.total) - lo, 0);
  const int nqt = (L + kWgRows - 1) / kWgRows;
  const int qt = nqt - 1 - static_cast<int>(blockIdx.z);
  if (qt < 0) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int q0 = qt * kWgRows + wave * kWaveRows;
  const bool wave_on = q0 < L;
  const int qpos = q0 + col;
  const int kvh = head / p.group;
  const int last_q0 = min(qt * kWgRows + kWgRows - kWaveRows, ((L - 1) / kWaveRows) * kWaveRows);
  const int wg_last_tile = last_q0 / kTileKeys;
  const int my_last_tile = q0 / kTileKeys;

  // this lane's Q^T operand
  bf16x8 qf[D / 16];
  if (wave_on && qpos < L) {
    const __bf16* qrow = p.q + (static_cast<int64_t>(lo + qpos) * p.hq + head) * D + 8 * h;
#pragma unroll
    for (int st = 0; st < D / 16; ++st) qf[st] = *reinterpret_cast<const bf16x8*>(qrow + 16 * st);
  } else {
#pragma unroll
    for (int st = 0; st < D / 16; ++st)
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[st][e] = static_cast<__bf16>(0.0f);
  }

  TileIO<D> io;
  const int r0 = TileIO<D>::first_row(tid);
  const int64_t row_stride = static_cast<int64_t>(p.hkv) * D;
  auto load_tile = [&](int t) {
    const int pos = t * kTileKeys + r0;
    io.load(p.k, p.v, (static_cast<int64_t>(lo + pos) * p.hkv + kvh) * D, row_stride, L - pos, tid);
  };

  f32x16 acc[NDB], A[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      acc[db][r] = 0.f;
      A[db][r] = 0.f;
    }
  float m = neg_inf(), l = 0.f, M = neg_inf(), Ls = 0.f;
  const float c = p.c;

  load_tile(0);
  for (int t = 0; t <= wg_last_tile; ++t) {
    __bf16* stage = lds + (t & 1) * Lds<D>::kStageElems;
    io.store(stage, tid);
    __syncthreads();
    if (t < wg_last_tile) load_tile(t + 1);
    if (wave_on && t <= my_last_tile) {
      f32x16 s[2];
      qk_scores<D>(stage, qf, s, lane);
      if (t == my_last_tile) mask_scores(s, t * kTileKeys, qpos, lane);
      const float alpha = softmax_tile(s, m, l, c);
      bf16x8 pb[4];
      pack_p(s, pb);
      pv_tile<D, NDB>(stage + Lds<D>::kKElems, pb, acc, alpha, 0, lane);
      if (t == my_last_tile || (t % kTilesPerChunk) == kTilesPerChunk - 1) {
        if (t < kTilesPerChunk) {
          M = m;
          Ls = l;
#pragma unroll
          for (int db = 0; db < NDB; ++db) A[db] = acc[db];
        } else {
          const FoldScale f = fold_scale(M, m, c);
          Ls = fold_val(f, Ls, l);
#pragma unroll
          for (int db = 0; db < NDB; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) A[db][r] = fold_val(f, A[db][r], acc[db][r]);
          M = f.m_new;
        }
        m = neg_inf();
        l = 0.f;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;
      }
    }
  }

  if (wave_on && qpos < L) {
    __bf16* orow = p.out + (static_cast<int64_t>(lo + qpos) * p.hq + head) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = finalize_val(A[db][4 * i + j], Ls);
        *reinterpret_cast<bf16x4*>(orow + 32 * db + 8 * i + 4 * h) = w;
      }
    if (p.lse != nullptr && h == 0) p.lse[static_cast<int64_t>(lo + qpos) * p.hq + head] = finalize_lse(M, Ls, c);
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
  const dim3 grid(a.num_q_heads, a.num_seqs, (a.max_seqlen + kWgRows - 1) / kWgRows);
  const dim3 block(256);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(prefill_kernel<128>, grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL(prefill_kernel<64>, grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace uattn
