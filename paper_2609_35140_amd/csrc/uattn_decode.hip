// Token-wise decode entry point: one query per sequence against a paged KV cache.
//
// Split kernel: workgroup = (256-key positional chunk, kv head, batch entry).
// The G query heads of the kv head sit in the MFMA columns (padded to 32), so
// each K/V tile is read from HBM once for the whole group.  The four waves
// compute the same scores and softmax state (the shared per-tile sequence of
// uattn_numerics.h) and each accumulates one 32-wide d block of the output.
// A chunk's result is either final (the context fits in one chunk) or an
// fp32 partial (m, l, acc) written to the workspace.
//
// Merge kernel: folds an entry's chunk partials left to right in chunk order
// and normalizes -- the same fold, in the same order, that the full-sequence
// kernel applies at its chunk boundaries.  Chunk boundaries depend only on
// key positions, so nothing here depends on the batch, its order, the grid or
// max_seqlen.
#include "uattn_internal.h"
#include "uattn_numerics.h"
#include "uattn_tile_io.h"

namespace uattn {
namespace {

struct DecodeParams {
  const __bf16* q;
  const __bf16* kp;
  const __bf16* vp;
  const int32_t* bt;
  const int32_t* seqlens;
  __bf16* out;
  float* lse;
  float* ws_acc;
  float* ws_ml;
  int hq, hkv, group, maxp, page_size, num_pages, max_seqlen, nchunk_max;
  float c;
};

template <int D>
__global__ __launch_bounds__(256, 2) void decode_split_kernel(DecodeParams p) {
  constexpr int NDB = D / 32;
  __shared__ __attribute__((aligned(16))) __bf16 lds[2 * Lds<D>::kStageElems];

  const int chunk = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int n = min(p.seqlens[b], p.max_seqlen);  // clamp (trusted) lengths to the sized grid
  const int nch = (n + kChunkKeys - 1) / kChunkKeys;
  if (n < 1 || chunk >= nch) return;
  const int t0 = chunk * kTilesPerChunk;
  const int last_tile = (n - 1) / kTileKeys;
  const int t1 = min(t0 + kTilesPerChunk - 1, last_tile);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int qpos = n - 1;
  const int head = kvh * p.group + col;

  bf16x8 qf[D / 16];
  if (col < p.group) {
    const __bf16* qrow = p.q + (static_cast<int64_t>(b) * p.hq + head) * D + 8 * h;
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
  const int32_t* bt_row = p.bt + static_cast<int64_t>(b) * p.maxp;
  auto row_offsets = [&](int t, int64_t (&offs)[TileIO<D>::kKPU]) {
#pragma unroll
    for (int i = 0; i < TileIO<D>::kKPU; ++i) {
      const int pos = t * kTileKeys + r0 + i;
      const int64_t page = pos < n ? bt_row[pos / p.page_size] : -1;
      offs[i] = (page >= 0 && page < p.num_pages) ? ((page * p.hkv + kvh) * p.page_size + (pos % p.page_size)) * D : -1;
    }
  };

  f32x16 acc[1];
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[0][r] = 0.f;
  float m = neg_inf(), l = 0.f;
  const float c = p.c;
  const bool pv_on = wave < NDB;

  {
    int64_t offs[TileIO<D>::kKPU];
    row_offsets(t0, offs);
    io.load(p.kp, p.vp, offs, tid);
  }
  for (int t = t0; t <= t1; ++t) {
    __bf16* stage = lds + ((t - t0) & 1) * Lds<D>::kStageElems;
    io.store(stage, tid);
    __syncthreads();
    if (t < t1) {
      int64_t offs[TileIO<D>::kKPU];
      row_offsets(t + 1, offs);
      io.load(p.kp, p.vp, offs, tid);
    }
    f32x16 s[2];
    qk_scores<D>(stage, qf, s, lane);
    if (t == last_tile) mask_scores(s, t * kTileKeys, qpos, lane);
    const float alpha = softmax_tile(s, m, l, c);
    bf16x8 pb[4];
    pack_p(s, pb);
    if (pv_on) pv_tile<D, 1>(stage + Lds<D>::kKElems, pb, acc, alpha, wave, lane);
  }

  if (!pv_on || col >= p.group) return;
  if (nch == 1) {
    __bf16* orow = p.out + (static_cast<int64_t>(b) * p.hq + head) * D + 32 * wave;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bf16x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = finalize_val(acc[0][4 * i + j], l);
      *reinterpret_cast<bf16x4*>(orow + 8 * i + 4 * h) = w;
    }
    if (p.lse != nullptr && wave == 0 && h == 0) p.lse[static_cast<int64_t>(b) * p.hq + head] = finalize_lse(m, l, c);
  } else {
    const int64_t slot = (static_cast<int64_t>(b) * p.hq + head) * p.nchunk_max + chunk;
    float* arow = p.ws_acc + slot * D + 32 * wave;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<f32x4*>(arow + 8 * i + 4 * h) =
          f32x4{acc[0][4 * i], acc[0][4 * i + 1], acc[0][4 * i + 2], acc[0][4 * i + 3]};
    if (wave == 0 && h == 0) {
      p.ws_ml[slot * 2] = m;
      p.ws_ml[slot * 2 + 1] = l;
    }
  }
}

// One workgroup of 64 threads per (q head, entry); thread t owns d = t + 64*j.
template <int D>
__global__ __launch_bounds__(64) void decode_merge_kernel(DecodeParams p) {
  constexpr int PER = D / 64;
  const int head = blockIdx.x, b = blockIdx.y;
  const int n = min(p.seqlens[b], p.max_seqlen);
  const int nch = (n + kChunkKeys - 1) / kChunkKeys;
  if (n < 1 || nch <= 1) return;
  const int tid = threadIdx.x;
  const int64_t base = (static_cast<int64_t>(b) * p.hq + head) * p.nchunk_max;
  const float* ml = p.ws_ml + base * 2;
  const float* ac = p.ws_acc + base * D;
  const float c = p.c;
  float M = ml[0], L = ml[1];
  float A[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) A[j] = ac[tid + 64 * j];
  for (int k = 1; k < nch; ++k) {
    const FoldScale f = fold_scale(M, ml[2 * k], c);
    L = fold_val(f, L, ml[2 * k + 1]);
#pragma unroll
    for (int j = 0; j < PER; ++j) A[j] = fold_val(f, A[j], ac[static_cast<int64_t>(k) * D + tid + 64 * j]);
    M = f.m_new;
  }
  __bf16* orow = p.out + (static_cast<int64_t>(b) * p.hq + head) * D;
#pragma unroll
  for (int j = 0; j < PER; ++j) orow[tid + 64 * j] = finalize_val(A[j], L);
  if (p.lse != nullptr && tid == 0) p.lse[static_cast<int64_t>(b) * p.hq + head] = finalize_lse(M, L, c);
}

}  // namespace

size_t decode_ws_acc_bytes(int64_t batch, int64_t nchunk_max, int64_t num_q_heads, int64_t head_dim) {
  return static_cast<size_t>(batch * num_q_heads * nchunk_max * head_dim) * sizeof(float);
}
size_t decode_ws_ml_bytes(int64_t batch, int64_t nchunk_max, int64_t num_q_heads) {
  return static_cast<size_t>(batch * num_q_heads * nchunk_max * 2) * sizeof(float);
}

hipError_t launch_decode(const DecodeLaunch& a, hipStream_t stream) {
  DecodeParams p;
  p.q = static_cast<const __bf16*>(a.q);
  p.kp = static_cast<const __bf16*>(a.k_pages);
  p.vp = static_cast<const __bf16*>(a.v_pages);
  p.bt = a.block_table;
  p.seqlens = a.seqlens;
  p.out = static_cast<__bf16*>(a.out);
  p.lse = a.lse;
  p.ws_acc = a.ws_acc;
  p.ws_ml = a.ws_ml;
  p.hq = a.num_q_heads;
  p.hkv = a.num_kv_heads;
  p.group = a.num_q_heads / a.num_kv_heads;
  p.maxp = a.max_pages_per_seq;
  p.page_size = a.page_size;
  p.num_pages = a.num_pages;
  p.max_seqlen = a.max_seqlen;
  p.nchunk_max = a.nchunk_max;
  p.c = a.c;
  const dim3 grid(a.nchunk_max, a.num_kv_heads, a.batch);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(decode_split_kernel<128>, grid, dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL(decode_split_kernel<64>, grid, dim3(256), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nchunk_max <= 1) return e;
  const dim3 mgrid(a.num_q_heads, a.batch);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(decode_merge_kernel<128>, mgrid, dim3(64), 0, stream, p);
  else
    hipLaunchKernelGGL(decode_merge_kernel<64>, mgrid, dim3(64), 0, stream, p);
  return hipGetLastError();
}

}  // namespace uattn
