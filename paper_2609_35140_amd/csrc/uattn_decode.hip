// Token-wise decode entry point: one query per sequence against a paged KV cache.
//
// One kernel: workgroup = (256-key positional chunk, kv head, batch entry).
// The G query heads of the kv head sit in the MFMA columns (16 per block), so
// each K/V tile is read from HBM once for the whole group.  The four waves
// compute the same scores and softmax state (the shared per-tile sequence of
// uattn_numerics.h) and each accumulates one 32-wide d block of the output.
// A chunk's result is either final (the context fits in one chunk) or an
// fp32 partial (m, l, acc) written to the workspace.  The page-table entries of
// the chunk are fetched up front; tiles move by direct-to-LDS loads into two
// stages, the next tile loading while the current one is computed.
//
// Merge: the workgroup that completes an entry's last outstanding chunk
// (an arrival counter per (entry, kv head), reset to zero after use) folds
// the entry's chunk partials left to right in chunk order and normalizes --
// the same fold, in the same order, that the full-sequence kernel applies at
// its chunk boundaries.  Chunk boundaries depend only on key positions, so
// nothing here depends on the batch, its order, the grid, max_seqlen or which
// workgroup merges.
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
  float* ws_acc;     // [batch][Hq][nchunk_max][D]
  float* ws_ml;      // [batch][Hq][nchunk_max][2]
  int32_t* ws_cnt;   // [batch][Hkv] arrival counters, zero between calls
  int hq, hkv, group, maxp, page_size, num_pages, max_seqlen, nchunk_max;
  float c;
};

// Partials cross workgroups (and XCDs, whose L2 caches are not coherent with
// each other for ordinary stores).  They are written and read with
// agent-scope relaxed atomic accesses, which go through to the device-
// coherent level, instead of full-cache release/acquire fences (an L2
// writeback and invalidate per workgroup).  Ordering: every writer waits
// for its stores to complete before the workgroup barrier, one thread then
// bumps the arrival counter; the merger reads the partials only after its
// counter increment has returned the final count.
__device__ __forceinline__ void st_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coherent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Fold the chunk partials of entry b, kv head kvh (all its q heads) in chunk
// order and write the normalized outputs.  Called by the workgroup that
// finished the entry's last outstanding chunk.
template <int D>
__device__ __forceinline__ void merge_entry(const DecodeParams& p, int b, int kvh, int nch, int tid) {
  const int nvals = p.group * D;
  for (int v = tid; v < nvals; v += 256) {
    const int g = v / D, d = v % D;
    const int head = kvh * p.group + g;
    const int64_t base = (static_cast<int64_t>(b) * p.hq + head) * p.nchunk_max;
    const float* ml = p.ws_ml + base * 2;
    const float* ac = p.ws_acc + base * D + d;
    float M = ld_coherent(ml), L = ld_coherent(ml + 1), A = ld_coherent(ac);
#pragma unroll 4
    for (int k = 1; k < nch; ++k) {
      const FoldScale f = fold_scale(M, ld_coherent(ml + 2 * k), p.c);
      L = fold_val(f, L, ld_coherent(ml + 2 * k + 1));
      A = fold_val(f, A, ld_coherent(ac + static_cast<int64_t>(k) * D));
      M = f.m_new;
    }
    p.out[(static_cast<int64_t>(b) * p.hq + head) * D + d] = finalize_val(A, L);
    if (p.lse != nullptr && d == 0) p.lse[static_cast<int64_t>(b) * p.hq + head] = finalize_lse(M, L, p.c);
  }
}

template <int D, int NB>
__global__ __launch_bounds__(256, 2) void decode_kernel(DecodeParams p) {
  using TL = TileLayout<D>;
  __shared__ __attribute__((aligned(1024))) __bf16 lds[2 * TL::kStageElems];
  __shared__ int s_last;
  constexpr int NDBW = D / 16 / 4;  // 16-wide d blocks of the output per wave

  const int chunk = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int n = min(p.seqlens[b], p.max_seqlen);  // clamp (trusted) lengths to the sized grid
  const int nch = (n + kChunkKeys - 1) / kChunkKeys;
  if (n < 1 || chunk >= nch) return;
  const int t0 = chunk * kTilesPerChunk;
  const int last_tile = (n - 1) / kTileKeys;
  const int ntiles = min(kTilesPerChunk, last_tile - t0 + 1);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, col = lane & 15;
  const int qpos = n - 1;

  // Where this wave's 16 rows of each tile of the chunk live (one page: pages
  // hold >= 16 keys).  Looked up once, up front.
  const int32_t* bt_row = p.bt + static_cast<int64_t>(b) * p.maxp;
  int64_t off0[kTilesPerChunk];
  int nvalid[kTilesPerChunk];
#pragma unroll
  for (int j = 0; j < kTilesPerChunk; ++j) {
    const int pos = (t0 + j) * kTileKeys + 16 * wave;
    const int64_t page = (j < ntiles && pos < n) ? bt_row[pos / p.page_size] : -1;
    const bool ok = page >= 0 && page < p.num_pages;
    off0[j] = ok ? ((page * p.hkv + kvh) * p.page_size + (pos % p.page_size)) * D : 0;
    nvalid[j] = ok ? n - pos : 0;
  }

  // Q^T operands: the group's q heads in the MFMA columns (16 per block)
  bf16x8 qf[NB][D / 32];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int gi = kQCols * nb + col;
    if (gi < p.group) {
      const __bf16* qrow = p.q + (static_cast<int64_t>(b) * p.hq + kvh * p.group + gi) * D + 8 * g;
#pragma unroll
      for (int st = 0; st < D / 32; ++st) qf[nb][st] = *reinterpret_cast<const bf16x8*>(qrow + 32 * st);
    } else {
#pragma unroll
      for (int st = 0; st < D / 32; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[nb][st][e] = static_cast<__bf16>(0.0f);
    }
  }

  // two LDS stages: tile j+1 loads while tile j is computed
  auto issue_tile = [&](int j) {
    load_tile_rows<D, 16>(lds + (j & 1) * TL::kStageElems, p.kp + off0[j], p.vp + off0[j], D, nvalid[j], wave, lane);
  };
  issue_tile(0);

  f32x4 acc[NB][NDBW], lsum[NB];
  float m[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int db = 0; db < NDBW; ++db) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    m[nb] = neg_inf();
    lsum[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float c = p.c;

#pragma unroll
  for (int j = 0; j < kTilesPerChunk; ++j) {
    if (j < ntiles) {
      __bf16* stage = lds + (j & 1) * TL::kStageElems;
      wait_tile_loads();
      __syncthreads();
      if (j + 1 < ntiles) issue_tile(j + 1);
      const int t = t0 + j;
      f32x4 s[NB][4];
      qk_scores<D, NB>(stage, qf, s, lane);
      float alpha[NB];
      bf16x8 pb[NB][2];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        if (t == last_tile) mask_scores(s[nb], t * kTileKeys, qpos, lane);
        alpha[nb] = softmax_tile(s[nb], m[nb], c);
        pack_p(s[nb], pb[nb]);
      }
      pv_tile<D, NB, NDBW>(stage, pb, acc, lsum, alpha, wave * NDBW, lane);
    }
  }

  if (nch == 1) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int gi = kQCols * nb + col;
      if (gi >= p.group) continue;
      const int64_t orow = (static_cast<int64_t>(b) * p.hq + kvh * p.group + gi);
      __bf16* o = p.out + orow * D + 16 * wave * NDBW + 4 * g;
#pragma unroll
      for (int db = 0; db < NDBW; ++db) {
        bf16x4 w;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) w[jj] = finalize_val(acc[nb][db][jj], lsum[nb][0]);
        *reinterpret_cast<bf16x4*>(o + 16 * db) = w;
      }
      if (p.lse != nullptr && wave == 0 && g == 0) p.lse[orow] = finalize_lse(m[nb], lsum[nb][0], c);
    }
    return;
  }

  // chunk partial -> workspace
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int gi = kQCols * nb + col;
    if (gi >= p.group) continue;
    const int64_t slot = (static_cast<int64_t>(b) * p.hq + kvh * p.group + gi) * p.nchunk_max + chunk;
    float* arow = p.ws_acc + slot * D + 16 * wave * NDBW + 4 * g;
#pragma unroll
    for (int db = 0; db < NDBW; ++db)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) st_coherent(arow + 16 * db + jj, acc[nb][db][jj]);
    if (wave == 0 && g == 0) {
      st_coherent(p.ws_ml + slot * 2, m[nb]);
      st_coherent(p.ws_ml + slot * 2 + 1, lsum[nb][0]);
    }
  }
  // The workgroup that completes the entry's last outstanding chunk folds
  // them all.  Which workgroup that is does not affect the arithmetic: the
  // fold order is the chunk order.
  __builtin_amdgcn_s_waitcnt(0);  // this thread's partial stores have completed
  __syncthreads();
  if (tid == 0) {
    const int prev = __hip_atomic_fetch_add(p.ws_cnt + static_cast<int64_t>(b) * p.hkv + kvh, 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev == nch - 1);
  }
  __syncthreads();
  if (!s_last) return;
  merge_entry<D>(p, b, kvh, nch, tid);
  if (tid == 0)
    __hip_atomic_store(p.ws_cnt + static_cast<int64_t>(b) * p.hkv + kvh, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

size_t decode_ws_acc_bytes(int64_t batch, int64_t nchunk_max, int64_t num_q_heads, int64_t head_dim) {
  return (static_cast<size_t>(batch * num_q_heads * nchunk_max * head_dim) * sizeof(float) + 255) / 256 * 256;
}
size_t decode_ws_ml_bytes(int64_t batch, int64_t nchunk_max, int64_t num_q_heads) {
  return (static_cast<size_t>(batch * num_q_heads * nchunk_max * 2) * sizeof(float) + 255) / 256 * 256;
}
// Counters are sized by the q-head count (an upper bound of the kv-head count)
// so that the size depends only on the arguments of uattn_decode_workspace_bytes.
size_t decode_ws_cnt_bytes(int64_t batch, int64_t num_q_heads) {
  return (static_cast<size_t>(batch * num_q_heads) * sizeof(int32_t) + 255) / 256 * 256;
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
  p.ws_cnt = a.ws_cnt;
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
  const bool two = p.group > kQCols;
  if (a.head_dim == 128) {
    if (two)
      hipLaunchKernelGGL((decode_kernel<128, 2>), grid, dim3(256), 0, stream, p);
    else
      hipLaunchKernelGGL((decode_kernel<128, 1>), grid, dim3(256), 0, stream, p);
  } else {
    if (two)
      hipLaunchKernelGGL((decode_kernel<64, 2>), grid, dim3(256), 0, stream, p);
    else
      hipLaunchKernelGGL((decode_kernel<64, 1>), grid, dim3(256), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace uattn
