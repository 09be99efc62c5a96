// Token-wise decode entry point: one query per sequence against a paged KV cache.
//
// Work item = (256-key positional chunk, kv head, batch entry).  The G query
// heads of the kv head sit in the MFMA columns (16 per block), so each K/V
// tile is read from HBM once for the whole group.  The four waves of a
// workgroup compute the same scores and softmax state (the shared per-tile
// sequence of uattn_numerics.h) and each accumulates a quarter of the
// output's d range.  An item's result is either final (the context fits in
// one chunk) or an fp32 partial (m, l, acc) written to the workspace.
//
// The grid is persistent: a fixed number of workgroups (two per CU) walk the
// items in chunk-major order, stride = grid size.  Per item, the entry's
// length, the page-table entries of the chunk and the queries are fetched in
// one round trip (the page lookups are speculative and clamped to the table,
// so they need not wait for the length); the next item's fetch is issued
// during the current item's first tile, and its first tile is loaded
// (direct-to-LDS, two stages) while the current item's last tile is computed.
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
  int batch, hq, hkv, group, maxp, page_size, num_pages, max_seqlen, nchunk_max;
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
// finished the entry's last outstanding chunk.  Loads are issued 8 chunks at
// a time so that each batch costs one memory round trip.
template <int D>
__device__ __forceinline__ void merge_entry(const DecodeParams& p, int b, int kvh, int nch, int tid) {
  constexpr int kBatch = 8;
  const int nvals = p.group * D;
  for (int v = tid; v < nvals; v += 256) {
    const int g = v / D, d = v % D;
    const int head = kvh * p.group + g;
    const int64_t base = (static_cast<int64_t>(b) * p.hq + head) * p.nchunk_max;
    const float* ml = p.ws_ml + base * 2;
    const float* ac = p.ws_acc + base * D + d;
    float M = 0.f, L = 0.f, A = 0.f;
    for (int k0 = 0; k0 < nch; k0 += kBatch) {
      float bm[kBatch], bl[kBatch], ba[kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int k = min(k0 + i, nch - 1);
        bm[i] = ld_coherent(ml + 2 * k);
        bl[i] = ld_coherent(ml + 2 * k + 1);
        ba[i] = ld_coherent(ac + static_cast<int64_t>(k) * D);
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int k = k0 + i;
        if (k >= nch) break;
        if (k == 0) {
          M = bm[i];
          L = bl[i];
          A = ba[i];
        } else {
          const FoldScale f = fold_scale(M, bm[i], p.c);
          L = fold_val(f, L, bl[i]);
          A = fold_val(f, A, ba[i]);
          M = f.m_new;
        }
      }
    }
    p.out[(static_cast<int64_t>(b) * p.hq + head) * D + d] = finalize_val(A, L);
    if (p.lse != nullptr && d == 0) p.lse[static_cast<int64_t>(b) * p.hq + head] = finalize_lse(M, L, p.c);
  }
}

// One work item's coordinates and the memory its tiles come from.
struct Item {
  int b, kvh, chunk, n, nch, ntiles;
  bool valid;
  int64_t off[kTilesPerChunk];   // element offset of this wave's first row of each tile
  int nvalid[kTilesPerChunk];    // rows of this wave's run that hold keys
};

// Issue the loads that describe candidate item `cand` (chunk-major order):
// the entry's length, the page of this wave's rows of each tile of the chunk
// (speculative, index clamped to the table) and this lane's query operands.
// Everything is resolved later by resolve_item, so the loads overlap.
template <int D, int NB>
__device__ __forceinline__ void fetch_item(const DecodeParams& p, int cand, int ncand, Item& it, int (&raw_page)[kTilesPerChunk],
                                           int& raw_n, bf16x8 (&qf)[NB][D / 32], int wave, int lane) {
  const int per_chunk = p.batch * p.hkv;
  it.valid = cand < ncand;
  const int c = it.valid ? cand : 0;
  it.chunk = c / per_chunk;
  it.b = (c % per_chunk) / p.hkv;
  it.kvh = c % p.hkv;
  raw_n = p.seqlens[it.b];
  const int32_t* bt_row = p.bt + static_cast<int64_t>(it.b) * p.maxp;
#pragma unroll
  for (int j = 0; j < kTilesPerChunk; ++j) {
    const int pos = (it.chunk * kTilesPerChunk + j) * kTileKeys + 16 * wave;
    raw_page[j] = bt_row[min(pos / p.page_size, p.maxp - 1)];
  }
  const int g = lane >> 4, col = lane & 15;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int gi = kQCols * nb + col;
    if (gi < p.group) {
      const __bf16* qrow = p.q + (static_cast<int64_t>(it.b) * p.hq + it.kvh * p.group + gi) * D + 8 * g;
#pragma unroll
      for (int st = 0; st < D / 32; ++st) qf[nb][st] = *reinterpret_cast<const bf16x8*>(qrow + 32 * st);
    } else {
#pragma unroll
      for (int st = 0; st < D / 32; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[nb][st][e] = static_cast<__bf16>(0.0f);
    }
  }
}

template <int D>
__device__ __forceinline__ void resolve_item(const DecodeParams& p, Item& it, const int (&raw_page)[kTilesPerChunk],
                                             int raw_n, int wave) {
  it.n = min(raw_n, p.max_seqlen);  // clamp (trusted) lengths to the sized workspace
  it.nch = (it.n + kChunkKeys - 1) / kChunkKeys;
  it.valid = it.valid && it.n >= 1 && it.chunk < it.nch;
  const int t0 = it.chunk * kTilesPerChunk;
  it.ntiles = it.valid ? min(kTilesPerChunk, (it.n - 1) / kTileKeys - t0 + 1) : 0;
#pragma unroll
  for (int j = 0; j < kTilesPerChunk; ++j) {
    const int pos = (t0 + j) * kTileKeys + 16 * wave;
    const int64_t page = raw_page[j];
    const bool ok = j < it.ntiles && pos < it.n && page >= 0 && page < p.num_pages;
    it.off[j] = ok ? ((page * p.hkv + it.kvh) * p.page_size + (pos % p.page_size)) * D : 0;
    it.nvalid[j] = ok ? it.n - pos : 0;
  }
}

template <int D, int NB>
__global__ __launch_bounds__(256, 2) void decode_kernel(DecodeParams p) {
  using TL = TileLayout<D>;
  using Loads = TileLoads<D, 16>;
  __shared__ __attribute__((aligned(1024))) __bf16 lds[2 * TL::kStageElems];
  __shared__ int s_last;
  constexpr int NDBW = D / 16 / 4;  // 16-wide d blocks of the output per wave

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, col = lane & 15;
  const int ncand = p.batch * p.hkv * p.nchunk_max;
  const int stride = gridDim.x;
  const float c = p.c;

  Item cur, nxt;
  int raw_page[kTilesPerChunk], raw_n;
  bf16x8 qf[NB][D / 32], qf_next[NB][D / 32];

  // first valid item of this workgroup
  int cand = blockIdx.x;
  fetch_item<D, NB>(p, cand, ncand, cur, raw_page, raw_n, qf, wave, lane);
  resolve_item<D>(p, cur, raw_page, raw_n, wave);
  while (!cur.valid && cand + stride < ncand) {
    cand += stride;
    fetch_item<D, NB>(p, cand, ncand, cur, raw_page, raw_n, qf, wave, lane);
    resolve_item<D>(p, cur, raw_page, raw_n, wave);
  }
  if (!cur.valid) return;

  int slot = 0;  // LDS stage of the next tile to compute
  auto issue = [&](const Item& it, int j, int stage) {
    load_tile_rows<D, 16>(lds + stage * TL::kStageElems, p.kp + it.off[j], p.vp + it.off[j], D, it.nvalid[j], wave,
                          lane);
  };
  issue(cur, 0, 0);

  while (true) {
    const int ncand_next = cand + stride;

    f32x4 acc[NB][NDBW], lsum[NB];
    float m[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int db = 0; db < NDBW; ++db) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
      m[nb] = neg_inf();
      lsum[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int qpos = cur.n - 1;
    const int last_tile = (cur.n - 1) / kTileKeys;

#pragma unroll
    for (int j = 0; j < kTilesPerChunk; ++j) {
      if (j < cur.ntiles) {
        __bf16* stage = lds + (slot & 1) * TL::kStageElems;
        // nothing is issued after this tile's loads until this point
        wait_tiles_pending<Loads::kPerTile>(0);
        __syncthreads();
        // Describe the next candidate now, before the next tile's loads: the
        // full drain at the next tile then also covers these loads, which by
        // issue order complete first, so they add no wait of their own.
        if (j == 0) fetch_item<D, NB>(p, ncand_next, ncand, nxt, raw_page, raw_n, qf_next, wave, lane);
        if (j + 1 < cur.ntiles) {
          issue(cur, j + 1, (slot + 1) & 1);
        } else {
          resolve_item<D>(p, nxt, raw_page, raw_n, wave);
          if (nxt.valid) issue(nxt, 0, (slot + 1) & 1);
        }
        const int t = cur.chunk * kTilesPerChunk + j;
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
        ++slot;
      }
    }

    if (cur.nch == 1) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int gi = kQCols * nb + col;
        if (gi >= p.group) continue;
        const int64_t orow = (static_cast<int64_t>(cur.b) * p.hq + cur.kvh * p.group + gi);
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
    } else {
      // chunk partial -> workspace
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int gi = kQCols * nb + col;
        if (gi >= p.group) continue;
        const int64_t ws_slot =
            (static_cast<int64_t>(cur.b) * p.hq + cur.kvh * p.group + gi) * p.nchunk_max + cur.chunk;
        float* arow = p.ws_acc + ws_slot * D + 16 * wave * NDBW + 4 * g;
#pragma unroll
        for (int db = 0; db < NDBW; ++db)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) st_coherent(arow + 16 * db + jj, acc[nb][db][jj]);
        if (wave == 0 && g == 0) {
          st_coherent(p.ws_ml + ws_slot * 2, m[nb]);
          st_coherent(p.ws_ml + ws_slot * 2 + 1, lsum[nb][0]);
        }
      }
      // The workgroup that completes the entry's last outstanding chunk folds
      // them all.  Which workgroup that is does not affect the arithmetic: the
      // fold order is the chunk order.
      wait_vmem_below<0>();  // this thread's partial stores have completed
      __syncthreads();
      if (tid == 0) {
        const int prev = __hip_atomic_fetch_add(p.ws_cnt + static_cast<int64_t>(cur.b) * p.hkv + cur.kvh, 1,
                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = (prev == cur.nch - 1);
      }
      __syncthreads();
      if (s_last) {
        merge_entry<D>(p, cur.b, cur.kvh, cur.nch, tid);
        if (tid == 0)
          __hip_atomic_store(p.ws_cnt + static_cast<int64_t>(cur.b) * p.hkv + cur.kvh, 0, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      }
    }

    // advance; if the prefetched candidate is empty, look further (no prefetch)
    cand = ncand_next;
    if (!nxt.valid) {
      while (!nxt.valid && cand + stride < ncand) {
        cand += stride;
        fetch_item<D, NB>(p, cand, ncand, nxt, raw_page, raw_n, qf_next, wave, lane);
        resolve_item<D>(p, nxt, raw_page, raw_n, wave);
      }
      if (!nxt.valid) break;
      __syncthreads();  // every wave is done with the stage the new first tile goes to
      issue(nxt, 0, slot & 1);
    }
    cur = nxt;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int st = 0; st < D / 32; ++st) qf[nb][st] = qf_next[nb][st];
  }
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
  p.batch = a.batch;
  const int64_t ncand = static_cast<int64_t>(a.batch) * a.num_kv_heads * a.nchunk_max;
  if (ncand > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  const int64_t slots = 2 * static_cast<int64_t>(a.num_cus);
  const dim3 grid(static_cast<unsigned>(ncand < slots ? ncand : slots));
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
