// Token-wise decode entry point: one query per sequence against a paged KV cache.
//
// Work item = (256-key positional chunk, kv head, batch entry).  The G query
// heads of the kv head sit in the MFMA columns (16 per block), so each K/V
// tile is read from HBM once for the whole group.  Per 64-key tile, wave w of
// the workgroup computes the scores of key block w (keys 16w .. 16w+15); the
// block maxima are exchanged through LDS to form the tile maximum (max is
// exact, so this equals the full-tile reduction of the shared per-tile
// sequence in uattn_numerics.h), each wave turns its block into bf16 weights,
// the weights are exchanged through LDS into the PV operand order, and each
// wave accumulates a quarter of the output's d range.  Every element sees
// the same operations as in the full-sequence kernel.  An item's result is
// either final (the context fits in one chunk) or an fp32 partial (m, l, acc)
// written to the workspace.
//
// The grid is persistent: as many workgroups as the CUs hold at once walk
// the items in chunk-major order, stride = grid size.  Each workgroup keeps
// one load stream: the tiles of its items in order (direct-to-LDS, a ring of
// stages), with the descriptor of the item two ahead (the entry length and,
// speculatively, the page of each tile row) and its query operands loaded
// into LDS in the same stream; tiles of the next items are loaded while the
// current item is still computed.
//
// Merge: finished partials are queued per workgroup and their arrivals are
// counted when the queue is full and after the workgroup's last item (one
// drain for many items).  The workgroup that counts an entry's last
// outstanding chunk (an arrival counter per (entry, kv head), reset to zero
// after use) folds the entry's chunk partials left to right in chunk order
// and normalizes -- the same fold, in the same order, that the full-sequence
// kernel applies at its chunk boundaries.  Chunk boundaries depend only on
// key positions, so nothing here depends on the batch, its order, the grid,
// max_seqlen or which workgroup merges.
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
// counted the entry's last outstanding chunk.  Each thread folds two output
// values and issues the loads of 16 chunks of both before folding, so a
// context of up to 4096 keys costs one memory round trip.
template <int D>
__device__ __forceinline__ void merge_entry(const DecodeParams& p, int b, int kvh, int nch, int tid) {
  constexpr int kBatch = 16;
  const int nvals = p.group * D;
  for (int v0 = tid; v0 < nvals; v0 += 512) {
    const int vv[2] = {v0, min(v0 + 256, nvals - 1)};
    const float* ml[2];
    const float* ac[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int head = kvh * p.group + vv[u] / D;
      const int64_t base = (static_cast<int64_t>(b) * p.hq + head) * p.nchunk_max;
      ml[u] = p.ws_ml + base * 2;
      ac[u] = p.ws_acc + base * D + vv[u] % D;
    }
    float M[2] = {0.f, 0.f}, L[2] = {0.f, 0.f}, A[2] = {0.f, 0.f};
    for (int k0 = 0; k0 < nch; k0 += kBatch) {
      float bm[2][kBatch], bl[2][kBatch], ba[2][kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int k = min(k0 + i, nch - 1);
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          bm[u][i] = ld_coherent(ml[u] + 2 * k);
          bl[u][i] = ld_coherent(ml[u] + 2 * k + 1);
          ba[u][i] = ld_coherent(ac[u] + static_cast<int64_t>(k) * D);
        }
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int k = k0 + i;
        if (k >= nch) break;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          if (k == 0) {
            M[u] = bm[u][i];
            L[u] = bl[u][i];
            A[u] = ba[u][i];
          } else {
            const FoldScale f = fold_scale(M[u], bm[u][i], p.c);
            L[u] = fold_val(f, L[u], bl[u][i]);
            A[u] = fold_val(f, A[u], ba[u][i]);
            M[u] = f.m_new;
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (u == 1 && v0 + 256 >= nvals) break;
      const int head = kvh * p.group + vv[u] / D, d = vv[u] % D;
      p.out[(static_cast<int64_t>(b) * p.hq + head) * D + d] = finalize_val(A[u], L[u]);
      if (p.lse != nullptr && d == 0) p.lse[static_cast<int64_t>(b) * p.hq + head] = finalize_lse(M[u], L[u], p.c);
    }
  }
}

// One work item of the prefetch ring: its coordinates, its descriptor once
// resolved, and its progress through the load stream.  All fields are
// workgroup-uniform (scalar registers); the pages of the chunk stay in the
// item's LDS descriptor slot.
struct Ring {
  int b, kvh, chunk;
  int n, nch, ntiles;          // resolved: entry length, its chunk count, tiles of this chunk
  int slot;                    // LDS slot of its descriptor and query operands
  int ftile;                   // tiles issued before its descriptor loads
  int nissued;                 // tiles of the item whose loads were issued
  bool valid, fetched, resolved;
};

constexpr int64_t kLdsBytesPerCu = 160 * 1024;
constexpr int kLenScanMax = 4096;  // batches up to this size skip chunks past their longest entry

template <int D, int NB>
struct DecodeSmem {
  using TL = TileLayout<D>;
  static constexpr int kStages = D == 128 ? 2 : 4;  // K/V tile ring (two workgroups share a CU's LDS)
  static constexpr int kSlots = 3;      // items described at once: the one computed and two ahead
  static constexpr int kQInstr = NB * D / 32;  // 1 KB query-operand pieces per item
  static constexpr int kMaxPend = 32;   // finished partials awaiting their arrival count
  __bf16 stage[kStages][TL::kStageElems];
  __bf16 q[kSlots][kQInstr * 64 * 8];
  int32_t desc[kSlots][4][8];           // per wave: [0] entry length, [1 + j] page of this wave's rows of tile j
  float xmax[NB][4][kQCols];            // per key block: column maxima of the tile's scores
  bf16x4 pbuf[NB][4][64];               // per key block: the bf16 weights, in the lanes' PV operand order
  int32_t pend[kMaxPend][2];            // (b * Hkv + kv head, chunk count)
  int32_t flag[kMaxPend];
  int32_t lenmax[4];                    // per wave: the longest entry it read
};

// Issue the descriptor and query loads of candidate `cand` (chunk-major
// order) into LDS slot `slot`: each wave loads its own descriptor (the entry
// length and, speculatively with the table index clamped, the page of each
// of its tile rows); the query-operand pieces are split over the waves.
// Nothing waits here.
template <int D, int NB>
__device__ __forceinline__ void fetch_item(const DecodeParams& p, DecodeSmem<D, NB>& sm, Ring& r, int cand,
                                           int ncand, int slot, int issued, int wave, int lane) {
  using SM = DecodeSmem<D, NB>;
  const int per_chunk = p.batch * p.hkv;
  r.valid = cand < ncand;
  const int c = r.valid ? cand : 0;
  r.chunk = c / per_chunk;
  r.b = (c % per_chunk) / p.hkv;
  r.kvh = c % p.hkv;
  r.ntiles = 0;
  r.slot = slot;
  r.ftile = issued;
  r.nissued = 0;
  r.fetched = true;
  r.resolved = !r.valid;
  if (!r.valid) return;
  const int32_t* src = p.seqlens + r.b;
  if (lane >= 1 && lane <= kTilesPerChunk) {
    const int pos = (r.chunk * kTilesPerChunk + lane - 1) * kTileKeys + 16 * wave;
    src = p.bt + static_cast<int64_t>(r.b) * p.maxp + min(pos / p.page_size, p.maxp - 1);
  }
  const uint32_t dbase = __builtin_amdgcn_readfirstlane(lds_addr(&sm.desc[slot][wave][0]));
  if (lane < 8) dma_b32(src, dbase);  // lanes 0-7 only: 32 bytes of LDS per wave
  const int g = lane >> 4, col = lane & 15;
  const __bf16* zero = reinterpret_cast<const __bf16*>(g_zero_rows) + 8 * col;
#pragma unroll 1
  for (int i = wave; i < SM::kQInstr; i += 4) {
    const int nb = i / (D / 32), st = i % (D / 32);
    const int gi = kQCols * nb + col;
    const __bf16* q = gi < p.group
                          ? p.q + (static_cast<int64_t>(r.b) * p.hq + r.kvh * p.group + gi) * D + 8 * g + 32 * st
                          : zero;
    dma_b128(q, __builtin_amdgcn_readfirstlane(lds_addr(&sm.q[slot][i * 64 * 8])));
  }
}

// Read a fetched descriptor (its loads have landed).
template <int D, int NB>
__device__ __forceinline__ void resolve_item(const DecodeParams& p, const DecodeSmem<D, NB>& sm, Ring& r, int wave) {
  r.resolved = true;
  if (!r.valid) return;
  const int32_t* d = &sm.desc[r.slot][wave][0];
  r.n = __builtin_amdgcn_readfirstlane(min(d[0], p.max_seqlen));  // clamp (trusted) lengths to the sized workspace
  r.nch = (r.n + kChunkKeys - 1) / kChunkKeys;
  r.valid = r.n >= 1 && r.chunk < r.nch;
  r.ntiles = r.valid ? min(kTilesPerChunk, (r.n - 1) / kTileKeys - r.chunk * kTilesPerChunk + 1) : 0;
}

// Scores of one 16-key block: s[nb] = K_kb Q_nb^T, the same MFMA sequence
// (d in ascending 32-wide steps from zero) as the full-tile product.
template <int D, int NB>
__device__ __forceinline__ void qk_block(const __bf16* stage, const bf16x8 (&qf)[NB][D / 32], f32x4 (&s)[NB], int kb,
                                         int lane) {
  using TL = TileLayout<D>;
  const int g = lane >> 4, row = lane & 15;
  const int swz = TL::k_swz(row);  // equals k_swz(16*kb + row) for every kb
  const __bf16* krow = stage + (16 * kb + row) * D;
  bf16x8 a[D / 32];
#pragma unroll
  for (int st = 0; st < D / 32; ++st) a[st] = *reinterpret_cast<const bf16x8*>(krow + 8 * ((4 * st + g) ^ swz));
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < D / 32; ++st) acc = mfma16(a[st], qf[nb][st], acc);
    s[nb] = acc;
  }
}

// -inf for keys after the query (block_base = position of the block's key 0).
__device__ __forceinline__ void mask_block(f32x4& s, int block_base, int qpos, int lane) {
  const int g = lane >> 4;
#pragma unroll
  for (int j = 0; j < 4; ++j) s[j] = (block_base + 4 * g + j > qpos) ? neg_inf() : s[j];
}

// The online-softmax step for one block given the tile maximum: the same
// operations, element for element, as the full-tile step.
__device__ __forceinline__ float softmax_block(f32x4& s, float& m, float tmax, float c) {
  const float m_new = vmax(m, tmax);
  const float mc_old = m * c;
  const float mc_new = m_new * c;
  const float alpha = hw_exp2(mc_old - mc_new);
#pragma unroll
  for (int j = 0; j < 4; ++j) s[j] = hw_exp2(__builtin_fmaf(s[j], c, -mc_new));
  m = m_new;
  return alpha;
}

// The load stream of a workgroup: the tiles of its items, in item order,
// into the LDS tile ring (two stages for d = 128, four for d = 64), with the
// descriptor and query loads of the item two ahead interleaved in the same
// stream.  Loads of one wave complete in issue order, so "tile k has landed"
// also means "everything this wave issued before tile k has landed"; that is
// the only fact the waits rely on.
template <int D, int NB>
__global__ __launch_bounds__(256, 2) void decode_kernel(DecodeParams p) {
  using TL = TileLayout<D>;
  using SM = DecodeSmem<D, NB>;
  using Loads = TileLoads<D, 16>;
  constexpr int kStages = SM::kStages;
  __shared__ __attribute__((aligned(1024))) SM sm;
  constexpr int NDBW = D / 16 / 4;  // 16-wide d blocks of the output per wave

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, col = lane & 15;
  const int ncand_all = p.batch * p.hkv * p.nchunk_max;
  const int stride = gridDim.x;
  const float c = p.c;

  // Chunks past the longest entry hold no work.  When this workgroup's walk
  // is longer than the three items described at start, read the batch's
  // lengths (the loads overlap the first descriptor fetches) and stop the
  // walk after the last chunk any entry has, so that a max_seqlen far above
  // the actual lengths costs no descriptor round trips for empty items.
  int lmax = 0;
  const bool scan = p.nchunk_max > 1 && p.batch <= kLenScanMax && ncand_all > 3 * stride;
  if (scan) {
#pragma unroll 4
    for (int i = tid; i < p.batch; i += 256) lmax = max(lmax, p.seqlens[i]);
  }

  int issued = 0;    // tiles whose loads were issued
  int computed = 0;  // tiles computed
  int wdone = -1;    // latest tile waited for
  int npend = 0;     // partials in sm.pend
  int seq = 0;       // item sequence number of r0: candidate blockIdx.x + seq * stride
  Ring r0, r1, r2;

  fetch_item<D, NB>(p, sm, r0, blockIdx.x, ncand_all, 0, issued, wave, lane);
  fetch_item<D, NB>(p, sm, r1, blockIdx.x + stride, ncand_all, 1, issued, wave, lane);
  fetch_item<D, NB>(p, sm, r2, blockIdx.x + 2 * stride, ncand_all, 2, issued, wave, lane);
  wait_vmem_asm<0>();
  int ncand = ncand_all;
  if (scan) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) lmax = max(lmax, __shfl_xor(lmax, m));
    if (lane == 0) sm.lenmax[wave] = lmax;
    lds_barrier();
    lmax = max(max(sm.lenmax[0], sm.lenmax[1]), max(sm.lenmax[2], sm.lenmax[3]));
    const int nch = min(max((min(lmax, p.max_seqlen) + kChunkKeys - 1) / kChunkKeys, 1), p.nchunk_max);
    ncand = __builtin_amdgcn_readfirstlane(p.batch * p.hkv * nch);
  }
  resolve_item<D, NB>(p, sm, r0, wave);
  resolve_item<D, NB>(p, sm, r1, wave);
  resolve_item<D, NB>(p, sm, r2, wave);
  bool fetch_pending = false;  // r2 still to be fetched, into the slot r0 had (after a barrier)

  // Issue tile loads up to tile cmp + kStages - 1.  Callers are past a
  // barrier that follows the computation of tile cmp - 1, so every stage but
  // that of tile cmp is free.
  auto issue_ahead = [&](int cmp) {
#pragma unroll 1
    for (int guard = 0; guard < kStages && issued < cmp + kStages; ++guard) {
      int w;  // ring item the next tile belongs to
      if (r0.nissued < r0.ntiles) {
        w = 0;
      } else {
        if (!r1.resolved) {
          if (!r1.fetched || r1.ftile > wdone) break;
          resolve_item<D, NB>(p, sm, r1, wave);
        }
        if (r1.nissued < r1.ntiles) {
          w = 1;
        } else {
          if (!r2.resolved) {
            if (!r2.fetched || r2.ftile > wdone) break;
            resolve_item<D, NB>(p, sm, r2, wave);
          }
          if (r2.nissued >= r2.ntiles) break;
          w = 2;
        }
      }
      const int j = w == 0 ? r0.nissued : w == 1 ? r1.nissued : r2.nissued;
      const int slot = w == 0 ? r0.slot : w == 1 ? r1.slot : r2.slot;
      const int page = __builtin_amdgcn_readfirstlane(sm.desc[slot][wave][1 + j]);
      const int chunk = w == 0 ? r0.chunk : w == 1 ? r1.chunk : r2.chunk;
      const int n = w == 0 ? r0.n : w == 1 ? r1.n : r2.n;
      const int kvh = w == 0 ? r0.kvh : w == 1 ? r1.kvh : r2.kvh;
      r0.nissued += w == 0;
      r1.nissued += w == 1;
      r2.nissued += w == 2;
      const int pos = (chunk * kTilesPerChunk + j) * kTileKeys + 16 * wave;
      const bool ok = pos < n && page >= 0 && page < p.num_pages;
      const int64_t off = ok ? ((static_cast<int64_t>(page) * p.hkv + kvh) * p.page_size + (pos % p.page_size)) * D : 0;
      load_tile_rows_async<D, 16>(&sm.stage[issued % kStages][0], p.kp + off, p.vp + off, D, ok ? n - pos : 0, wave,
                                  lane);
      ++issued;
    }
  };

#pragma unroll 1
  while (blockIdx.x + seq * stride < ncand) {
    if (r0.valid) {
      f32x4 acc[NB][NDBW], lsum[NB];
      float m[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int db = 0; db < NDBW; ++db) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
        m[nb] = neg_inf();
        lsum[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
      const int qpos = r0.n - 1;
      const int last_tile = (r0.n - 1) / kTileKeys;
      bf16x8 qf[NB][D / 32];

#pragma unroll 1
      for (int j = 0; j < r0.ntiles; ++j) {
        if (issued == computed) {  // nothing in flight: start this tile's loads
          lds_barrier();
          issue_ahead(computed);
        }
        // tiles issued after this one may still be loading
        wait_tiles_barrier<Loads::kPerTile>(issued - computed - 1);
        wdone = computed;
        if (fetch_pending) {
          fetch_item<D, NB>(p, sm, r2, blockIdx.x + (seq + 2) * stride, ncand, (seq + 2) % SM::kSlots, issued, wave,
                            lane);
          fetch_pending = false;
        }
        issue_ahead(computed);
        if (j == 0) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int st = 0; st < D / 32; ++st)
              qf[nb][st] = *reinterpret_cast<const bf16x8*>(&sm.q[r0.slot][((nb * (D / 32) + st) * 64 + lane) * 8]);
        }
        const __bf16* stage = &sm.stage[computed % kStages][0];
        const int t = r0.chunk * kTilesPerChunk + j;
        // This wave's 16-key block of the scores (key block = wave index).
        f32x4 s[NB];
        qk_block<D, NB>(stage, qf, s, wave, lane);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          if (t == last_tile) mask_block(s[nb], t * kTileKeys + 16 * wave, qpos, lane);
          float bmax = vmax(vmax(s[nb][0], s[nb][1]), vmax(s[nb][2], s[nb][3]));
          bmax = max_xor16(bmax);
          bmax = max_xor32(bmax);
          if (g == 0) sm.xmax[nb][wave][col] = bmax;
        }
        lds_barrier();
        // The tile maximum (max is exact, so combining the four block maxima
        // equals the full-tile reduction), then this block's weights.
        float alpha[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const float tmax = vmax(vmax(sm.xmax[nb][0][col], sm.xmax[nb][1][col]),
                                  vmax(sm.xmax[nb][2][col], sm.xmax[nb][3][col]));
          alpha[nb] = softmax_block(s[nb], m[nb], tmax, c);
          bf16x4 pw;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) pw[jj] = to_bf16(s[nb][jj]);
          sm.pbuf[nb][wave][lane] = pw;
        }
        lds_barrier();
        // PV operand of step st: key blocks 2*st and 2*st + 1 (the pack_p order)
        bf16x8 pb[NB][2];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int st = 0; st < 2; ++st) {
            const bf16x4 lo = sm.pbuf[nb][2 * st][lane], hi = sm.pbuf[nb][2 * st + 1][lane];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              pb[nb][st][e] = lo[e];
              pb[nb][st][4 + e] = hi[e];
            }
          }
        pv_tile<D, NB, NDBW>(stage, pb, acc, lsum, alpha, wave * NDBW, lane);
        ++computed;
      }

      if (r0.nch == 1) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int gi = kQCols * nb + col;
          if (gi >= p.group) continue;
          const int64_t orow = (static_cast<int64_t>(r0.b) * p.hq + r0.kvh * p.group + gi);
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
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int gi = kQCols * nb + col;
          if (gi >= p.group) continue;
          const int64_t ws_slot =
              (static_cast<int64_t>(r0.b) * p.hq + r0.kvh * p.group + gi) * p.nchunk_max + r0.chunk;
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
        if (tid == 0) {
          sm.pend[npend][0] = r0.b * p.hkv + r0.kvh;
          sm.pend[npend][1] = r0.nch;
        }
        ++npend;
      }
    }

    // Arrivals of the pending partials, when the list is full and after the
    // last item: the workgroup that counts an entry's last outstanding chunk
    // folds them all (always in chunk order).  The drain and the barrier
    // make every wave's partial stores complete first.
    const bool last_item = blockIdx.x + (seq + 1) * stride >= ncand;
    if (npend == SM::kMaxPend || (last_item && npend > 0)) {
      wait_vmem_asm<0>();
      lds_barrier();
      if (tid < npend) {
        const int prev = __hip_atomic_fetch_add(p.ws_cnt + sm.pend[tid][0], 1, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
        sm.flag[tid] = (prev == sm.pend[tid][1] - 1);
      }
      lds_barrier();
#pragma unroll 1
      for (int i = 0; i < npend; ++i) {
        if (sm.flag[i]) {
          const int e = sm.pend[i][0];
          merge_entry<D>(p, e / p.hkv, e % p.hkv, sm.pend[i][1], tid);
          if (tid == 0) __hip_atomic_store(p.ws_cnt + e, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      // the merge issues clamped loads it does not consume; retire them with
      // a counted wait so that no load result stays pending across the loop
      wait_vmem_below<0>();
      lds_barrier();
      npend = 0;
    }

    // next item: r1 -> r0, r2 -> r1; r2 is refilled into the slot r0 used,
    // after a barrier (other waves may still read its query operands)
    if (fetch_pending) {
      lds_barrier();
      fetch_item<D, NB>(p, sm, r2, blockIdx.x + (seq + 2) * stride, ncand, (seq + 2) % SM::kSlots, issued, wave,
                        lane);
    }
    r0 = r1;
    r1 = r2;
    r2.fetched = false;
    r2.resolved = false;
    fetch_pending = true;
    ++seq;
    if (!r0.resolved) {
      if (r0.ftile > wdone) wait_vmem_asm<0>();
      resolve_item<D, NB>(p, sm, r0, wave);
    }
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
  const bool two = p.group > kQCols;
  auto launch = [&](auto kernel, size_t smem_bytes) {
    // persistent grid: as many workgroups as the CUs hold at once (LDS-bound)
    const int64_t per_cu = 2 * smem_bytes + 1024 <= kLdsBytesPerCu ? 2 : 1;
    const int64_t slots = per_cu * a.num_cus;
    const dim3 grid(static_cast<unsigned>(ncand < slots ? ncand : slots));
    hipLaunchKernelGGL(kernel, grid, dim3(256), 0, stream, p);
  };
  if (a.head_dim == 128) {
    if (two)
      launch(decode_kernel<128, 2>, sizeof(DecodeSmem<128, 2>));
    else
      launch(decode_kernel<128, 1>, sizeof(DecodeSmem<128, 1>));
  } else {
    if (two)
      launch(decode_kernel<64, 2>, sizeof(DecodeSmem<64, 2>));
    else
      launch(decode_kernel<64, 1>, sizeof(DecodeSmem<64, 1>));
  }
  return hipGetLastError();
}

}  // namespace uattn
