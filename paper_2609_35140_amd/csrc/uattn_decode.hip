// Token-wise decode entry point: one query per sequence against a paged KV cache.
//
// Work item = (256-key positional chunk, kv head, batch entry).  The G query
// heads of the kv head sit in the MFMA columns (16 per block), so each K/V
// tile is read from HBM once for the whole group.  The four waves of a
// workgroup take the chunk's four 64-key tiles, one each:
//
//   1. wave w loads the K rows of tile w straight into its score-product
//      operand registers (no LDS) and the query operands;
//   2. wave w computes the scores of tile w -- the same product, mask and
//      tile maximum as the full-sequence kernel -- publishes the column
//      maxima in LDS, and only then copies the V rows of tile w into LDS
//      slot w (direct-to-LDS), so that the K rows meet a memory system
//      without the V stream;
//   3. after one barrier every wave forms the chunk's running reference
//      maximum through its tiles in order (advance_max on the exact tile
//      maxima: the sequential online-softmax reference), wave w turns its tile
//      into bf16 weights against the reference after tile w and publishes them
//      in the PV operand order;
//   4. after a second barrier each wave walks the chunk's tiles in ascending
//      order for a quarter of the output's d range: rescale by that tile's
//      alpha (skipped when it is 1 in every lane), then accumulate V^T P^T,
//      exactly the full-sequence sequence.
//
// So every element sees the same operations, in the same order, as in the
// full-sequence kernel, with two barriers per chunk.  An item's result is
// either final (the context fits in one chunk) or an fp32 partial (m, l, acc)
// written to the workspace.
//
// The grid is persistent: as many workgroups as the CUs hold at once walk
// the items in chunk-major order, stride = grid size; the length of the next
// item's entry is read while the current item is computed.
//
// Merge: finished partials are queued per workgroup and their arrivals are
// counted when the queue is full and when the workgroup has no further
// non-empty item (one drain for many items).  The workgroup that counts an
// entry's last outstanding chunk (an arrival counter per (entry, kv head),
// reset to zero after use) folds the entry's chunk partials left to right in
// chunk order and normalizes -- the same fold, in the same order, that the
// full-sequence kernel applies at its chunk boundaries.  Chunk boundaries
// depend only on key positions, so nothing here depends on the batch, its
// order, the grid, max_seqlen or which workgroup merges.
#include <type_traits>

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
  float* ws_acc;     // [batch][Hq][nslot][D]
  float* ws_ml;      // [batch][Hq][nslot][2]
  int32_t* ws_cnt;   // [batch][Hkv] arrival counters, zero between calls
  int batch, hq, hkv, group, maxp, page_size, page_shift, num_pages, max_seqlen, nchunk_max;
  int nslot;         // partial slots per (entry, q head): nchunk_max rounded up to even
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
// Buffer access with a wave-uniform base and size: loads at (vector +
// instruction) offsets past `bytes` return zero without touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), bytes, 0x00020000);
}
__device__ __forceinline__ bf16x8 buffer_load16(__amdgpu_buffer_rsrc_t r, int voffset, int soffset) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, voffset, soffset, 0));
}

// 16 bytes per lane with the same device-coherent cache policy (sc1) as the
// scalar stores above, through a buffer resource: one store instruction per
// four partial values instead of four, and lanes whose offset lies past the
// resource's size store nothing.
constexpr int kCoherentPolicy = 16;  // the sc1 bit of the buffer instructions' cache-policy operand
__device__ __forceinline__ void st_coherent16(__amdgpu_buffer_rsrc_t r, int voffset, const f32x4& v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, voffset, 0, kCoherentPolicy);
}

// Fold the chunk partials of entry b, kv head kvh (all its q heads) in chunk
// order and write the normalized outputs.  Called by the workgroup that
// counted the entry's last outstanding chunk.  A thread folds four
// consecutive d of one q head (D/4 threads per head, 256 threads cover
// 4*256/D heads per pass), reading each chunk's four partial values with one
// 16-byte device-coherent load and the (m, l) pairs of two chunks with one
// more; the loads of kMergeBatch chunks are issued before they are folded
// (1.5 * kMergeBatch loads, below the 63 a wave can have outstanding), so a
// pass costs one memory round trip per kMergeBatch chunks.
template <int D, int kMergeBatch>
__device__ __forceinline__ void merge_entry(const DecodeParams& p, int b, int kvh, int nch, int tid) {
  static_assert(kMergeBatch % 2 == 0 && kMergeBatch * 3 / 2 < 64, "loads in flight");
  constexpr int kThreadsPerHead = D / 4;
  constexpr int kHeadsPerPass = 256 / kThreadsPerHead;
  const int d4 = 4 * (tid % kThreadsPerHead);
  // resources over the group's partials (wave-uniform); a lane's head and
  // chunk go into its offset, and offsets past the group read as zero
  const int64_t slot_g = (static_cast<int64_t>(b) * p.hq + kvh * p.group) * p.nslot;
  const auto racc = buffer_rsrc(p.ws_acc + slot_g * D, p.group * p.nslot * D * 4);
  const auto rml = buffer_rsrc(p.ws_ml + slot_g * 2, p.group * p.nslot * 2 * 4);
  for (int h0 = 0; h0 < p.group; h0 += kHeadsPerPass) {
    const int gi = h0 + tid / kThreadsPerHead;
    if (gi >= p.group) break;
    const int head = kvh * p.group + gi;
    const int k_base = gi * p.nslot;  // even, so every (m, l) pair load is 16-byte aligned
    float M = 0.f, L = 0.f;
    f32x4 A = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < nch; k0 += kMergeBatch) {
      f32x4 ba[kMergeBatch];
      f32x4 bml[kMergeBatch / 2];  // (m, l) of chunks k0 + 2i and k0 + 2i + 1
#pragma unroll
      for (int i = 0; i < kMergeBatch; ++i)
        // loads of chunks past nch are never folded (past the group's slots they read zero)
        ba[i] = __builtin_bit_cast(
            f32x4, __builtin_amdgcn_raw_buffer_load_b128(racc, ((k_base + k0 + i) * D + d4) * 4, 0, kCoherentPolicy));
#pragma unroll
      for (int i = 0; i < kMergeBatch / 2; ++i)
        bml[i] = __builtin_bit_cast(
            f32x4, __builtin_amdgcn_raw_buffer_load_b128(rml, (k_base + k0 + 2 * i) * 8, 0, kCoherentPolicy));
      // keep the scheduler from sinking the loads into the fold below (they
      // must all be in flight before the first result is needed)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < kMergeBatch; ++i) {
        const int k = k0 + i;
        const float m = bml[i / 2][2 * (i % 2)], l = bml[i / 2][2 * (i % 2) + 1];
        if (k == 0) {
          M = m;
          L = l;
#pragma unroll
          for (int j = 0; j < 4; ++j) A[j] = ba[i][j];
        } else if (k < nch) {
          const FoldScale f = fold_scale(M, m, p.c);
          L = fold_val(f, L, l);
#pragma unroll
          for (int j = 0; j < 4; ++j) A[j] = fold_val(f, A[j], ba[i][j]);
          M = f.m_new;
        }
      }
    }
    bf16x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = finalize_val(A[j], L);
    const int64_t orow = static_cast<int64_t>(b) * p.hq + head;
    *reinterpret_cast<bf16x4*>(p.out + orow * D + d4) = o;
    if (p.lse != nullptr && d4 == 0) p.lse[orow] = finalize_lse(M, L, p.c);
  }
}

// The same fold as merge_entry, in a kernel of its own that runs after a long
// walk (whose merges would otherwise all fall at its end, one workgroup per
// (entry, kv head) reading 256-chunk histories alone).  A workgroup folds
// 256 / D consecutive (entry, q head) rows, one d per thread, kMergePass chunks
// per pass.  Every wave first copies its share of the pass's partials and
// (m, l) pairs into LDS with direct-to-LDS loads, 1 KB per instruction and the
// same count in every wave (lanes of chunks past a row's count read the zero
// block): the (m, l) rows, then the first 64 chunks of every row, then the
// other 64 -- all in flight at once, which a fold from registers (at most 63
// loads per wave, each a 256-byte row piece) cannot have.  The first group is
// folded while the second lands.  Per group of 64 chunks the fold scales are
// formed lane-parallel: the running maximum before each chunk is an inclusive
// scan of the chunk maxima (the IEEE maximum is exact, associative and
// commutative, so the scan reproduces the left-to-right chain bit for bit),
// and lane i evaluates fold_scale for chunk i of the group with exactly the
// arguments the sequential fold passes.  The fold itself stays sequential in
// chunk order, reading each chunk's (a, b, l) back as one broadcast LDS load.
constexpr int kMergePass = 128;  // chunks per pass: 256 threads x 128 x 4 bytes = 128 KB of LDS

template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeParams p) {
  constexpr int R = 256 / D;                            // rows per workgroup
  constexpr int kLanesPerChunk = D / 4;                 // 16 bytes per lane
  constexpr int kChunksPerUnit = 64 / kLanesPerChunk;   // chunks per 1 KB instruction
  constexpr int kGroupUnits = R * 64 / kChunksPerUnit;  // instructions per group of 64 chunks (all rows)
  static_assert(kGroupUnits % 4 == 0 && R <= 4, "units split evenly over the waves");
  constexpr int kUnitsPerWave = kGroupUnits / 4;
  __shared__ __attribute__((aligned(1024))) float part[R][kMergePass][D];
  __shared__ __attribute__((aligned(1024))) float2 mlp[R][kMergePass];
  __shared__ f32x4 scl[4][64];  // per wave: (a, b, l) of the group's chunks

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nrows = p.batch * p.hq;
  const int row0 = blockIdx.x * R;
  const char* zero = reinterpret_cast<const char*>(g_zero_rows) + 16 * (lane & 15);
  // chunk counts of the workgroup's rows (0 past the last row and for
  // one-chunk entries, whose outputs the walk wrote)
  int nch_r[R];
  int nmax = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int row = row0 + r;
    const int n = row < nrows ? min(p.seqlens[row / p.hq], p.max_seqlen) : 0;
    nch_r[r] = (n + kChunkKeys - 1) / kChunkKeys;
    if (nch_r[r] < 2) nch_r[r] = 0;
    nmax = max(nmax, nch_r[r]);
  }
  // this thread's row (wave-uniform: D >= 64) and d
  const int my_r = __builtin_amdgcn_readfirstlane(wave * 64 / D);
  const int d = tid % D;
  const int row = row0 + my_r;
  int nch = 0;
#pragma unroll
  for (int r = 0; r < R; ++r)
    if (r == my_r) nch = nch_r[r];
  nch = __builtin_amdgcn_readfirstlane(nch);

  // group h of this wave's share of the pass at k0: kUnitsPerWave 1 KB pieces
  auto issue_group = [&](int k0, int h) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kUnitsPerWave; ++i) {
      const int u = wave + 4 * i;
      const int r = u / (64 / kChunksPerUnit);
      const int kk0 = 64 * h + (u % (64 / kChunksPerUnit)) * kChunksPerUnit;  // wave-uniform
      const int kk = kk0 + lane / kLanesPerChunk;
      int nr = 0;
#pragma unroll
      for (int rr = 0; rr < R; ++rr)
        if (rr == r) nr = nch_r[rr];
      const char* src =
          k0 + kk < nr ? reinterpret_cast<const char*>(p.ws_acc + (static_cast<int64_t>(row0 + r) * p.nslot + k0 + kk) * D +
                                                       4 * (lane % kLanesPerChunk))
                       : zero;
      dma_b128(src, __builtin_amdgcn_readfirstlane(lds_addr(&part[r][kk0][0])));
    }
  };
  // the sequential fold of chunks kb .. kb + cnt - 1 (kFull: cnt == 64)
  float M = 0.f, L = 0.f, A = 0.f;
  auto fold_group = [&](int kb, int cnt, int h, auto full_const) __attribute__((always_inline)) {
    constexpr bool kFull = decltype(full_const)::value;
    const float2 mlv = mlp[my_r][64 * h + lane];
    // running maximum through chunk kb + lane (lanes past cnt come after
    // every valid one and change none of their values)
    float run = mlv.x;
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) {
      const float o = __shfl_up(run, sh, 64);
      if (lane >= sh) run = vmax(run, o);
    }
    if (kb > 0) run = vmax(M, run);
    float before = __shfl_up(run, 1, 64);
    if (lane == 0) before = M;
    const FoldScale mine = fold_scale(before, mlv.x, p.c);
    scl[wave][lane] = f32x4{mine.a, mine.b, mlv.y, 0.f};
#pragma unroll
    for (int i0 = 0; i0 < 64; i0 += 16) {
      if (kFull || i0 < cnt) {
        float x[16];
        f32x4 f4[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          x[j] = part[my_r][64 * h + i0 + j][d];
          f4[j] = scl[wave][i0 + j];
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          if (kFull || i0 + j < cnt) {
            if (kb + i0 + j == 0) {
              L = f4[j][2];
              A = x[j];
            } else {
              FoldScale f;
              f.a = f4[j][0];
              f.b = f4[j][1];
              L = fold_val(f, L, f4[j][2]);
              A = fold_val(f, A, x[j]);
            }
          }
        }
      }
    }
    M = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, run), cnt - 1));
  };
  auto fold = [&](int kb, int h) __attribute__((always_inline)) {
    if (kb < nch) {
      const int cnt = min(64, nch - kb);
      if (cnt == 64)
        fold_group(kb, 64, h, std::true_type{});
      else
        fold_group(kb, cnt, h, std::false_type{});
    }
  };

  for (int k0 = 0; k0 < nmax; k0 += kMergePass) {
    if (wave < R) {
      // (m, l) of chunks k0 .. k0 + 127 of row `wave`: lane j holds chunks
      // k0 + 2j and k0 + 2j + 1 (the slot count is even, so both exist)
      int nr = 0;
#pragma unroll
      for (int rr = 0; rr < R; ++rr)
        if (rr == wave) nr = nch_r[rr];
      const char* src = k0 + 2 * lane < nr
                            ? reinterpret_cast<const char*>(p.ws_ml + ((static_cast<int64_t>(row0 + wave) * p.nslot + k0 + 2 * lane) * 2))
                            : zero;
      dma_b128(src, __builtin_amdgcn_readfirstlane(lds_addr(&mlp[wave][0])));
    }
    issue_group(k0, 0);
    issue_group(k0, 1);
    // the (m, l) rows and the first group have landed in every wave
    wait_barrier<kUnitsPerWave>();
    fold(k0, 0);
    wait_barrier<0>();
    fold(k0 + 64, 1);
    // every wave is done with this pass's LDS rows before the next fills them
    lds_barrier();
  }
  if (nch >= 2) {
    p.out[static_cast<int64_t>(row) * D + d] = finalize_val(A, L);
    if (p.lse != nullptr && d == 0) p.lse[row] = finalize_lse(M, L, p.c);
  }
}

constexpr int64_t kLdsBytesPerCu = 160 * 1024;
constexpr int kLenScanMax = 4096;  // batches up to this size skip chunks past their longest entry

// Buffered variant, for long walks: finished partials wait in LDS and go to
// the workspace in one burst per drain, instead of a few stores per item mixed
// into the K/V read stream (writes interleaved with a saturated read stream
// cost far more than their bytes), and decode_merge_kernel folds them after
// the walk.  Room for 16 items of 8 q heads x 128 d.
constexpr int kBufFloats = 17152;

template <int D, int NB, bool kBuf>
struct DecodeSmem {
  using TL = TileLayout<D>;
  static constexpr int kMaxPend = 32;          // finished partials awaiting their arrival count
  __bf16 v[kTilesPerChunk][TL::kTileElems];    // V tile t of the item, TileLayout V swizzle
  bf16x8 pw[kTilesPerChunk][NB][2][64];        // bf16 weights of tile t in each lane's PV operand order
  float tmax[kTilesPerChunk][NB][kQCols];      // column maxima of tile t's scores
  int32_t pend[kMaxPend][3];                   // (b * Hkv + kv head, chunk count, chunk)
  int32_t flag[kMaxPend];
  int32_t lenmax[4];                           // per wave: the longest entry it read
  // kBuf: per pending item, G rows of D + 4 floats (acc; the padding spreads
  // the 16 heads of a store over the banks), then G (m, l) pairs
  alignas(16) float pbuf[kBuf ? kBufFloats : 4];
};


// One item as a wave sees it (all fields wave-uniform).
struct Item {
  int chunk, b, kvh;
  int n;       // entry length (clamped to max_seqlen); 0 past the walk
  int nch;     // the entry's chunk count
  int ntiles;  // tiles of this chunk that hold keys (0: nothing to do)
};

template <int D, int NB, bool kBuf>
__global__ __launch_bounds__(256, kBuf ? 1 : 2) void decode_kernel(DecodeParams p, const int32_t* __restrict__ seqlens,
                                                                   const int32_t* __restrict__ block_table) {
  using TL = TileLayout<D>;
  using SM = DecodeSmem<D, NB, kBuf>;
  constexpr int KS = D / 32;                   // K steps of the score product
  constexpr int NDBW = D / 16 / 4;             // 16-wide d blocks of the output per wave
  constexpr int kVInstr = TL::kPieces;         // 1 KB direct-to-LDS instructions per V tile
  constexpr int kRowsPerInstr = 64 / TL::kPieces;
  static_assert(16 % kRowsPerInstr == 0, "an instruction's rows lie in one 16-key block");
  __shared__ __attribute__((aligned(1024))) SM sm;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, col = lane & 15, row16 = lane & 15;
  const int per_chunk = p.batch * p.hkv;
  const int ncand_all = per_chunk * p.nchunk_max;
  const int stride = gridDim.x;
  const float c = p.c;
  const __bf16* zero = reinterpret_cast<const __bf16*>(g_zero_rows);

  // Chunks past the longest entry hold no work.  When this workgroup's walk
  // is longer than two items, read the batch's lengths first and stop the
  // walk after the last chunk any entry has, so that a max_seqlen far above
  // the actual lengths costs no round trips for empty items.
  int ncand = ncand_all;
  if (p.nchunk_max > 1 && p.batch <= kLenScanMax && ncand_all > 2 * stride) {
    int lmax = 0;
    for (int i = tid; i < p.batch; i += 256) lmax = max(lmax, p.seqlens[i]);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) lmax = max(lmax, __shfl_xor(lmax, m));
    if (lane == 0) sm.lenmax[wave] = lmax;
    __syncthreads();
    lmax = max(max(sm.lenmax[0], sm.lenmax[1]), max(sm.lenmax[2], sm.lenmax[3]));
    const int nch = min(max((min(lmax, p.max_seqlen) + kChunkKeys - 1) / kChunkKeys, 1), p.nchunk_max);
    ncand = __builtin_amdgcn_readfirstlane(per_chunk * nch);
  }

  // An item's descriptor, for this wave: the entry length and the page of
  // each 16-key block of the wave's tile (table index clamped, so
  // speculative).  Wave-uniform loads of read-only arguments, so they are
  // scalar loads, counted apart from the vector loads and stores; the next
  // item's are issued before the current item's operand loads.
  struct Desc {
    int len;
    int page[kKeyBlocks];
  };
  auto load_desc = [&](int it) -> Desc {
    Desc d;
    const int chunk = it / per_chunk, b = (it % per_chunk) / p.hkv;
    const int32_t* row = block_table + static_cast<int64_t>(b) * p.maxp;
    d.len = seqlens[b];
#pragma unroll
    for (int kb = 0; kb < kKeyBlocks; ++kb) {
      const int pos = (chunk * kTilesPerChunk + wave) * kTileKeys + 16 * kb;
      d.page[kb] = row[min(pos >> p.page_shift, p.maxp - 1)];
    }
    return d;
  };
  auto make_item = [&](int it, const Desc& desc) -> Item {
    Item r;
    r.chunk = it / per_chunk;
    r.b = (it % per_chunk) / p.hkv;
    r.kvh = it % p.hkv;
    r.n = it < ncand ? min(desc.len, p.max_seqlen) : 0;
    r.nch = (r.n + kChunkKeys - 1) / kChunkKeys;
    r.ntiles = (r.n >= 1 && r.chunk < r.nch) ? min(kTilesPerChunk, (r.n - 1) / kTileKeys - r.chunk * kTilesPerChunk + 1) : 0;
    return r;
  };

  // Count the arrivals of the pending partials: the workgroup that counts an
  // entry's last outstanding chunk folds them all (always in chunk order).
  // The drain and the barrier make every wave's partial stores complete first.
  int npend = 0;
  // kBatch: chunks whose partials a merging thread loads at once (fewer in the
  // drains inside the walk, where the next item's operands hold registers)
  // buffered partials: one slot per pending item (16-byte aligned)
  const int item_floats = (p.group * (D + 4) + 2 * p.group + 3) & ~3;
  const int cap = kBuf ? min(SM::kMaxPend, kBufFloats / item_floats) : SM::kMaxPend;
  auto drain = [&](auto batch_const) {
    constexpr int kBatch = decltype(batch_const)::value;
    if constexpr (kBuf) {
      // the pending partials from LDS to their workspace rows, 16 bytes per
      // thread and step, consecutive threads along a row; plain stores, read
      // only by the merge kernel that follows, so nothing waits for them
      lds_barrier();
      constexpr int kRowPieces = D / 4;
      const int per_item = p.group * kRowPieces;
#pragma unroll 1
      for (int k = tid; k < npend * per_item; k += 256) {
        const int sl = k / per_item, r = k % per_item;
        const int gi = r / kRowPieces, pc = r % kRowPieces;
        const int e = sm.pend[sl][0];
        const int64_t row =
            (static_cast<int64_t>(e / p.hkv) * p.hq + (e % p.hkv) * p.group + gi) * p.nslot + sm.pend[sl][2];
        *reinterpret_cast<f32x4*>(p.ws_acc + row * D + 4 * pc) =
            *reinterpret_cast<const f32x4*>(sm.pbuf + sl * item_floats + gi * (D + 4) + 4 * pc);
      }
#pragma unroll 1
      for (int k = tid; k < npend * p.group; k += 256) {
        const int sl = k / p.group, gi = k % p.group;
        const int e = sm.pend[sl][0];
        const int64_t row =
            (static_cast<int64_t>(e / p.hkv) * p.hq + (e % p.hkv) * p.group + gi) * p.nslot + sm.pend[sl][2];
        *reinterpret_cast<float2*>(p.ws_ml + row * 2) =
            *reinterpret_cast<const float2*>(sm.pbuf + sl * item_floats + p.group * (D + 4) + 2 * gi);
      }
      // every thread's reads of the slots are done before they are refilled
      lds_barrier();
      npend = 0;
      return;
    }
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
        merge_entry<D, kBatch>(p, e / p.hkv, e % p.hkv, sm.pend[i][1], tid);
        if (tid == 0) __hip_atomic_store(p.ws_cnt + e, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    // the merge issues clamped loads it does not consume; retire them with
    // a counted wait so that no load result stays pending
    wait_vmem_below<0>();
    lds_barrier();
    npend = 0;
  };

  // per-lane offsets of the buffer loads (the bounds check covers the vector
  // and instruction offsets, so every per-lane part goes there): query
  // operands (+ the 16-head block + 64*step) and K operands (+ 64*step)
  const int q_off = col * D * 2 + 16 * g;
  const int k_off = row16 * D * 2 + 16 * g;

  // This wave's operands of an item: the group's query rows and the K rows
  // of its tile, both in the score product's operand registers (query
  // column col, d = 32*step + 8*g .. +7; key 16*kb + row, the same d), and
  // where the tile's 16-key blocks live.  Every block is loaded through a
  // buffer resource sized to its valid bytes, so rows past the context,
  // blocks on a page outside the pool and tiles or items outside the walk
  // read as zero without touching memory -- and the number of loads is always
  // kOpLoads, which the V wait below relies on.
  constexpr int kOpLoads = (kKeyBlocks + NB) * KS;
  struct Operands {
    bf16x8 qf[NB][KS];
    bf16x8 kf[kKeyBlocks][KS];
    int64_t boff[kKeyBlocks];  // element offset of key 16*kb of the tile in the pools, -1 if none
    int rows[kKeyBlocks];      // keys of block kb inside the context
  };
  auto issue_ops = [&](const Item& it, const Desc& desc, Operands& op) {
    const __bf16* qb = p.q + (static_cast<int64_t>(it.b) * p.hq + it.kvh * p.group) * D;
    const auto rq = buffer_rsrc(qb, it.ntiles > 0 ? p.group * D * 2 : 0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int st = 0; st < KS; ++st) op.qf[nb][st] = buffer_load16(rq, q_off + nb * kQCols * D * 2 + 64 * st, 0);
    const int tile = it.chunk * kTilesPerChunk + wave;
    const bool on = wave < it.ntiles;
#pragma unroll
    for (int kb = 0; kb < kKeyBlocks; ++kb) {
      const int pos = tile * kTileKeys + 16 * kb;
      const int page = desc.page[kb];
      const bool ok = on && page >= 0 && page < p.num_pages && pos < it.n;
      op.rows[kb] = ok ? min(it.n - pos, 16) : 0;
      op.boff[kb] = ok ? ((static_cast<int64_t>(page) * p.hkv + it.kvh) * p.page_size + (pos & (p.page_size - 1))) * D
                       : -1;
      const auto rk = buffer_rsrc(p.kp + (ok ? op.boff[kb] : 0), op.rows[kb] * D * 2);
#pragma unroll
      for (int st = 0; st < KS; ++st) op.kf[kb][st] = buffer_load16(rk, k_off + 64 * st, 0);
    }
  };

  // Software-pipelined walk: an item's query and K operands are loaded
  // during the previous item (issued right after that item's V copies), so
  // every workgroup keeps one item's K rows in flight through the softmax
  // and PV phases.
  Desc desc = load_desc(blockIdx.x);
  Item cur = make_item(blockIdx.x, desc);
  Desc desc_next = load_desc(min(blockIdx.x + stride, ncand_all - 1));
  Operands op;
  issue_ops(cur, desc, op);
#pragma unroll 1
  for (int item = blockIdx.x; item < ncand; item += stride) {
    const Item next = make_item(item + stride, desc_next);   // empty past the walk
    const Desc desc_after = load_desc(min(item + 2 * stride, ncand_all - 1));
    const int tile = cur.chunk * kTilesPerChunk + wave;  // this wave's tile (sequence-relative)
    const bool tile_on = wave < cur.ntiles;

    // V rows go into LDS slot `wave` by direct-to-LDS loads (16-byte pieces
    // XOR-swizzled per row), rows past the context from the zero block, so
    // that V rows meeting zero weights are zero, never stale or NaN.
    f32x4 s[NB][kKeyBlocks];
    if (cur.ntiles > 0) {
      // scores of this wave's tile and their column maxima
      if (tile_on) {
#pragma unroll
        for (int kb = 0; kb < kKeyBlocks; ++kb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int st = 0; st < KS; ++st) a = mfma16(op.kf[kb][st], op.qf[nb][st], a);
            s[nb][kb] = a;
          }
        const int last_tile = (cur.n - 1) / kTileKeys;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          if (tile == last_tile) mask_scores(s[nb], tile * kTileKeys, cur.n - 1, lane);
          const float tm = tile_max(s[nb]);
          if (g == 0) sm.tmax[wave][nb][col] = tm;
        }
        // V rows into LDS slot `wave` once the scores are formed, so that
        // the K rows had the memory system to themselves
        const uint32_t vbase = __builtin_amdgcn_readfirstlane(lds_addr(&sm.v[wave][0]));
#pragma unroll
        for (int i = 0; i < kVInstr; ++i) {
          const int slot = i * 64 + lane;
          const int row = slot / TL::kPieces, piece = slot % TL::kPieces;
          const int kb = (i * kRowsPerInstr) / 16;
          const bool ok = (row & 15) < op.rows[kb];
          const __bf16* src =
              ok ? p.vp + op.boff[kb] + (row & 15) * D + 8 * (piece ^ TL::v_swz(row)) : zero + 8 * (lane & 15);
          dma_b128(src, vbase + i * 64 * 16);
        }
      }
    }
    // the next item's operands: exactly kOpLoads loads after this item's V copies
    Operands op_next;
    issue_ops(next, desc_next, op_next);

    if (cur.ntiles > 0) {
      lds_barrier();

      // the chunk's running reference through its tiles in order, each
      // tile's alpha, and this wave's weights against its tile's reference
      float alpha[kTilesPerChunk][NB], m_end[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        float m = neg_inf(), m_mine = neg_inf();
#pragma unroll
        for (int t = 0; t < kTilesPerChunk; ++t) {
          if (t < cur.ntiles) {
            alpha[t][nb] = advance_max(m, sm.tmax[t][nb][col], c);
            if (t == wave) m_mine = m;
          }
        }
        m_end[nb] = m;
        if (tile_on) {
          tile_weights(s[nb], m_mine, c);
          bf16x8 pb[2];
          pack_p(s[nb], pb);
          sm.pw[wave][nb][0][lane] = pb[0];
          sm.pw[wave][nb][1][lane] = pb[1];
        }
      }
      // this wave's V rows have landed (only the next item's operand loads
      // may still be in flight); after the barrier every wave's have
      wait_barrier<kOpLoads>();
      // PV over the chunk's tiles in ascending order, d blocks NDBW*wave ..
      f32x4 acc[NB][NDBW], lsum[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int db = 0; db < NDBW; ++db) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
        lsum[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int t = 0; t < kTilesPerChunk; ++t) {
        if (t < cur.ntiles) {
          bf16x8 pb[NB][2];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            pb[nb][0] = sm.pw[t][nb][0][lane];
            pb[nb][1] = sm.pw[t][nb][1][lane];
          }
          pv_tile<D, NB, NDBW>(&sm.v[t][0], pb, acc, lsum, alpha[t], wave * NDBW, lane);
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
          if (p.lse != nullptr && wave == 0 && g == 0) p.lse[orow] = finalize_lse(m_end[nb], lsum[nb][0], c);
        }
      } else if constexpr (kBuf) {
        // this chunk's partial into LDS slot npend (the drain writes it out)
        float* slotp = sm.pbuf + npend * item_floats;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int gi = kQCols * nb + col;
          if (gi < p.group) {
#pragma unroll
            for (int db = 0; db < NDBW; ++db)
              *reinterpret_cast<f32x4*>(slotp + gi * (D + 4) + 16 * (wave * NDBW + db) + 4 * g) = acc[nb][db];
            if (wave == 0 && g == 0) {
              slotp[p.group * (D + 4) + 2 * gi] = m_end[nb];
              slotp[p.group * (D + 4) + 2 * gi + 1] = lsum[nb][0];
            }
          }
        }
        if (tid == 0) {
          sm.pend[npend][0] = cur.b * p.hkv + cur.kvh;
          sm.pend[npend][1] = cur.nch;
          sm.pend[npend][2] = cur.chunk;
        }
        ++npend;
      } else {
        // the group's partial rows of this chunk: [head gi][chunk][d], heads
        // past the group fall outside the resource and store nothing
        const int64_t slot0 = (static_cast<int64_t>(cur.b) * p.hq + cur.kvh * p.group) * p.nslot;
        const auto racc = buffer_rsrc(p.ws_acc + slot0 * D, p.group * p.nslot * D * 4);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int gi = kQCols * nb + col;
          const int voff = ((gi * p.nslot + cur.chunk) * D + 16 * wave * NDBW + 4 * g) * 4;
#pragma unroll
          for (int db = 0; db < NDBW; ++db) st_coherent16(racc, voff + 64 * db, acc[nb][db]);
          if (gi < p.group && wave == 0 && g == 0) {
            const int64_t ws_slot = slot0 + static_cast<int64_t>(gi) * p.nslot + cur.chunk;
            st_coherent(p.ws_ml + ws_slot * 2, m_end[nb]);
            st_coherent(p.ws_ml + ws_slot * 2 + 1, lsum[nb][0]);
          }
        }
        if (tid == 0) {
          sm.pend[npend][0] = cur.b * p.hkv + cur.kvh;
          sm.pend[npend][1] = cur.nch;
          sm.pend[npend][2] = cur.chunk;
        }
        ++npend;
      }
      // every wave is done with the V tiles, weights and maxima of this item
      lds_barrier();
    }
    if (npend == cap) drain(std::integral_constant<int, 8>{});
    cur = next;
    op = op_next;
    desc_next = desc_after;
  }
  // the end of the walk: count what is pending, and retire the last
  // (empty) operand prefetch
  if (npend > 0) drain(std::integral_constant<int, 32>{});
  wait_vmem_below<0>();
}

}  // namespace

int64_t decode_slots(int64_t nchunk) { return (nchunk + 1) / 2 * 2; }
size_t decode_ws_acc_bytes(int64_t batch, int64_t nchunk, int64_t num_q_heads, int64_t head_dim) {
  return (static_cast<size_t>(batch * num_q_heads * decode_slots(nchunk) * head_dim) * sizeof(float) + 255) / 256 * 256;
}
size_t decode_ws_ml_bytes(int64_t batch, int64_t nchunk, int64_t num_q_heads) {
  return (static_cast<size_t>(batch * num_q_heads * decode_slots(nchunk) * 2) * sizeof(float) + 255) / 256 * 256;
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
  p.page_shift = __builtin_ctz(static_cast<unsigned>(a.page_size));
  p.num_pages = a.num_pages;
  p.max_seqlen = a.max_seqlen;
  p.nchunk_max = a.nchunk_max;
  p.nslot = static_cast<int>(decode_slots(a.nchunk_max));
  p.c = a.c;
  p.batch = a.batch;
  const int64_t ncand = static_cast<int64_t>(a.batch) * a.num_kv_heads * a.nchunk_max;
  if (ncand > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  const bool two = p.group > kQCols;
  // long walks (at least 16 items per CU): the buffered variant, one
  // workgroup per CU
  const bool buffered = a.nchunk_max > 1 && ncand >= 16 * static_cast<int64_t>(a.num_cus);
  auto launch = [&](auto kernel, size_t smem_bytes) {
    // persistent grid: as many workgroups as the CUs hold at once (LDS-bound)
    const int64_t per_cu = 2 * smem_bytes + 1024 <= kLdsBytesPerCu ? 2 : 1;
    const int64_t slots = per_cu * a.num_cus;
    const dim3 grid(static_cast<unsigned>(ncand < slots ? ncand : slots));
    hipLaunchKernelGGL(kernel, grid, dim3(256), 0, stream, p, p.seqlens, p.bt);
  };
  auto pick = [&](auto d_const, auto nb_const) {
    constexpr int kD = decltype(d_const)::value, kNB = decltype(nb_const)::value;
    if (buffered) {
      launch(decode_kernel<kD, kNB, true>, sizeof(DecodeSmem<kD, kNB, true>));
      constexpr int kRows = 256 / kD;
      const int64_t rows = static_cast<int64_t>(a.batch) * a.num_q_heads;
      hipLaunchKernelGGL(decode_merge_kernel<kD>, dim3(static_cast<unsigned>((rows + kRows - 1) / kRows)), dim3(256), 0,
                         stream, p);
    } else {
      launch(decode_kernel<kD, kNB, false>, sizeof(DecodeSmem<kD, kNB, false>));
    }
  };
  if (a.head_dim == 128) {
    if (two)
      pick(std::integral_constant<int, 128>{}, std::integral_constant<int, 2>{});
    else
      pick(std::integral_constant<int, 128>{}, std::integral_constant<int, 1>{});
  } else {
    if (two)
      pick(std::integral_constant<int, 64>{}, std::integral_constant<int, 2>{});
    else
      pick(std::integral_constant<int, 64>{}, std::integral_constant<int, 1>{});
  }
  return hipGetLastError();
}

}  // namespace uattn
