// Full-sequence entry point: causal GQA attention over a packed varlen batch.
//
// Workgroup = 8 waves = 256 consecutive query rows of one q head of one
// sequence; each wave owns 32 rows (two 16-column MFMA blocks, one row per
// column).  Waves w and w+4 share SIMD w%4 and own adjacent 32-row runs, so
// the two waves of a SIMD walk the same number of tiles.
//
// Ping-pong schedule.  A wave's work per 64-key tile t is a matrix phase
// (the weighted V of tile t-1, then the scores of tile t: MFMAs and LDS reads
// only) and a vector phase (the fold of a finished chunk, the softmax step of
// tile t and, when its reference moved, the rescale of the accumulators by
// its alpha: VALU only).  Each phase runs in a slot opened by a workgroup
// barrier; waves 4-7 run one slot behind waves 0-3, so in every slot one wave
// of each SIMD issues matrix products (at raised priority) while the other
// issues the vector work, and the two units run side by side.  The
// arithmetic of every row is the shared per-tile sequence of
// uattn_numerics.h in the same order (alpha multiplies the accumulators
// before the product adds to them; chunks of 4 tiles folded left to right),
// so the results are the same bits as the token-wise decode.
//
// LDS: two slots, slot u%2 holding K of tile u and V of tile u-1 (what the
// matrix phase of step u reads).  Waves 0-3 load the slots: slot (u+1)%2 is
// issued when they open the matrix phase of step u (its previous contents'
// last readers, the late waves' matrix phase of step u-1, are done) and has
// landed before they open the matrix phase of step u+1 (a wait for all their
// loads), two slots later.
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

constexpr int kWaves = 8;
constexpr int kNB = 2;                       // 16-column MFMA blocks (query groups) per wave
constexpr int kWaveRows = kNB * kQCols;
constexpr int kWgRows = kWaves * kWaveRows;
constexpr int kLoadWaves = 4;                // waves 0-3 issue every tile load
constexpr int kRowsPerLoadWave = kTileKeys / kLoadWaves;

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

// Byte offset, from the address of the wave's first row, of the 16-byte
// piece this lane fetches in the first load instruction of a K (V) tile.
// Instruction i of a wave covers rows 64/pieces*i further on, and its swizzle
// differs from the first instruction's by a constant XOR of bits the row term
// does not touch (row_stride*2 is a multiple of 16*pieces), so
//   offset(i) = (64/pieces*i) * row_stride*2  +  (offset(0) ^ tile_xor(i)).
template <int D, bool kIsV>
__device__ __forceinline__ uint32_t load_lane_offset(int lane, int64_t row_stride) {
  using TL = TileLayout<D>;
  const int gp = lane / TL::kPieces, piece = lane % TL::kPieces;
  const int swz = kIsV ? TL::v_swz(gp) : TL::k_swz(gp);
  return static_cast<uint32_t>((gp * row_stride + 8 * (piece ^ swz)) * 2);
}
template <int D, bool kIsV>
__device__ __forceinline__ constexpr uint32_t tile_xor(int i) {
  return kIsV ? (D == 128 ? 128u * (i & 1) : 0u) : 64u * i;
}

// Issue this wave's rows of one K or V tile (rows RPW*w .. RPW*w+RPW-1, RPW =
// 64 / kLoadWaves) into the LDS tile at `tile`, swizzled as TileLayout reads
// them.  nvalid: rows RPW*w + r with r < nvalid hold keys; the rest are zeros.
//   lane_off : load_lane_offset<D, kIsV>(lane, row_stride)
template <int D, bool kIsV>
__device__ __forceinline__ void load_rows(__bf16* tile, const __bf16* base, int64_t row_stride, int nvalid, int w,
                                          int lane, uint32_t lane_off) {
  using TL = TileLayout<D>;
  constexpr int RPW = kRowsPerLoadWave;
  constexpr int kInstr = RPW * TL::kPieces / 64;
  constexpr int kRowsPerInstr = 64 / TL::kPieces;
  static_assert(kInstr >= 1 && RPW * TL::kPieces == 64 * kInstr, "tile split");
  const uint32_t d0 = __builtin_amdgcn_readfirstlane(lds_addr(tile + w * kInstr * 64 * 8));
  if (nvalid >= RPW) {
#pragma unroll
    for (int i = 0; i < kInstr; ++i)
      dma_b128_based(base + kRowsPerInstr * i * row_stride, lane_off ^ tile_xor<D, kIsV>(i), d0 + i * 64 * 16);
    return;
  }
  // a tile past the end of the sequence (rare): the per-lane addresses are
  // formed here, from a lane index the compiler cannot hoist out of the tile
  // loop (held there they would cost registers every tile)
  asm volatile("" : "+v"(lane));
  const __bf16* zero = reinterpret_cast<const __bf16*>(g_zero_rows) + 8 * (lane & 15);
#pragma unroll
  for (int i = 0; i < kInstr; ++i) {
    const int slot = (w * kInstr + i) * 64 + lane;
    const int row = slot / TL::kPieces, piece = slot % TL::kPieces;
    const int r = row - RPW * w;
    const int swz = kIsV ? TL::v_swz(row) : TL::k_swz(row);
    const __bf16* src = r < nvalid ? base + r * row_stride + 8 * (piece ^ swz) : zero;
    dma_b128(src, d0 + i * 64 * 16);
  }
}

// Matrix phase of one step: O^T += V^T P^T for the previous tile (the
// vector phase has already multiplied acc and lsum by its alpha; kFirst
// starts the products from zero), then S^T = K Q^T for this tile.  The
// LDS reads run kVAhead d blocks (and two key blocks) ahead of the products
// that use them, in a fixed order, so that one wave alone keeps the matrix
// unit fed while the other wave of its SIMD runs vector work.
template <int D, int NB, bool kFirst>
__device__ __forceinline__ void matrix_phase(const __bf16* slot, const bf16x8 (&pb)[NB][2],
                                             const bf16x8 (&qf)[NB][D / 32], f32x4 (&acc)[NB][D / 16],
                                             f32x4 (&lsum)[NB], f32x4 (&s)[NB][4], int lane) {
  using TL = TileLayout<D>;
  constexpr int NDB = D / 16, KS = D / 32;
  constexpr int kVAhead = 3;
  const int g = lane >> 4, src = lane & 15;
  // V operands (transposing reads), as pv_tile.  The d block enters the LDS
  // address only through a XOR of bits that the rest of it leaves clear
  // (rows are D*2 bytes, the swizzle is even), so one register holds the
  // address of d block 0 and each block's is one XOR away; it is made opaque
  // so that the compiler keeps one register rather than all the blocks'.
  const int key = 4 * g + (src >> 2);
  const int sub = src & 3;
  uint32_t va0 = lds_addr(slot + TL::kTileElems + key * D + 4 * (sub & 1)) + 16 * (sub >> 1) + 16 * TL::v_swz(key);
  asm volatile("" : "+v"(va0));
  auto vread = [&](int db, bf16x8(&a)[2]) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const lds_s16x4* vp = reinterpret_cast<const lds_s16x4*>(static_cast<uintptr_t>(va0 ^ (32u * db)));
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_s16x4*>(vp + (32 * st) * D / 4));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_s16x4*>(vp + (32 * st + 16) * D / 4));
      const s16x4 w[2] = {lo, hi};
      __builtin_memcpy(&a[st], w, sizeof(bf16x8));
    }
  };
  // K operands, as qk_scores, addressed the same way: the K step enters the
  // address as a XOR of bits 6-7 (rows of D*2 bytes, pieces of 16)
  const int row = lane & 15;
  uint32_t ka0 = lds_addr(slot + row * D) + 16 * (g ^ TL::k_swz(row));
  asm volatile("" : "+v"(ka0));
  auto kread = [&](int kb, bf16x8(&a)[KS]) {
    typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      const lds_bf16x8* kp = reinterpret_cast<const lds_bf16x8*>(static_cast<uintptr_t>(ka0 ^ (64u * st)));
      a[st] = kp[16 * kb * D / 8];
    }
  };
  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = static_cast<__bf16>(1.0f);

  bf16x8 va[kVAhead][2];
  bf16x8 ka[2][KS];
#pragma unroll
  for (int i = 0; i < kVAhead; ++i) vread(i, va[i]);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if constexpr (kFirst) lsum[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 2; ++st) lsum[nb] = mfma16(ones, pb[nb][st], lsum[nb]);
  }
  __builtin_amdgcn_sched_barrier(0);
  // d block db: its four products, the LDS reads kVAhead blocks ahead
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    bf16x8(&a)[2] = va[db % kVAhead];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if constexpr (kFirst) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 2; ++st) acc[nb][db] = mfma16(a[st], pb[nb][st], acc[nb][db]);
    }
    if (db + kVAhead < NDB) vread(db + kVAhead, va[db % kVAhead]);
    if (db == NDB - 3) kread(0, ka[0]);
    if (db == NDB - 1) kread(1, ka[1]);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int kb = 0; kb < kKeyBlocks; ++kb) {
    bf16x8(&a)[KS] = ka[kb & 1];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4 r = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < KS; ++st) r = mfma16(a[st], qf[nb][st], r);
      s[nb][kb] = r;
    }
    if (kb + 2 < kKeyBlocks) kread(kb + 2, ka[kb & 1]);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int D>
__global__ __launch_bounds__(kWaves * 64, 1) void prefill_kernel(PrefillParams p) {
  constexpr int NDB = D / 16;  // 16-wide d blocks of the output
  using TL = TileLayout<D>;
  __shared__ __attribute__((aligned(1024))) __bf16 lds[2 * TL::kStageElems];

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
  const int simd = wave & 3;
  const bool late = wave >= 4;  // runs one slot behind
  const int g = lane >> 4, col = lane & 15;
  // waves w and w+4 (one SIMD) own rows 64*(w%4) .. +63 of the workgroup's 256
  const int q0 = qt * kWgRows + 2 * kWaveRows * simd + (late ? kWaveRows : 0);
  const bool wave_on = q0 < L;
  const int wg_last_tile = min(qt * kWgRows + kWgRows - 1, L - 1) / kTileKeys;
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

  const int64_t row_stride = static_cast<int64_t>(p.hkv) * D;
  const uint32_t koff = load_lane_offset<D, false>(lane, row_stride);
  const uint32_t voff = load_lane_offset<D, true>(lane, row_stride);
  // slot u%2 <- K of tile u (if u <= wg_last_tile), V of tile u-1 (if u >= 1); waves 0-3 only
  auto issue_slot = [&](int u) {
    __bf16* slot = lds + (u & 1) * TL::kStageElems;
    if (u <= wg_last_tile) {
      const int pos = u * kTileKeys + kRowsPerLoadWave * wave;
      load_rows<D, false>(slot, p.k + (static_cast<int64_t>(lo + pos) * p.hkv + kvh) * D, row_stride, L - pos, wave,
                          lane, koff);
    }
    if (u >= 1) {
      const int pos = (u - 1) * kTileKeys + kRowsPerLoadWave * wave;
      load_rows<D, true>(slot + TL::kTileElems, p.v + (static_cast<int64_t>(lo + pos) * p.hkv + kvh) * D, row_stride,
                         L - pos, wave, lane, voff);
    }
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
  f32x4 s[kNB][4];
  bf16x8 pb[kNB][2];

  // (M, Ls, A) <- (M, Ls, A) (+) (m, lsum, acc): the chunk ending with tile u
  auto fold = [&](int u) {
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
      if (u < kTilesPerChunk) {
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
    }
  };

  if (!late) issue_slot(0);
  // The Q^T operands and slot 0 have landed: said with the compiler's own
  // wait, so that it keeps no load pending into the loop.
  wait_vmem_below<0>();
  if (late) __builtin_amdgcn_s_barrier();  // the late waves' extra slot (nothing is pending here)
  const int T = wg_last_tile + 1;  // steps 0 .. T; step T only adds tile T-1's weighted V
  // step u at position POS = u % 4 of its chunk (so slot u%2 = POS%2)
  auto step = [&](int u, auto pos_const) {
    constexpr int POS = decltype(pos_const)::value;
    constexpr int PPOS = (POS + kTilesPerChunk - 1) % kTilesPerChunk;  // (u-1) % 4
    __bf16* slot = lds + (POS & 1) * TL::kStageElems;
    // ---- matrix phase: slot u is complete in every wave (the loading waves
    // wait for all their loads: slot u+1 is not issued yet), slot u-1's
    // readers are done
    // (the wait is the compiler's own, so that it knows nothing is pending;
    // the late waves issue no loads, so for them it is free)
    __builtin_amdgcn_sched_barrier(0);
    wait_vmem_below<0>();
    lds_barrier();
    // the matrix phase first: its wave takes the issue slots it can use, the
    // other wave of the SIMD fills the rest with its vector work
    __builtin_amdgcn_s_setprio(2);
    __builtin_amdgcn_sched_barrier(0);
    if (!late && u + 1 <= T) issue_slot(u + 1);
    // the previous tile's weighted V (if this wave has one) and this tile's
    // scores (discarded past the wave's last tile, and at step T where the
    // slot holds no K); s and pb are written on every path, so that no old
    // value of them stays live around the loop
    if (wave_on && u >= 1 && u - 1 <= my_last_tile) {
      matrix_phase<D, kNB, PPOS == 0>(slot, pb, qf, acc, lsum, s, lane);
    } else if (wave_on && u == 0) {
      qk_scores<D, kNB>(slot, qf, s, lane);
    } else {
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) asm volatile("" : "=v"(s[nb][kb]));
    }
    // ---- vector phase
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    __builtin_amdgcn_s_setprio(0);
    __builtin_amdgcn_sched_barrier(0);
    if (wave_on && u <= my_last_tile) {
      if constexpr (POS == 0) {
        // a new chunk: fold the finished one (its last weighted V was added in
        // this step's matrix phase); acc and lsum restart in the products
        if (u >= kTilesPerChunk) fold(u - 1);
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) m[nb] = neg_inf();
      }
      float alpha[kNB];
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) {
        if (u == my_last_tile) mask_scores(s[nb], u * kTileKeys, q0 + kQCols * nb + col, lane);
        alpha[nb] = softmax_tile(s[nb], m[nb], c);
        pack_p(s[nb], pb[nb]);
      }
      // a later tile of the chunk: acc and lsum follow a moved reference
      // before the next matrix phase adds this tile's weighted V
      if constexpr (POS != 0) rescale_acc<kNB, NDB>(acc, lsum, alpha);
    } else {
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) {
        asm volatile("" : "=v"(pb[nb][0]));
        asm volatile("" : "=v"(pb[nb][1]));
      }
    }
  };
  for (int u = 0; u <= T; u += 4) {
    step(u, std::integral_constant<int, 0>{});
    if (u + 1 <= T) step(u + 1, std::integral_constant<int, 1>{});
    if (u + 2 <= T) step(u + 2, std::integral_constant<int, 2>{});
    if (u + 3 <= T) step(u + 3, std::integral_constant<int, 3>{});
  }
  if (!late) lds_barrier();  // the early waves' matching slot
  // the last (possibly partial) chunk
  if (wave_on) fold(my_last_tile);

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
