// Backward of the full-sequence path: dQ, dK and dV of causal GQA attention
// over a packed varlen batch, from the forward's output and log-sum-exp.
//
// For one (sequence, q head), with S = scale * Q K^T masked causally,
// P = softmax(S), O = P V (Section 3.2) and an upstream gradient dO:
//   dV = P^T dO,   dP = dO V^T,   dS = P * (dP - D) with D_i = dO_i . O_i,
//   dQ = scale * dS K,   dK = scale * dS^T Q,
// and the q heads of a group add their dK and dV.  P is recomputed from the
// saved log-sum-exp: P_ij = exp2(s_ij * c - lse_i * log2(e)), c = scale * log2(e).
//
// Deterministic and batch-invariant by construction: there are no atomics,
// and every output row is accumulated by exactly one workgroup, in an order
// that depends on nothing but its own sequence:
//   bwd_prep_kernel  D_i and lse_i * log2(e) of every (token, q head), written
//                    head-major into the workspace;
//   bwd_dkdv_kernel  one workgroup per (128-key tile, sequence, kv head); wave w
//                    owns keys 32w .. 32w+31 and keeps their K and V operands and
//                    the dK^T, dV^T accumulators in registers while it walks the
//                    group's q heads, then the 64-query tiles at or after its
//                    keys, in ascending order (S = Q K^T with the keys as MFMA
//                    columns, so P and dS already sit in the layout the dV^T and
//                    dK^T products consume);
//   bwd_dq_kernel    one workgroup per (256-query tile, sequence, q head), laid
//                    out as the forward (queries as MFMA columns): walks the
//                    64-key tiles up to each wave's diagonal in ascending order.
// Both products of dS and P with Q, dO or K take their transposed operand
// from the transposing LDS read (ds_read_b64_tr_b16); all tiles move by
// direct-to-LDS loads with explicit wait counts, as in the forward.
#include <type_traits>

#include "uattn_internal.h"
#include "uattn_numerics.h"
#include "uattn_tile_io.h"

namespace uattn {
namespace {

// One [64 rows][D] bf16 tile in LDS, read two ways: row fragments
// (ds_read_b128, a 16-lane group reads 16 consecutive rows at one logical
// 16-byte piece) and transposing reads (ds_read_b64_tr_b16, a 16-lane group
// reads 4 consecutive rows x 2 adjacent pieces; 32 lanes share an LDS cycle).
// The 16-byte pieces of each row are XOR-swizzled by 2 * (row & 7).  For
// d = 128 this was measured with the LDS bank-conflict counter on gfx950: it
// leaves both patterns conflict-free, while swizzles that spread 16 rows over
// 16 distinct pieces conflict on one pattern or the other.  For d = 64, whose
// 128-byte rows pair up in a 256-byte bank line, the same permutation is
// applied to row pairs (2 * ((row >> 1) & 3)).
template <int D>
struct BwdTile {
  static constexpr int kPieces = D / 8;
  static constexpr int kElems = kTileKeys * D;
  __device__ __forceinline__ static int swz(int row) { return D == 128 ? 2 * (row & 7) : 2 * ((row >> 1) & 3); }
  __device__ __forceinline__ static int off(int row, int piece) { return row * D + 8 * (piece ^ swz(row)); }
};

// Issue this wave's RPW rows (RPW*wave .. RPW*wave + RPW-1) of two [64][D]
// matrices into `dst` (first matrix) and dst + kElems (second); rows r with
// r >= nvalid are filled from the zero block.
template <int D, int RPW>
__device__ __forceinline__ void load_pair_async(__bf16* dst, const __bf16* abase, const __bf16* bbase,
                                                int64_t row_stride, int nvalid, int wave, int lane) {
  using BT = BwdTile<D>;
  constexpr int kInstr = RPW * BT::kPieces / 64;
  static_assert(kInstr >= 1 && RPW * BT::kPieces == 64 * kInstr, "tile split");
  const __bf16* zero = reinterpret_cast<const __bf16*>(g_zero_rows) + 8 * (lane & 15);
  const uint32_t d0 = __builtin_amdgcn_readfirstlane(lds_addr(dst + wave * kInstr * 64 * 8));
  if (nvalid >= RPW) {
    // every row of this wave is in the sequence: uniform bases and per-lane
    // byte offsets that do not change from tile to tile
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      const int slot = (wave * kInstr + i) * 64 + lane;
      const int row = slot / BT::kPieces, piece = slot % BT::kPieces;
      const int r = row - RPW * wave;
      const uint32_t o = static_cast<uint32_t>((r * row_stride + 8 * (piece ^ BT::swz(row))) * 2);
      dma_b128_based(abase, o, d0 + i * 1024);
      dma_b128_based(bbase, o, d0 + i * 1024 + BT::kElems * 2);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < kInstr; ++i) {
    const int slot = (wave * kInstr + i) * 64 + lane;  // 16-byte LDS piece of the tile
    const int row = slot / BT::kPieces, piece = slot % BT::kPieces;
    const int r = row - RPW * wave;
    const bool ok = r < nvalid;
    const int lp = piece ^ BT::swz(row);  // logical piece held by this LDS piece
    const __bf16* as = ok ? abase + r * row_stride + 8 * lp : zero;
    const __bf16* bs = ok ? bbase + r * row_stride + 8 * lp : zero;
    dma_b128(as, d0 + i * 1024);
    dma_b128(bs, d0 + i * 1024 + BT::kElems * 2);
  }
}

// Transposed operand of a product that contracts over the 64 rows of a tile:
// lane i of 16-lane group g gets column 16*db + i and, for step st, rows
// 32*st + 16*h + 4*g + k in element 4*h + k (the row order pack_rows uses).
template <int D>
__device__ __forceinline__ void read_tr_operand(const __bf16* tile, int db, int lane, bf16x8 (&a)[2]) {
  using BT = BwdTile<D>;
  const int g = lane >> 4, src = lane & 15;
  const int row = 4 * g + (src >> 2);  // + 32*st + 16*h: bits 4-5, which the swizzle ignores
  const int sub = src & 3;
  const int piece = (2 * db + (sub >> 1)) ^ BT::swz(row);
  const __bf16* base = tile + row * D + 8 * piece + 4 * (sub & 1);
#pragma unroll
  for (int st = 0; st < 2; ++st) {
    const s16x4 lo = lds_read_tr16(base + (32 * st) * D);
    const s16x4 hi = lds_read_tr16(base + (32 * st + 16) * D);
    const s16x4 w[2] = {lo, hi};
    __builtin_memcpy(&a[st], w, sizeof(bf16x8));
  }
}

// Row-fragment operand: lane (g, i) gets row 16*blk + i, d = 32*st + 8*g .. +7.
template <int D>
__device__ __forceinline__ void read_row_operand(const __bf16* tile, int blk, int lane, bf16x8 (&a)[D / 32]) {
  using BT = BwdTile<D>;
  const int g = lane >> 4, row = 16 * blk + (lane & 15);
#pragma unroll
  for (int st = 0; st < D / 32; ++st) a[st] = *reinterpret_cast<const bf16x8*>(tile + BT::off(row, 4 * st + g));
}

// Values in the MFMA result layout of four 16-row blocks (x[blk][j] at row
// 16*blk + 4*g + j) -> the bf16 B operand of a product contracting over those
// 64 rows, in the order read_tr_operand delivers: step st, element e holds
// row 32*st + 16*(e/4) + 4*g + e%4.
__device__ __forceinline__ void pack_rows(const float (&x)[4][4], bf16x8 (&b)[2]) {
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int e = 0; e < 8; ++e) b[st][e] = to_bf16(x[2 * st + (e >> 2)][e & 3]);
}

struct BwdParams {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* out;
  const __bf16* dout;
  const float* lse;
  const int32_t* cu;
  float* ws_d;   // [Hq][T] D_i
  float* ws_l2;  // [Hq][T] lse_i * log2(e)
  __bf16* dq;
  __bf16* dk;
  __bf16* dv;
  int hq, hkv, group, total, num_seqs;
  float c, scale;
};

__device__ __forceinline__ void seq_range(const BwdParams& p, int seq, int& lo, int& L) {
  // clamp the (trusted) offsets so that a malformed table cannot index outside the tensors
  lo = min(max(p.cu[seq], 0), p.total);
  L = max(min(p.cu[seq + 1], p.total) - lo, 0);
}

// ---------------------------------------------------------------------------
// D_i = dO_i . O_i (fp32, lane-ordered partial sums then an xor butterfly) and
// lse_i * log2(e), for every (token, q head) row.  D/8 lanes per row.  Rows
// are enumerated head-major (r = h * T + t), the order of the two workspace
// planes, so consecutive rows write consecutive words (each row's out and
// dout reads are one 2*D-byte run either way).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdParams p) {
  constexpr int LPR = D / 8;
  constexpr int kRows = 256 / LPR;
  const int64_t rows = static_cast<int64_t>(p.total) * p.hq;
  const int64_t r = static_cast<int64_t>(blockIdx.x) * kRows + threadIdx.x / LPR;
  const int sub = threadIdx.x % LPR;
  int64_t row = 0;  // token-major index of (t, h) in out, dout and lse
  float acc = 0.f;
  if (r < rows) {
    const int h = static_cast<int>(r / p.total);
    const int64_t t = r % p.total;
    row = t * p.hq + h;
    const bf16x8 o = *reinterpret_cast<const bf16x8*>(p.out + row * D + 8 * sub);
    const bf16x8 d = *reinterpret_cast<const bf16x8*>(p.dout + row * D + 8 * sub);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = acc + static_cast<float>(o[e]) * static_cast<float>(d[e]);
  }
#pragma unroll
  for (int m = LPR / 2; m >= 1; m >>= 1) acc = acc + __shfl_xor(acc, m, LPR);
  if (r < rows && sub == 0) {
    p.ws_d[r] = acc;
    p.ws_l2[r] = p.lse[row] * 1.44269504088896340736f;
  }
}

// ---------------------------------------------------------------------------
// dK, dV
// ---------------------------------------------------------------------------
constexpr int kKvWaves = 4;
constexpr int kKeysPerWave = 32;
constexpr int kKeyTile = kKvWaves * kKeysPerWave;  // keys per workgroup
constexpr int kQTile = kTileKeys;                  // queries per step

template <int D>
__global__ __launch_bounds__(kKvWaves * 64, 1) void bwd_dkdv_kernel(BwdParams p) {
  using BT = BwdTile<D>;
  constexpr int NST = D / 32, NDB = D / 16;
  constexpr int kRpw = kQTile / kKvWaves;
  // a stage: the Q tile, the dO tile, then 4 x 64 floats (D, lse2, and copies)
  constexpr int kStageElems = 2 * BT::kElems + 512;
  __shared__ __attribute__((aligned(1024))) __bf16 lds[2 * kStageElems];

  const int per_kt = p.num_seqs * p.hkv;
  const int kt = blockIdx.x / per_kt;
  const int seq = (blockIdx.x % per_kt) / p.hkv;
  const int kvh = blockIdx.x % p.hkv;
  int lo, L;
  seq_range(p, seq, lo, L);
  const int k0 = kt * kKeyTile;
  if (k0 >= L) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int g = lane >> 4, col = lane & 15;
  const int kw0 = k0 + kKeysPerWave * wave;

  // B operands of this wave's keys: kf[nb][st] = K[kw0 + 16*nb + col][32*st + 8*g .. +7]
  bf16x8 kf[2][NST], vf[2][NST];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int kp = kw0 + 16 * nb + col;
    if (kp < L) {
      const int64_t off = (static_cast<int64_t>(lo + kp) * p.hkv + kvh) * D + 8 * g;
#pragma unroll
      for (int st = 0; st < NST; ++st) {
        kf[nb][st] = *reinterpret_cast<const bf16x8*>(p.k + off + 32 * st);
        vf[nb][st] = *reinterpret_cast<const bf16x8*>(p.v + off + 32 * st);
      }
    } else {
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          kf[nb][st][e] = static_cast<__bf16>(0.0f);
          vf[nb][st][e] = static_cast<__bf16>(0.0f);
        }
    }
  }

  const int nqt = (L + kQTile - 1) / kQTile;
  const int qt0 = k0 / kQTile;
  const int nq = nqt - qt0;  // >= 1 since k0 < L
  const int n = p.group * nq;
  const int64_t qstride = static_cast<int64_t>(p.hq) * D;
  const float* zero_f = reinterpret_cast<const float*>(g_zero_rows) + lane;

  auto issue = [&](int it) {
    const int head = kvh * p.group + it / nq;
    const int q0 = (qt0 + it % nq) * kQTile;
    __bf16* st = lds + (it & 1) * kStageElems;
    const int pos = q0 + kRpw * wave;
    const int64_t off = (static_cast<int64_t>(lo + pos) * p.hq + head) * D;
    load_pair_async<D, kRpw>(st, p.q + off, p.dout + off, qstride, L - pos, wave, lane);
    const float* plane = (wave & 1) ? p.ws_l2 : p.ws_d;
    const int qq = q0 + lane;
    const float* src = qq < L ? plane + static_cast<int64_t>(head) * p.total + lo + qq : zero_f;
    dma_b32(src, __builtin_amdgcn_readfirstlane(lds_addr(st + 2 * BT::kElems + 128 * wave)));
  };

  f32x4 dv_acc[NDB][2], dk_acc[NDB][2];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      dv_acc[db][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      dk_acc[db][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  const float c = p.c;

  issue(0);
  // the K/V operands (and stage 0) have landed; the compiler's own wait, so
  // that it does not keep those register loads pending into the loop, where
  // its waits would also cover the next stage's loads
  wait_vmem_below<0>();
  auto step = [&](int it, auto stage_const) {  // step it, in stage SI = it % 2
    constexpr int SI = decltype(stage_const)::value;
    // stage it has landed in every wave, and every wave is done with stage it-1
    wait_barrier<0>();
    if (it + 1 < n) issue(it + 1);
    const __bf16* qs = lds + SI * kStageElems;
    const __bf16* dos = qs + BT::kElems;
    const float* dvec = reinterpret_cast<const float*>(qs + 2 * BT::kElems);
    const float* lvec = dvec + 64;
    const int q0 = (qt0 + it % nq) * kQTile;

    // S = Q K^T and dP = dO V^T: rows = queries 16*qb + 4*g + j, column = key 16*nb + col
    f32x4 s[4][2], dp[4][2];
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      bf16x8 a[NST], b[NST];
      read_row_operand<D>(qs, qb, lane, a);
      read_row_operand<D>(dos, qb, lane, b);
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        f32x4 x = {0.f, 0.f, 0.f, 0.f}, y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < NST; ++st) x = mfma16(a[st], kf[nb][st], x);
#pragma unroll
        for (int st = 0; st < NST; ++st) y = mfma16(b[st], vf[nb][st], y);
        s[qb][nb] = x;
        dp[qb][nb] = y;
      }
    }

    // P and dS = P (dP - D); keys after the query, and rows past the
    // sequence, get P = 0
    const bool full = (q0 >= kw0 + kKeysPerWave - 1) && (q0 + kQTile <= L);  // wave-uniform
    float pv[2][4][4], dsv[2][4][4];
    auto weights = [&](auto masked) {
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) {
        const f32x4 l2 = *reinterpret_cast<const f32x4*>(lvec + 16 * qb + 4 * g);
        const f32x4 dd = *reinterpret_cast<const f32x4*>(dvec + 16 * qb + 4 * g);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            float x = hw_exp2(__builtin_fmaf(s[qb][nb][j], c, -l2[j]));
            if constexpr (decltype(masked)::value) {
              const int qp = q0 + 16 * qb + 4 * g + j;
              const int kp = kw0 + 16 * nb + col;
              x = (kp <= qp && qp < L) ? x : 0.f;
            }
            pv[nb][qb][j] = x;
            dsv[nb][qb][j] = x * (dp[qb][nb][j] - dd[j]);
          }
      }
    };
    if (full)
      weights(std::false_type{});
    else
      weights(std::true_type{});
    bf16x8 pb[2][2], sb[2][2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      pack_rows(pv[nb], pb[nb]);
      pack_rows(dsv[nb], sb[nb]);
    }

    // dV^T += dO^T P and dK^T += Q^T dS (contracting over the 64 queries)
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      bf16x8 ot[2], qtr[2];
      read_tr_operand<D>(dos, db, lane, ot);
      read_tr_operand<D>(qs, db, lane, qtr);
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
        for (int st = 0; st < 2; ++st) dv_acc[db][nb] = mfma16(ot[st], pb[nb][st], dv_acc[db][nb]);
#pragma unroll
        for (int st = 0; st < 2; ++st) dk_acc[db][nb] = mfma16(qtr[st], sb[nb][st], dk_acc[db][nb]);
      }
    }
  };
  // unrolled by the stage count: stage addresses are constant offsets
  for (int it = 0; it < n; it += 2) {
    step(it, std::integral_constant<int, 0>{});
    if (it + 1 < n) step(it + 1, std::integral_constant<int, 1>{});
  }

  // lane (g, col): key kw0 + 16*nb + col, d = 16*db + 4*g .. +3
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int kp = kw0 + 16 * nb + col;
    if (kp < L) {
      const int64_t off = (static_cast<int64_t>(lo + kp) * p.hkv + kvh) * D + 4 * g;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        bf16x4 wk, wv;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          wk[j] = to_bf16(dk_acc[db][nb][j] * p.scale);
          wv[j] = to_bf16(dv_acc[db][nb][j]);
        }
        *reinterpret_cast<bf16x4*>(p.dk + off + 16 * db) = wk;
        *reinterpret_cast<bf16x4*>(p.dv + off + 16 * db) = wv;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// dQ
// ---------------------------------------------------------------------------
constexpr int kDqWaves = 8;
constexpr int kDqNB = 2;
constexpr int kDqWaveRows = kDqNB * kQCols;
constexpr int kDqRows = kDqWaves * kDqWaveRows;

template <int D>
__global__ __launch_bounds__(kDqWaves * 64, 1) void bwd_dq_kernel(BwdParams p) {
  using BT = BwdTile<D>;
  constexpr int NST = D / 32, NDB = D / 16;
  constexpr int kRpw = kTileKeys / kDqWaves;
  constexpr int kStageElems = 2 * BT::kElems;  // K tile, V tile
  __shared__ __attribute__((aligned(1024))) __bf16 lds[2 * kStageElems];

  const int per_qt = p.num_seqs * p.hq;
  const int zrev = blockIdx.x / per_qt;  // query tiles counted from the end: longest work first
  const int seq = (blockIdx.x % per_qt) / p.hq;
  const int head = blockIdx.x % p.hq;
  const int kvh = head / p.group;
  int lo, L;
  seq_range(p, seq, lo, L);
  const int nqt = (L + kDqRows - 1) / kDqRows;
  const int qt = nqt - 1 - zrev;
  if (qt < 0) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int g = lane >> 4, col = lane & 15;
  const int q0 = qt * kDqRows + wave * kDqWaveRows;
  const bool wave_on = q0 < L;
  const int last_q0 = min(qt * kDqRows + kDqRows - kDqWaveRows, ((L - 1) / kDqWaveRows) * kDqWaveRows);
  const int wg_last_tile = last_q0 / kTileKeys;
  const int my_last_tile = q0 / kTileKeys;

  // B operands of this lane's query columns: qf[nb][st] = Q[q0 + 16*nb + col][32*st + 8*g .. +7]
  bf16x8 qf[kDqNB][NST], df[kDqNB][NST];
  float ddv[kDqNB], l2v[kDqNB];
#pragma unroll
  for (int nb = 0; nb < kDqNB; ++nb) {
    const int qp = q0 + kQCols * nb + col;
    if (wave_on && qp < L) {
      const int64_t row = static_cast<int64_t>(lo + qp) * p.hq + head;
#pragma unroll
      for (int st = 0; st < NST; ++st) {
        qf[nb][st] = *reinterpret_cast<const bf16x8*>(p.q + row * D + 8 * g + 32 * st);
        df[nb][st] = *reinterpret_cast<const bf16x8*>(p.dout + row * D + 8 * g + 32 * st);
      }
      const int64_t w = static_cast<int64_t>(head) * p.total + lo + qp;
      ddv[nb] = p.ws_d[w];
      l2v[nb] = p.ws_l2[w];
    } else {
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          qf[nb][st][e] = static_cast<__bf16>(0.0f);
          df[nb][st][e] = static_cast<__bf16>(0.0f);
        }
      ddv[nb] = 0.f;
      l2v[nb] = 0.f;
    }
  }

  const int64_t kstride = static_cast<int64_t>(p.hkv) * D;
  auto issue = [&](int t) {
    const int pos = t * kTileKeys + kRpw * wave;
    const int64_t off = (static_cast<int64_t>(lo + pos) * p.hkv + kvh) * D;
    load_pair_async<D, kRpw>(lds + (t & 1) * kStageElems, p.k + off, p.v + off, kstride, L - pos, wave, lane);
  };

  f32x4 acc[kDqNB][NDB];
#pragma unroll
  for (int nb = 0; nb < kDqNB; ++nb)
#pragma unroll
    for (int db = 0; db < NDB; ++db) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float c = p.c;

  issue(0);
  // the Q/dO operands, D and lse (and stage 0) have landed; see bwd_dkdv_kernel
  wait_vmem_below<0>();
  auto tile_step = [&](int t, auto stage_const) {  // tile t, in stage SI = t % 2
    constexpr int SI = decltype(stage_const)::value;
    wait_barrier<0>();
    if (t + 1 <= wg_last_tile) issue(t + 1);
    if (wave_on && t <= my_last_tile) {
      const __bf16* ks = lds + SI * kStageElems;
      const __bf16* vs = ks + BT::kElems;
      // S^T = K Q^T and dP^T = V dO^T: rows = keys 16*kb + 4*g + j, column = query 16*nb + col
      f32x4 s[kDqNB][4], dp[kDqNB][4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        bf16x8 a[NST], b[NST];
        read_row_operand<D>(ks, kb, lane, a);
        read_row_operand<D>(vs, kb, lane, b);
#pragma unroll
        for (int nb = 0; nb < kDqNB; ++nb) {
          f32x4 x = {0.f, 0.f, 0.f, 0.f}, y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int st = 0; st < NST; ++st) x = mfma16(a[st], qf[nb][st], x);
#pragma unroll
          for (int st = 0; st < NST; ++st) y = mfma16(b[st], df[nb][st], y);
          s[nb][kb] = x;
          dp[nb][kb] = y;
        }
      }
      bf16x8 sb[kDqNB][2];
      // only the diagonal tile holds keys after a query: their scores become
      // -inf there (a branch on the wave-uniform condition, not a select on
      // every tile), and exp2 turns them into P = +0, as the forward's mask
      if (t == my_last_tile) {
#pragma unroll
        for (int nb = 0; nb < kDqNB; ++nb) mask_scores(s[nb], t * kTileKeys, q0 + kQCols * nb + col, lane);
      }
#pragma unroll
      for (int nb = 0; nb < kDqNB; ++nb) {
        float dsv[4][4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float x = hw_exp2(__builtin_fmaf(s[nb][kb][j], c, -l2v[nb]));
            dsv[kb][j] = x * (dp[nb][kb][j] - ddv[nb]);
          }
        pack_rows(dsv, sb[nb]);
      }
      // dQ^T += K^T dS^T (contracting over the 64 keys)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        bf16x8 kt[2];
        read_tr_operand<D>(ks, db, lane, kt);
#pragma unroll
        for (int nb = 0; nb < kDqNB; ++nb)
#pragma unroll
          for (int st = 0; st < 2; ++st) acc[nb][db] = mfma16(kt[st], sb[nb][st], acc[nb][db]);
      }
    }
  };
  // unrolled by the stage count: stage addresses are constant offsets
  for (int t = 0; t <= wg_last_tile; t += 2) {
    tile_step(t, std::integral_constant<int, 0>{});
    if (t + 1 <= wg_last_tile) tile_step(t + 1, std::integral_constant<int, 1>{});
  }

#pragma unroll
  for (int nb = 0; nb < kDqNB; ++nb) {
    const int qp = q0 + kQCols * nb + col;
    if (wave_on && qp < L) {
      __bf16* row = p.dq + (static_cast<int64_t>(lo + qp) * p.hq + head) * D + 4 * g;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = to_bf16(acc[nb][db][j] * p.scale);
        *reinterpret_cast<bf16x4*>(row + 16 * db) = w;
      }
    }
  }
}

template <int D>
hipError_t launch_backward_d(const BwdParams& p, int max_seqlen, hipStream_t stream) {
  const int64_t rows = static_cast<int64_t>(p.total) * p.hq;
  constexpr int kPrepRows = 256 / (D / 8);
  const int64_t nprep = (rows + kPrepRows - 1) / kPrepRows;
  const int64_t nkv = (static_cast<int64_t>(max_seqlen) + kKeyTile - 1) / kKeyTile * p.num_seqs * p.hkv;
  const int64_t ndq = (static_cast<int64_t>(max_seqlen) + kDqRows - 1) / kDqRows * p.num_seqs * p.hq;
  if (nprep > 0x7FFFFFFF || nkv > 0x7FFFFFFF || ndq > 0x7FFFFFFF) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(bwd_prep_kernel<D>, dim3(static_cast<unsigned>(nprep)), dim3(256), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(bwd_dkdv_kernel<D>, dim3(static_cast<unsigned>(nkv)), dim3(kKvWaves * 64), 0, stream, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(bwd_dq_kernel<D>, dim3(static_cast<unsigned>(ndq)), dim3(kDqWaves * 64), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

size_t backward_ws_bytes(int64_t total_tokens, int64_t num_q_heads) {
  return static_cast<size_t>(2 * total_tokens * num_q_heads) * sizeof(float);
}

hipError_t launch_backward(const BackwardLaunch& a, hipStream_t stream) {
  BwdParams p;
  p.q = static_cast<const __bf16*>(a.q);
  p.k = static_cast<const __bf16*>(a.k);
  p.v = static_cast<const __bf16*>(a.v);
  p.out = static_cast<const __bf16*>(a.out);
  p.dout = static_cast<const __bf16*>(a.dout);
  p.lse = a.lse;
  p.cu = a.cu_seqlens;
  p.ws_d = static_cast<float*>(a.workspace);
  p.ws_l2 = p.ws_d + static_cast<int64_t>(a.total_tokens) * a.num_q_heads;
  p.dq = static_cast<__bf16*>(a.dq);
  p.dk = static_cast<__bf16*>(a.dk);
  p.dv = static_cast<__bf16*>(a.dv);
  p.hq = a.num_q_heads;
  p.hkv = a.num_kv_heads;
  p.group = a.num_q_heads / a.num_kv_heads;
  p.total = a.total_tokens;
  p.num_seqs = a.num_seqs;
  p.c = a.c;
  p.scale = a.scale;
  return a.head_dim == 128 ? launch_backward_d<128>(p, a.max_seqlen, stream)
                           : launch_backward_d<64>(p, a.max_seqlen, stream);
}

}  // namespace uattn
