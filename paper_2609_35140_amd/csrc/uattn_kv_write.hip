// Indexed write of new K/V rows into the paged cache.
//
// A pure copy: every 16-byte piece of a token's row of one kv head goes to
// the same offset of its (page, head, slot) row in k_pages and v_pages.
// One workgroup per token, consecutive threads on consecutive pieces of a
// row, then heads, so both the reads (token rows, heads contiguous) and the
// writes (one 128- or 256-byte row per (token, head)) are full coalesced
// segments; the token's destination page is looked up once.  Destinations come only from device integers that are
// checked against the table and pool bounds; a token that fails a check is
// skipped, never clamped onto another slot.
#include "uattn_internal.h"

namespace uattn {
namespace {

struct KvWriteParams {
  const uint4* k_new;
  const uint4* v_new;
  int64_t token_stride16;  // in 16-byte pieces
  const int32_t* bt;
  const int32_t* seq_idx;
  const int32_t* positions;
  uint4* kp;
  uint4* vp;
  int32_t num_tokens, batch, maxp, page_size, num_pages, hkv, pieces;  // pieces = head_dim / 8
};

// One workgroup per token; its threads copy the token's 16-byte pieces
// (heads x pieces per head), all from one workgroup-uniform destination page.
__global__ __launch_bounds__(256) void kv_write_kernel(KvWriteParams p) {
  const int per_token = p.hkv * p.pieces;
  for (int64_t n = blockIdx.x; n < p.num_tokens; n += gridDim.x) {
    const int32_t pos = p.positions[n];
    const int32_t s = p.seq_idx[n];
    if (pos < 0 || s < 0 || s >= p.batch) continue;
    const int32_t lp = pos / p.page_size;
    if (lp >= p.maxp) continue;
    const int32_t page = p.bt[static_cast<int64_t>(s) * p.maxp + lp];
    if (page < 0 || page >= p.num_pages) continue;
    const int64_t src0 = n * p.token_stride16;
    const int64_t dst0 = (static_cast<int64_t>(page) * p.hkv * p.page_size + (pos % p.page_size)) * p.pieces;
    for (int i = threadIdx.x; i < per_token; i += blockDim.x) {
      const int h = i / p.pieces, c = i % p.pieces;
      const int64_t src = src0 + static_cast<int64_t>(h) * p.pieces + c;
      const int64_t dst = dst0 + static_cast<int64_t>(h) * p.page_size * p.pieces + c;
      const uint4 kv = p.k_new[src];
      const uint4 vv = p.v_new[src];
      p.kp[dst] = kv;
      p.vp[dst] = vv;
    }
  }
}

}  // namespace

hipError_t launch_kv_write(const KvWriteLaunch& a, hipStream_t stream) {
  KvWriteParams p;
  p.k_new = static_cast<const uint4*>(a.k_new);
  p.v_new = static_cast<const uint4*>(a.v_new);
  p.token_stride16 = a.token_stride / 8;
  p.bt = a.block_table;
  p.seq_idx = a.seq_idx;
  p.positions = a.positions;
  p.kp = static_cast<uint4*>(a.k_pages);
  p.vp = static_cast<uint4*>(a.v_pages);
  p.num_tokens = a.num_tokens;
  p.batch = a.batch;
  p.maxp = a.max_pages_per_seq;
  p.page_size = a.page_size;
  p.num_pages = a.num_pages;
  p.hkv = a.num_kv_heads;
  p.pieces = a.head_dim / 8;
  // one workgroup per token, sized to its pieces (a multiple of the wave)
  const int per_token = a.num_kv_heads * p.pieces;
  const int threads = per_token >= 256 ? 256 : (per_token + 63) / 64 * 64;
  const dim3 grid(static_cast<unsigned>(a.num_tokens));
  const dim3 block(static_cast<unsigned>(threads));
  hipLaunchKernelGGL(kv_write_kernel, grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace uattn
