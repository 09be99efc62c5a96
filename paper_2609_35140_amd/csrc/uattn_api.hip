// extern "C" boundary of libuattn: argument validation, grid sizing and
// launch on the caller's stream.  No allocation, no synchronization (except
// the opt-in UATTN_VALIDATE debug copies), no global mutable state.
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../../include/uattn.h"
#include "uattn_internal.h"
#include "uattn_numerics.h"

namespace {

using uattn::kChunkKeys;

constexpr double kLog2e = 1.4426950408889634;

bool scale_ok(float s) { return s > 0.f && s < __builtin_inff(); }

bool validate_env() {
  const char* e = getenv("UATTN_VALIDATE");
  return e != nullptr && e[0] != '\0' && e[0] != '0';
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// fp32(scale * log2(e)), the one constant both attention paths fold into exp2.
float exp2_scale(float softmax_scale) { return static_cast<float>(static_cast<double>(softmax_scale) * kLog2e); }

template <class T>
bool copy_back(std::vector<T>& host, const T* dev, size_t n) {
  host.resize(n);
  if (n == 0) return true;
  return hipMemcpy(host.data(), dev, n * sizeof(T), hipMemcpyDeviceToHost) == hipSuccess;
}

}  // namespace

namespace uattn {
int32_t device_cus() {
  static int32_t cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] > 0) return cached[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  cached[dev] = n;
  return n;
}
}  // namespace uattn

extern "C" {

int32_t uattn_abi_version(void) { return UATTN_ABI_VERSION; }

const char* uattn_status_string(int32_t status) {
  switch (status) {
    case UATTN_OK: return "UATTN_OK";
    case UATTN_EINVAL: return "UATTN_EINVAL: invalid argument";
    case UATTN_EUNSUPPORTED: return "UATTN_EUNSUPPORTED: unsupported shape";
    case UATTN_EWORKSPACE: return "UATTN_EWORKSPACE: workspace missing or too small";
    case UATTN_ELAUNCH: return "UATTN_ELAUNCH: kernel launch failed";
    case UATTN_ESCRATCH: return "UATTN_ESCRATCH: these sizes need more decode scratch than the library's static array holds";
    default: return "UATTN_UNKNOWN_STATUS";
  }
}

uattn_status uattn_prefill(const void* q, const void* k, const void* v, const int32_t* cu_seqlens, int32_t num_seqs,
                           int32_t total_tokens, int32_t max_seqlen, int32_t num_q_heads, int32_t num_kv_heads,
                           int32_t head_dim, float softmax_scale, void* out, float* lse, void* stream) {
  if (num_seqs < 0 || total_tokens < 0 || max_seqlen < 0 || num_q_heads <= 0 || num_kv_heads <= 0)
    return UATTN_EINVAL;
  if (num_q_heads % num_kv_heads != 0 || !scale_ok(softmax_scale)) return UATTN_EINVAL;
  if (head_dim != 64 && head_dim != 128) return UATTN_EUNSUPPORTED;
  if (num_seqs > 65535) return UATTN_EUNSUPPORTED;
  if (num_seqs == 0 || total_tokens == 0 || max_seqlen == 0) return UATTN_OK;
  if (!q || !k || !v || !cu_seqlens || !out) return UATTN_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out)) return UATTN_EINVAL;
  if (validate_env()) {
    std::vector<int32_t> cu;
    if (!copy_back(cu, cu_seqlens, static_cast<size_t>(num_seqs) + 1)) return UATTN_EINVAL;
    if (cu[0] != 0 || cu[num_seqs] != total_tokens) return UATTN_EINVAL;
    for (int32_t s = 0; s < num_seqs; ++s) {
      const int32_t len = cu[s + 1] - cu[s];
      if (len < 0 || len > max_seqlen) return UATTN_EINVAL;
    }
  }
  uattn::PrefillLaunch a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.cu_seqlens = cu_seqlens;
  a.out = out;
  a.lse = lse;
  a.num_seqs = num_seqs;
  a.total_tokens = total_tokens;
  a.max_seqlen = max_seqlen;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.c = exp2_scale(softmax_scale);
  return uattn::launch_prefill(a, static_cast<hipStream_t>(stream)) == hipSuccess ? UATTN_OK : UATTN_ELAUNCH;
}

size_t uattn_decode_workspace_bytes(int32_t batch, int32_t max_seqlen, int32_t num_q_heads, int32_t head_dim) {
  if (batch <= 0 || max_seqlen <= 0 || num_q_heads <= 0 || head_dim <= 0) return 0;
  const int64_t nchunk = (static_cast<int64_t>(max_seqlen) + kChunkKeys - 1) / kChunkKeys;
  if (nchunk <= 1) return 0;
  return uattn::decode_ws_cnt_bytes(batch, num_q_heads) +
         uattn::decode_ws_acc_bytes(batch, nchunk, num_q_heads, head_dim) +
         uattn::decode_ws_ml_bytes(batch, nchunk, num_q_heads);
}

}  // extern "C"

namespace uattn {
uattn_status decode_prepare(const void* q, const void* k_pages, const void* v_pages, const int32_t* block_table,
                            const int32_t* seqlens, int32_t batch, int32_t max_pages_per_seq, int32_t page_size,
                            int32_t num_pages, int32_t max_seqlen, int32_t num_q_heads, int32_t num_kv_heads,
                            int32_t head_dim, float softmax_scale, void* out, float* lse, void* workspace,
                            size_t workspace_bytes, DecodeLaunch* launch) {
  if (batch < 0 || max_pages_per_seq < 0 || max_seqlen < 0 || num_pages < 0 || num_q_heads <= 0 ||
      num_kv_heads <= 0)
    return UATTN_EINVAL;
  if (num_q_heads % num_kv_heads != 0 || !scale_ok(softmax_scale)) return UATTN_EINVAL;
  if (head_dim != 64 && head_dim != 128) return UATTN_EUNSUPPORTED;
  if (page_size < 16 || (page_size & (page_size - 1)) != 0) return UATTN_EUNSUPPORTED;
  if (num_q_heads / num_kv_heads > uattn::kMaxGroup) return UATTN_EUNSUPPORTED;
  if (batch > 65535 || num_kv_heads > 65535) return UATTN_EUNSUPPORTED;
  if (max_seqlen > (1 << 24)) return UATTN_EUNSUPPORTED;  // keeps every 32-bit workspace offset in range
  if (batch == 0) {
    launch->batch = 0;
    return UATTN_OK;
  }
  if (max_seqlen == 0 || num_pages == 0) return UATTN_EINVAL;  // every entry holds at least its own token
  if (static_cast<int64_t>(max_pages_per_seq) * page_size < max_seqlen) return UATTN_EINVAL;
  if (!q || !k_pages || !v_pages || !block_table || !seqlens || !out) return UATTN_EINVAL;
  if (!aligned16(q) || !aligned16(k_pages) || !aligned16(v_pages) || !aligned16(out)) return UATTN_EINVAL;
  const size_t need = uattn_decode_workspace_bytes(batch, max_seqlen, num_q_heads, head_dim);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need || !aligned16(workspace))) return UATTN_EWORKSPACE;
  const int64_t nchunk = (static_cast<int64_t>(max_seqlen) + kChunkKeys - 1) / kChunkKeys;
  if (validate_env()) {
    std::vector<int32_t> sl, bt;
    if (!copy_back(sl, seqlens, static_cast<size_t>(batch))) return UATTN_EINVAL;
    if (!copy_back(bt, block_table, static_cast<size_t>(batch) * max_pages_per_seq)) return UATTN_EINVAL;
    for (int32_t b = 0; b < batch; ++b) {
      if (sl[b] < 1 || sl[b] > max_seqlen) return UATTN_EINVAL;
      const int32_t used = (sl[b] + page_size - 1) / page_size;
      for (int32_t j = 0; j < used; ++j)
        if (bt[static_cast<size_t>(b) * max_pages_per_seq + j] < 0 ||
            bt[static_cast<size_t>(b) * max_pages_per_seq + j] >= num_pages)
          return UATTN_EINVAL;
    }
  }
  DecodeLaunch a;
  a.q = q;
  a.k_pages = k_pages;
  a.v_pages = v_pages;
  a.block_table = block_table;
  a.seqlens = seqlens;
  a.out = out;
  a.lse = lse;
  // counters at the start, partials at the end of the caller's buffer: a
  // workspace sized for one call can be reused by any call it is large enough for
  // without a partial region ever covering a counter that a later call relies on
  // being zero (see the zero-fill rule in uattn.h)
  if (need > 0) {
    const size_t acc_b = uattn::decode_ws_acc_bytes(batch, nchunk, num_q_heads, head_dim);
    const size_t ml_b = uattn::decode_ws_ml_bytes(batch, nchunk, num_q_heads);
    char* end = static_cast<char*>(workspace) + (workspace_bytes & ~static_cast<size_t>(15));
    a.ws_cnt = static_cast<int32_t*>(workspace);
    a.ws_ml = reinterpret_cast<float*>(end - ml_b);
    a.ws_acc = reinterpret_cast<float*>(end - ml_b - acc_b);
  } else {
    a.ws_cnt = nullptr;
    a.ws_ml = nullptr;
    a.ws_acc = nullptr;
  }
  a.batch = batch;
  a.max_pages_per_seq = max_pages_per_seq;
  a.page_size = page_size;
  a.num_pages = num_pages;
  a.max_seqlen = max_seqlen;
  a.nchunk_max = static_cast<int32_t>(nchunk);
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.num_cus = uattn::device_cus();
  a.c = exp2_scale(softmax_scale);
  *launch = a;
  return UATTN_OK;
}
}  // namespace uattn

extern "C" {

uattn_status uattn_decode(const void* q, const void* k_pages, const void* v_pages, const int32_t* block_table,
                          const int32_t* seqlens, int32_t batch, int32_t max_pages_per_seq, int32_t page_size,
                          int32_t num_pages, int32_t max_seqlen, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                          float softmax_scale, void* out, float* lse, void* workspace, size_t workspace_bytes,
                          void* stream) {
  uattn::DecodeLaunch a;
  const uattn_status st =
      uattn::decode_prepare(q, k_pages, v_pages, block_table, seqlens, batch, max_pages_per_seq, page_size, num_pages,
                            max_seqlen, num_q_heads, num_kv_heads, head_dim, softmax_scale, out, lse, workspace,
                            workspace_bytes, &a);
  if (st != UATTN_OK || a.batch == 0) return st;
  return uattn::launch_decode(a, static_cast<hipStream_t>(stream)) == hipSuccess ? UATTN_OK : UATTN_ELAUNCH;
}

uattn_status uattn_logprob(const void* logits, int64_t row_stride, const int32_t* targets, int32_t num_rows,
                           int32_t vocab, float inv_temperature, float* logp, void* stream) {
  if (num_rows < 0 || vocab <= 0 || row_stride < vocab || !scale_ok(inv_temperature)) return UATTN_EINVAL;
  if (num_rows == 0) return UATTN_OK;
  if (!logits || !targets || !logp) return UATTN_EINVAL;
  if (!aligned16(logits) || (row_stride % 8) != 0) return UATTN_EINVAL;
  if (validate_env()) {
    std::vector<int32_t> tg;
    if (!copy_back(tg, targets, static_cast<size_t>(num_rows))) return UATTN_EINVAL;
    for (int32_t t : tg)
      if (t < 0 || t >= vocab) return UATTN_EINVAL;
  }
  uattn::LogprobLaunch a;
  a.logits = logits;
  a.row_stride = row_stride;
  a.targets = targets;
  a.logp = logp;
  a.num_rows = num_rows;
  a.vocab = vocab;
  a.inv_temperature = inv_temperature;
  return uattn::launch_logprob(a, static_cast<hipStream_t>(stream)) == hipSuccess ? UATTN_OK : UATTN_ELAUNCH;
}

uattn_status uattn_kv_write(const void* k_new, const void* v_new, int64_t token_stride, const int32_t* block_table,
                            const int32_t* seq_idx, const int32_t* positions, int32_t num_tokens, int32_t batch,
                            int32_t max_pages_per_seq, int32_t page_size, int32_t num_pages, int32_t num_kv_heads,
                            int32_t head_dim, void* k_pages, void* v_pages, void* stream) {
  if (num_tokens < 0 || batch < 0 || max_pages_per_seq < 0 || num_pages < 0 || num_kv_heads <= 0) return UATTN_EINVAL;
  if (head_dim != 64 && head_dim != 128) return UATTN_EUNSUPPORTED;
  if (page_size < 16 || (page_size & (page_size - 1)) != 0) return UATTN_EUNSUPPORTED;
  if (token_stride < static_cast<int64_t>(num_kv_heads) * head_dim || (token_stride % 8) != 0) return UATTN_EINVAL;
  if (num_tokens == 0 || batch == 0 || max_pages_per_seq == 0 || num_pages == 0) return UATTN_OK;
  if (!k_new || !v_new || !block_table || !seq_idx || !positions || !k_pages || !v_pages) return UATTN_EINVAL;
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pages) || !aligned16(v_pages)) return UATTN_EINVAL;
  if (validate_env()) {
    std::vector<int32_t> si, ps, bt;
    if (!copy_back(si, seq_idx, static_cast<size_t>(num_tokens)) ||
        !copy_back(ps, positions, static_cast<size_t>(num_tokens)) ||
        !copy_back(bt, block_table, static_cast<size_t>(batch) * max_pages_per_seq))
      return UATTN_EINVAL;
    for (int32_t n = 0; n < num_tokens; ++n) {
      if (ps[n] < 0) continue;
      if (si[n] < 0 || si[n] >= batch || ps[n] / page_size >= max_pages_per_seq) return UATTN_EINVAL;
      const int32_t pg = bt[static_cast<size_t>(si[n]) * max_pages_per_seq + ps[n] / page_size];
      if (pg < 0 || pg >= num_pages) return UATTN_EINVAL;
    }
  }
  uattn::KvWriteLaunch a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.token_stride = token_stride;
  a.block_table = block_table;
  a.seq_idx = seq_idx;
  a.positions = positions;
  a.k_pages = k_pages;
  a.v_pages = v_pages;
  a.num_tokens = num_tokens;
  a.batch = batch;
  a.max_pages_per_seq = max_pages_per_seq;
  a.page_size = page_size;
  a.num_pages = num_pages;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  return uattn::launch_kv_write(a, static_cast<hipStream_t>(stream)) == hipSuccess ? UATTN_OK : UATTN_ELAUNCH;
}

uattn_status uattn_qk_norm_rope(const void* q, const void* k, const int32_t* positions, const void* q_weight,
                                const void* k_weight, float eps, const float* cos_sin, int32_t max_position,
                                int32_t num_tokens, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                void* q_out, void* k_out, void* stream) {
  if (num_tokens < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || max_position <= 0) return UATTN_EINVAL;
  if (!(eps >= 0.f) || !(eps < __builtin_inff())) return UATTN_EINVAL;
  if (head_dim != 64 && head_dim != 128) return UATTN_EUNSUPPORTED;
  if (num_tokens == 0) return UATTN_OK;
  if (!q || !k || !positions || !q_weight || !k_weight || !cos_sin || !q_out || !k_out) return UATTN_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(q_out) || !aligned16(k_out) || !aligned16(cos_sin) ||
      !aligned16(q_weight) || !aligned16(k_weight))
    return UATTN_EINVAL;
  uattn::NormRopeLaunch a;
  a.q = q;
  a.k = k;
  a.positions = positions;
  a.q_weight = q_weight;
  a.k_weight = k_weight;
  a.cos_sin = cos_sin;
  a.q_out = q_out;
  a.k_out = k_out;
  a.eps = eps;
  a.max_position = max_position;
  a.num_tokens = num_tokens;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  return uattn::launch_qk_norm_rope(a, static_cast<hipStream_t>(stream)) == hipSuccess ? UATTN_OK : UATTN_ELAUNCH;
}

uattn_status uattn_rope_cache(float* cos_sin, int32_t max_position, int32_t head_dim, double theta, void* stream) {
  if (max_position < 0 || !(theta > 1.0) || !(theta < 1e300)) return UATTN_EINVAL;
  if (head_dim != 64 && head_dim != 128) return UATTN_EUNSUPPORTED;
  if (max_position == 0) return UATTN_OK;
  if (!cos_sin || !aligned16(cos_sin)) return UATTN_EINVAL;
  return uattn::launch_rope_cache(cos_sin, max_position, head_dim, theta, static_cast<hipStream_t>(stream)) ==
                 hipSuccess
             ? UATTN_OK
             : UATTN_ELAUNCH;
}

uattn_status uattn_lm_head(const void* hidden, int64_t hidden_stride, const void* weight, int64_t weight_stride,
                           int32_t num_rows, int32_t vocab, int32_t hidden_dim, void* logits, int64_t logits_stride,
                           void* stream) {
  if (num_rows < 0 || vocab < 0 || hidden_dim <= 0 || (hidden_dim % 64) != 0) return UATTN_EINVAL;
  if (hidden_stride < hidden_dim || weight_stride < hidden_dim || logits_stride < vocab) return UATTN_EINVAL;
  if ((hidden_stride % 8) != 0 || (weight_stride % 8) != 0 || (logits_stride % 8) != 0) return UATTN_EINVAL;
  if (num_rows == 0 || vocab == 0) return UATTN_OK;
  if (!hidden || !weight || !logits) return UATTN_EINVAL;
  if (!aligned16(hidden) || !aligned16(weight) || !aligned16(logits)) return UATTN_EINVAL;
  uattn::LmHeadLaunch a;
  a.hidden = hidden;
  a.hidden_stride = hidden_stride;
  a.weight = weight;
  a.weight_stride = weight_stride;
  a.logits = logits;
  a.logits_stride = logits_stride;
  a.num_rows = num_rows;
  a.vocab = vocab;
  a.hidden_dim = hidden_dim;
  return uattn::launch_lm_head(a, static_cast<hipStream_t>(stream)) == hipSuccess ? UATTN_OK : UATTN_ELAUNCH;
}

size_t uattn_lm_head_logprob_workspace_bytes(int32_t num_rows, int32_t vocab) {
  if (num_rows <= 0 || vocab <= 0) return 0;
  return uattn::lm_head_logprob_ws_bytes(num_rows, vocab);
}

uattn_status uattn_lm_head_logprob(const void* hidden, int64_t hidden_stride, const void* weight,
                                   int64_t weight_stride, const int32_t* targets, int32_t num_rows, int32_t vocab,
                                   int32_t hidden_dim, float inv_temperature, float* logp, void* logits,
                                   int64_t logits_stride, void* workspace, size_t workspace_bytes, void* stream) {
  if (num_rows < 0 || vocab < 0 || hidden_dim <= 0 || (hidden_dim % 64) != 0) return UATTN_EINVAL;
  if (hidden_stride < hidden_dim || weight_stride < hidden_dim) return UATTN_EINVAL;
  if ((hidden_stride % 8) != 0 || (weight_stride % 8) != 0) return UATTN_EINVAL;
  if (logits != nullptr && (logits_stride < vocab || (logits_stride % 8) != 0 || !aligned16(logits)))
    return UATTN_EINVAL;
  if (!scale_ok(inv_temperature)) return UATTN_EINVAL;
  if (num_rows == 0) return UATTN_OK;
  if (vocab == 0) return UATTN_EINVAL;  // log-softmax over an empty vocabulary
  if (!hidden || !weight || !targets || !logp) return UATTN_EINVAL;
  if (!aligned16(hidden) || !aligned16(weight)) return UATTN_EINVAL;
  const size_t need = uattn_lm_head_logprob_workspace_bytes(num_rows, vocab);
  if (workspace == nullptr || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 3u) != 0)
    return UATTN_EWORKSPACE;
  if (validate_env()) {
    std::vector<int32_t> tg;
    if (!copy_back(tg, targets, static_cast<size_t>(num_rows))) return UATTN_EINVAL;
    for (int32_t t : tg)
      if (t < 0 || t >= vocab) return UATTN_EINVAL;
  }
  uattn::LmHeadLaunch a;
  a.hidden = hidden;
  a.hidden_stride = hidden_stride;
  a.weight = weight;
  a.weight_stride = weight_stride;
  a.logits = logits;
  a.logits_stride = logits != nullptr ? logits_stride : 0;
  a.num_rows = num_rows;
  a.vocab = vocab;
  a.hidden_dim = hidden_dim;
  return uattn::launch_lm_head_logprob(a, targets, inv_temperature, logp, workspace,
                                       static_cast<hipStream_t>(stream)) == hipSuccess
             ? UATTN_OK
             : UATTN_ELAUNCH;
}

size_t uattn_prefill_backward_workspace_bytes(int32_t total_tokens, int32_t num_q_heads) {
  if (total_tokens <= 0 || num_q_heads <= 0) return 0;
  return uattn::backward_ws_bytes(total_tokens, num_q_heads);
}

uattn_status uattn_prefill_backward(const void* q, const void* k, const void* v, const void* out, const void* dout,
                                    const float* lse, const int32_t* cu_seqlens, int32_t num_seqs,
                                    int32_t total_tokens, int32_t max_seqlen, int32_t num_q_heads,
                                    int32_t num_kv_heads, int32_t head_dim, float softmax_scale, void* dq, void* dk,
                                    void* dv, void* workspace, size_t workspace_bytes, void* stream) {
  if (num_seqs < 0 || total_tokens < 0 || max_seqlen < 0 || num_q_heads <= 0 || num_kv_heads <= 0)
    return UATTN_EINVAL;
  if (num_q_heads % num_kv_heads != 0 || !scale_ok(softmax_scale)) return UATTN_EINVAL;
  if (head_dim != 64 && head_dim != 128) return UATTN_EUNSUPPORTED;
  if (num_seqs > 65535) return UATTN_EUNSUPPORTED;
  if (num_seqs == 0 || total_tokens == 0 || max_seqlen == 0) return UATTN_OK;
  if (!q || !k || !v || !out || !dout || !lse || !cu_seqlens || !dq || !dk || !dv) return UATTN_EINVAL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) || !aligned16(dout) || !aligned16(dq) ||
      !aligned16(dk) || !aligned16(dv) || (reinterpret_cast<uintptr_t>(lse) & 3u) != 0)
    return UATTN_EINVAL;
  const size_t need = uattn_prefill_backward_workspace_bytes(total_tokens, num_q_heads);
  if (workspace == nullptr || workspace_bytes < need || !aligned16(workspace)) return UATTN_EWORKSPACE;
  if (validate_env()) {
    std::vector<int32_t> cu;
    if (!copy_back(cu, cu_seqlens, static_cast<size_t>(num_seqs) + 1)) return UATTN_EINVAL;
    if (cu[0] != 0 || cu[num_seqs] != total_tokens) return UATTN_EINVAL;
    for (int32_t s = 0; s < num_seqs; ++s) {
      const int32_t len = cu[s + 1] - cu[s];
      if (len < 0 || len > max_seqlen) return UATTN_EINVAL;
    }
  }
  uattn::BackwardLaunch a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.dout = dout;
  a.lse = lse;
  a.cu_seqlens = cu_seqlens;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.workspace = workspace;
  a.num_seqs = num_seqs;
  a.total_tokens = total_tokens;
  a.max_seqlen = max_seqlen;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.c = exp2_scale(softmax_scale);
  a.scale = softmax_scale;
  return uattn::launch_backward(a, static_cast<hipStream_t>(stream)) == hipSuccess ? UATTN_OK : UATTN_ELAUNCH;
}

}  // extern "C"
