// Internal launcher interface between the C-ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/uattn.h"

namespace uattn {

struct PrefillLaunch {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* cu_seqlens;
  void* out;
  float* lse;
  int32_t num_seqs;
  int32_t total_tokens;
  int32_t max_seqlen;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  float c;  // fp32(scale * log2(e))
};

struct DecodeLaunch {
  const void* q;
  const void* k_pages;
  const void* v_pages;
  const int32_t* block_table;
  const int32_t* seqlens;
  void* out;
  float* lse;
  float* ws_acc;  // [batch][Hq][decode_slots(nchunk_max)][head_dim]
  float* ws_ml;   // [batch][Hq][decode_slots(nchunk_max)][2]
  int32_t* ws_cnt; // [batch][Hkv] arrival counters
  int32_t batch;
  int32_t max_pages_per_seq;
  int32_t page_size;
  int32_t num_pages;
  int32_t max_seqlen;
  int32_t nchunk_max;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t num_cus;  // compute units of the current device (sizes the persistent grid)
  float c;
};

struct LogprobLaunch {
  const void* logits;
  int64_t row_stride;
  const int32_t* targets;
  float* logp;
  int32_t num_rows;
  int32_t vocab;
  float inv_temperature;
};

struct KvWriteLaunch {
  const void* k_new;
  const void* v_new;
  int64_t token_stride;
  const int32_t* block_table;
  const int32_t* seq_idx;
  const int32_t* positions;
  void* k_pages;
  void* v_pages;
  int32_t num_tokens, batch, max_pages_per_seq, page_size, num_pages, num_kv_heads, head_dim;
};

hipError_t launch_kv_write(const KvWriteLaunch& a, hipStream_t stream);

struct NormRopeLaunch {
  const void* q;
  const void* k;
  const int32_t* positions;
  const void* q_weight;
  const void* k_weight;
  const float* cos_sin;
  void* q_out;
  void* k_out;
  float eps;
  int32_t max_position, num_tokens, num_q_heads, num_kv_heads, head_dim;
};

hipError_t launch_qk_norm_rope(const NormRopeLaunch& a, hipStream_t stream);
hipError_t launch_rope_cache(float* cos_sin, int32_t max_position, int32_t head_dim, double theta, hipStream_t stream);

struct LmHeadLaunch {
  const void* hidden;
  int64_t hidden_stride;
  const void* weight;
  int64_t weight_stride;
  void* logits;
  int64_t logits_stride;
  int32_t num_rows, vocab, hidden_dim;
};

hipError_t launch_lm_head(const LmHeadLaunch& a, hipStream_t stream);
// LM head with the fused log-probability epilogue (a.logits may be nullptr):
// partials in `workspace` (lm_head_logprob_ws_bytes), then their fold into logp.
hipError_t launch_lm_head_logprob(const LmHeadLaunch& a, const int32_t* targets, float inv_temperature, float* logp,
                                  void* workspace, hipStream_t stream);
size_t lm_head_logprob_ws_bytes(int64_t num_rows, int64_t vocab);

struct BackwardLaunch {
  const void* q;
  const void* k;
  const void* v;
  const void* out;
  const void* dout;
  const float* lse;
  const int32_t* cu_seqlens;
  void* dq;
  void* dk;
  void* dv;
  void* workspace;  // backward_ws_bytes(total_tokens, num_q_heads)
  int32_t num_seqs, total_tokens, max_seqlen, num_q_heads, num_kv_heads, head_dim;
  float c;      // fp32(scale * log2(e))
  float scale;  // softmax scale
};

hipError_t launch_backward(const BackwardLaunch& a, hipStream_t stream);
size_t backward_ws_bytes(int64_t total_tokens, int64_t num_q_heads);

// Compute units of the current device (cached per device; 256 if the query fails).
int32_t device_cus();

// Each returns hipSuccess or the launch error.
hipError_t launch_prefill(const PrefillLaunch& a, hipStream_t stream);
hipError_t launch_decode(const DecodeLaunch& a, hipStream_t stream);
hipError_t launch_logprob(const LogprobLaunch& a, hipStream_t stream);

// Checks uattn_decode's arguments (every rule of uattn.h) and fills the launch
// record, laying the workspace out as counters at its start and partials at
// its end.  Returns the status uattn_decode reports; `launch->batch` is 0
// when there is nothing to launch.
uattn_status decode_prepare(const void* q, const void* k_pages, const void* v_pages, const int32_t* block_table,
                            const int32_t* seqlens, int32_t batch, int32_t max_pages_per_seq, int32_t page_size,
                            int32_t num_pages, int32_t max_seqlen, int32_t num_q_heads, int32_t num_kv_heads,
                            int32_t head_dim, float softmax_scale, void* out, float* lse, void* workspace,
                            size_t workspace_bytes, DecodeLaunch* launch);

// Decode workspace: arrival counters at the start (kept zero between calls),
// the fp32 partials (acc, then m/l) at the end of the caller's buffer.
// Partial slots per (entry, q head) for nchunk chunks: rounded up to even, so
// that the (m, l) pairs of two consecutive chunks are one 16-byte load.
int64_t decode_slots(int64_t nchunk);
size_t decode_ws_acc_bytes(int64_t batch, int64_t nchunk, int64_t num_q_heads, int64_t head_dim);
size_t decode_ws_ml_bytes(int64_t batch, int64_t nchunk, int64_t num_q_heads);
size_t decode_ws_cnt_bytes(int64_t batch, int64_t num_q_heads);

}  // namespace uattn
