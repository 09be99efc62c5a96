/*
 * uattn -- unified, batch-invariant causal GQA attention for MI355X (gfx950).
 *
 * C ABI of libuattn.so.  Two entry points compute the same attention for
 * the two execution regimes the paper couples (Section 1 and Section 4.1):
 *
 *   uattn_prefill  -- the full-sequence entry point, used by the policy
 *                     update over whole prompt+response trajectories and by
 *                     rollout prefill over prompts;
 *   uattn_decode   -- the token-wise decode entry point, one new query per
 *                     sequence against a paged KV cache.
 *
 * For the same token, query, causal KV prefix and weights, the two return
 * bit-identical outputs (the operator-level form of Eq. (1), Section 3.2),
 * independent of batch size, batch order, max_seqlen and how decode splits
 * its work.  uattn_logprob is the per-token log-softmax gather whose equality
 * across the two regimes makes the reuse ratio exp(l_upd - l_roll) exactly 1
 * (Section 3.1).
 *
 * Conventions shared by every call:
 *   - every pointer argument is a DEVICE pointer unless stated otherwise;
 *   - bf16 tensors are raw 16-bit bfloat16 values, row-major, contiguous;
 *   - the caller owns every buffer; the library never allocates, frees or
 *     synchronizes; each call enqueues kernels on `stream` (a hipStream_t,
 *     NULL for the default stream) and returns;
 *   - outputs must not alias inputs;
 *   - integer data that lives on the device (cu_seqlens, seqlens,
 *     block_table, targets) is trusted: it is not read by the host.  Setting
 *     the environment variable UATTN_VALIDATE=1 makes the host copy it back
 *     (synchronously) and check it before launching, for debugging;
 *   - errors are reported by the return code only; nothing is printed and
 *     nothing aborts.  On any non-OK code no kernel was launched, except
 *     UATTN_ELAUNCH, which reports a failure of the launch itself.
 */
#ifndef UATTN_H
#define UATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define UATTN_ABI_VERSION 1

typedef enum {
  UATTN_OK = 0,
  UATTN_EINVAL = 1,       /* null pointer, negative or inconsistent sizes, Hq % Hkv != 0, bad scale */
  UATTN_EUNSUPPORTED = 2, /* head_dim not 64/128, page_size not a power of two >= 16, group > 32, decode max_seqlen > 2^24 */
  UATTN_EWORKSPACE = 3,   /* decode workspace missing or smaller than uattn_decode_workspace_bytes() */
  UATTN_ELAUNCH = 4,      /* the HIP runtime rejected a kernel launch */
  UATTN_ESCRATCH = 5      /* uattn_decode_noalloc: the sizes need more than UATTN_DECODE_SCRATCH_BYTES */
} uattn_status;

/* Version of this ABI (UATTN_ABI_VERSION). */
int32_t uattn_abi_version(void);

/* Static, human-readable name of a status code (never NULL). */
const char* uattn_status_string(int32_t status);

/*
 * Full-sequence causal attention over a packed varlen batch (Section 3.2:
 * scores Q K^T, weights P = softmax, output P V; Section 4.1: one invocation
 * processes a whole trajectory under causal masking).
 *
 *   q          [total_tokens, num_q_heads, head_dim]  bf16
 *   k, v       [total_tokens, num_kv_heads, head_dim] bf16
 *   cu_seqlens [num_seqs + 1] int32, cu_seqlens[0] = 0, non-decreasing,
 *              cu_seqlens[num_seqs] = total_tokens; sequence s holds packed
 *              rows cu_seqlens[s] .. cu_seqlens[s+1]-1 (offsets outside
 *              [0, total_tokens] are clamped, so a bad table cannot make the
 *              kernel read or write outside the tensors)
 *   max_seqlen host int >= every sequence length (sizes the launch grid
 *              only; results do not depend on it)
 *   softmax_scale  finite, > 0 (usually 1/sqrt(head_dim))
 *   out        [total_tokens, num_q_heads, head_dim] bf16 (written)
 *   lse        [total_tokens, num_q_heads] fp32 natural-log sum of
 *              exp(scale * score) per row, or NULL
 *
 * Row i of a sequence attends keys 0..i of the same sequence (positions
 * are sequence-relative).  Query head h reads kv head h / (Hq / Hkv).
 * Empty sequences are allowed.  head_dim must be 64 or 128.
 */
uattn_status uattn_prefill(const void* q, const void* k, const void* v, const int32_t* cu_seqlens,
                           int32_t num_seqs, int32_t total_tokens, int32_t max_seqlen,
                           int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                           float softmax_scale, void* out, float* lse, void* stream);

/*
 * Bytes of device workspace uattn_decode needs for these sizes (the fp32
 * partials of the positional split; 0 when no entry can span two chunks).
 * Pure host arithmetic; returns 0 for invalid sizes.
 */
size_t uattn_decode_workspace_bytes(int32_t batch, int32_t max_seqlen, int32_t num_q_heads, int32_t head_dim);

/*
 * Token-wise decode against a paged KV cache (Section 3.1: the cache
 * represents the prefix x_i; Section 3.2: one new query at a time).
 *
 *   q            [batch, num_q_heads, head_dim] bf16; entry b's query is the
 *                token at position seqlens[b]-1
 *   k_pages,
 *   v_pages      [num_pages, num_kv_heads, page_size, head_dim] bf16 (HND);
 *                logical position j of entry b lives in physical page
 *                block_table[b * max_pages_per_seq + j / page_size], slot
 *                j % page_size.  The current token's K/V must already be
 *                written.  Slots at positions >= seqlens[b] are never read,
 *                nor are block_table entries past the last used page.
 *   num_pages    number of physical pages P; a block_table entry outside
 *                [0, P) is never dereferenced (its keys read as zeros)
 *   block_table  [batch, max_pages_per_seq] int32
 *   seqlens      [batch] int32, 1 <= seqlens[b] <= max_seqlen (includes the
 *                current token); values outside that range are clamped to
 *                it (an entry with seqlens[b] < 1 is left unwritten)
 *   max_seqlen   host int >= every seqlens[b] (sizes grid and workspace only),
 *                at most 2^24 (UATTN_EUNSUPPORTED above)
 *   out          [batch, num_q_heads, head_dim] bf16 (written)
 *   lse          [batch, num_q_heads] fp32, or NULL
 *   workspace    device scratch of at least
 *                uattn_decode_workspace_bytes(batch, max_seqlen, Hq, d) bytes
 *                (may be NULL when that is 0), 16-byte aligned.  Its first
 *                C = round_up(4 * batch * num_q_heads, 256) bytes hold one
 *                arrival counter per (entry, kv head); the fp32 chunk
 *                partials go at its end.  The C counter bytes must be zero
 *                when a call starts.  Every call leaves its own counter bytes
 *                zero again (also under HIP graph replay), so: zero-fill a
 *                new workspace once, and zero it again only before a call
 *                whose C is larger than the previous call's on the same
 *                workspace (or after an aborted call).  Calls that share a
 *                workspace must be ordered on one stream.
 *
 * Keys are split into fixed 256-position chunks; each chunk's partial
 * softmax state is folded in ascending chunk order (by whichever workgroup
 * finishes an entry's last chunk), so results do not depend on the batch,
 * its order or the split.  (num_q_heads / num_kv_heads) <= 32.
 */
uattn_status uattn_decode(const void* q, const void* k_pages, const void* v_pages,
                          const int32_t* block_table, const int32_t* seqlens, int32_t batch,
                          int32_t max_pages_per_seq, int32_t page_size, int32_t num_pages, int32_t max_seqlen,
                          int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                          float softmax_scale, void* out, float* lse,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * uattn_decode for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops or harnesses that forbid hipMalloc).
 *
 * Arguments, results and errors are those of uattn_decode, without the
 * workspace: the fp32 partials and arrival counters live in a static device
 * array of UATTN_DECODE_SCRATCH_BYTES bytes that the library owns, one per
 * GPU, held until the process ends.  The call allocates and frees nothing:
 * on the first call on a device it looks up that device's array
 * (hipGetSymbolAddress); every call then zeroes the array's counter region
 * with a small kernel and launches the decode kernel on `stream`, so the
 * call may be captured into a HIP graph.  Results are bit-identical to
 * uattn_decode's.
 *
 * Sizes whose uattn_decode_workspace_bytes(batch, max_seqlen, num_q_heads,
 * head_dim) exceeds UATTN_DECODE_SCRATCH_BYTES return UATTN_ESCRATCH before
 * any HIP call (e.g. 64 MiB holds batch 8 x 64 q heads x 32K keys, or batch
 * 64 x 32 q heads x 16K keys).  Every call on a GPU shares that GPU's array
 * and leaves its contents behind: calls that overlap on one GPU (streams
 * not ordered with respect to each other) race and give wrong results; order
 * them on one stream.
 */
#define UATTN_DECODE_SCRATCH_BYTES ((size_t)64 << 20)

/* UATTN_DECODE_SCRATCH_BYTES, as built into the library. */
size_t uattn_decode_scratch_limit(void);

uattn_status uattn_decode_noalloc(const void* q, const void* k_pages, const void* v_pages,
                                  const int32_t* block_table, const int32_t* seqlens, int32_t batch,
                                  int32_t max_pages_per_seq, int32_t page_size, int32_t num_pages, int32_t max_seqlen,
                                  int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                  float softmax_scale, void* out, float* lse, void* stream);

/*
 * Per-token log-probability of the recorded token (Section 3.1: the same
 * deterministic logit processing and normalization in both regimes):
 *
 *   logp[t] = x_t[targets[t]] - log sum_v exp(x_t[v]),  x_t = logits[t] * inv_temperature
 *
 *   logits       [num_rows, row_stride] bf16, the first `vocab` entries of
 *                each row are used; the pointer must be 16-byte aligned and
 *                row_stride a multiple of 8 (elements)
 *   targets      [num_rows] int32 in [0, vocab); a row whose target is
 *                outside that range gets NaN
 *   inv_temperature  finite, > 0
 *   logp         [num_rows] fp32 (written)
 *
 * Each row is reduced by one workgroup in a fixed order that depends only on
 * vocab, so a row's result is bit-identical whatever num_rows or its position.
 */
uattn_status uattn_logprob(const void* logits, int64_t row_stride, const int32_t* targets,
                           int32_t num_rows, int32_t vocab, float inv_temperature, float* logp,
                           void* stream);

/*
 * Indexed write of new keys and values into the paged cache (the rollout-only
 * KV-cache operator whose post-write state is checked exactly, Section 6 Q3
 * and its table of prescribed bitwise checks):
 *
 *   for every token n with positions[n] >= 0, every kv head h, every d:
 *     page = block_table[seq_idx[n] * max_pages_per_seq + positions[n] / page_size]
 *     k_pages[page][h][positions[n] % page_size][:] = k_new[n * token_stride + h * head_dim + :]
 *     v_pages[...same...]                             = v_new[n * token_stride + h * head_dim + :]
 *
 *   k_new, v_new   token rows of num_kv_heads * head_dim bf16 (heads contiguous),
 *                  token_stride elements apart (>= num_kv_heads * head_dim, a
 *                  multiple of 8); 16-byte aligned
 *   block_table    [batch, max_pages_per_seq] int32 (the decode layout)
 *   seq_idx        [num_tokens] int32, row of block_table of each token
 *   positions      [num_tokens] int32, position of each token in its sequence
 *                  (< 0: padding, the token is not written)
 *   k_pages, v_pages  [num_pages, num_kv_heads, page_size, head_dim] bf16 (written
 *                  in place; every slot no token maps to keeps its bits)
 *
 * A token whose seq_idx is outside [0, batch), whose position / page_size is
 * not below max_pages_per_seq, or whose table entry is outside
 * [0, num_pages) is not written (device values are trusted but never used to
 * form an address outside the tensors).  Two tokens mapping to one slot
 * write it in unspecified order.  head_dim 64 or 128; page_size a power of
 * two >= 16.  Values are copied bit for bit.
 */
uattn_status uattn_kv_write(const void* k_new, const void* v_new, int64_t token_stride,
                            const int32_t* block_table, const int32_t* seq_idx, const int32_t* positions,
                            int32_t num_tokens, int32_t batch, int32_t max_pages_per_seq, int32_t page_size,
                            int32_t num_pages, int32_t num_kv_heads, int32_t head_dim,
                            void* k_pages, void* v_pages, void* stream);

/*
 * Query/key normalization and rotary position embedding before attention, in
 * one pass (the Q RMSNorm, K RMSNorm and NeoX RoPE operators of Section 6 Q3,
 * whose full-sequence and token-wise outputs must agree bit for bit).  For
 * every token t and every head row x = q[t][h][:] (and k[t][h][:]):
 *
 *   r      = 1 / sqrt(sum_i x_i^2 / head_dim + eps)     (fp32, fixed order)
 *   y_i    = bf16( w_i * bf16(x_i * r) )                 (w = q_weight or k_weight)
 *   for i < head_dim / 2, with c = cos_sin[pos][i][0], s = cos_sin[pos][i][1], pos = positions[t]:
 *     out_i              = bf16( y_i * c - y_{i+head_dim/2} * s )
 *     out_{i+head_dim/2} = bf16( y_{i+head_dim/2} * c + y_i * s )
 *
 *   q, k           [num_tokens, num_q_heads | num_kv_heads, head_dim] bf16, contiguous
 *   positions      [num_tokens] int32 in [0, max_position)
 *   q_weight, k_weight  [head_dim] bf16
 *   cos_sin        [max_position, head_dim / 2, 2] fp32 (uattn_rope_cache)
 *   q_out, k_out   same shapes as q, k (written; may be q, k themselves)
 *
 * Every row is computed by the same instruction sequence whatever num_tokens
 * or the row's place in the batch.  A token whose position is outside
 * [0, max_position) gets NaN rows.  head_dim 64 or 128; every tensor
 * argument except positions 16-byte aligned.
 */
uattn_status uattn_qk_norm_rope(const void* q, const void* k, const int32_t* positions, const void* q_weight,
                                const void* k_weight, float eps, const float* cos_sin, int32_t max_position,
                                int32_t num_tokens, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                void* q_out, void* k_out, void* stream);

/*
 * The rotary table for uattn_qk_norm_rope (NeoX layout):
 *   cos_sin[p][i][0] = fp32(cos(p * theta^(-2i/head_dim))),  cos_sin[p][i][1] = fp32(sin(...))
 * with the angle and both functions evaluated in fp64, for p < max_position
 * and i < head_dim / 2.  theta > 1.
 */
uattn_status uattn_rope_cache(float* cos_sin, int32_t max_position, int32_t head_dim, double theta, void* stream);

/*
 * Batch-invariant LM head: the logits the log-probability reads (Section 3.1
 * requires the same deterministic logit processing in both regimes, so the
 * logits themselves must not depend on how many rows are computed together):
 *
 *   logits[t][v] = bf16( sum_k hidden[t][k] * weight[v][k] )
 *
 * accumulated in fp32 on v_mfma_f32_16x16x32_bf16 over k in ascending 32-wide
 * steps from zero; no split over k, and the tiling over t never changes a
 * row's arithmetic, so a row's logits are bit-identical whatever num_rows or
 * the row's place in the batch.
 *
 *   hidden   [num_rows, hidden_stride] bf16, first hidden_dim used
 *   weight   [vocab, weight_stride] bf16, first hidden_dim used
 *   logits   [num_rows, logits_stride] bf16, first vocab written
 *   hidden_dim a multiple of 64; strides >= the used widths and multiples of
 *   8 elements; pointers 16-byte aligned.
 */
uattn_status uattn_lm_head(const void* hidden, int64_t hidden_stride, const void* weight, int64_t weight_stride,
                           int32_t num_rows, int32_t vocab, int32_t hidden_dim, void* logits, int64_t logits_stride,
                           void* stream);

/*
 * Bytes of device workspace uattn_lm_head_logprob needs for these sizes:
 * two fp32 partials per (row, 256-entry vocabulary tile) and one per row.
 * Pure host arithmetic; 0 for invalid sizes.
 */
size_t uattn_lm_head_logprob_workspace_bytes(int32_t num_rows, int32_t vocab);

/*
 * The LM head fused with the per-token log-probability (Section 3.1: the
 * token log-probability after one deterministic logit processing, with the
 * logits themselves batch-invariant):
 *
 *   z[t][v]  = bf16( sum_k hidden[t][k] * weight[v][k] )     (exactly uattn_lm_head's logits)
 *   logp[t]  = x[t][targets[t]] - log sum_v exp(x[t][v]),   x = z * inv_temperature
 *
 * computed without a round trip of the logits through memory: the GEMM's
 * epilogue reduces each row's logits of every 256-entry vocabulary tile to a
 * (max, sum of exp) pair in a fixed order (lanes, then the tile's four waves)
 * and picks out the target's logit; a second kernel folds each row's pairs in
 * ascending tile order.  The order depends only on vocabulary positions, so
 * a row's logp is bit-identical whatever num_rows or its place in the batch
 * (the reuse ratio of the two regimes is exactly 1).  It is not bit-identical
 * to uattn_logprob over the same logits, whose reduction is ordered
 * differently (both are within rounding of the exact value).
 *
 *   hidden, weight, num_rows, vocab, hidden_dim, strides: as uattn_lm_head
 *   targets    [num_rows] int32; a target outside [0, vocab) gives NaN
 *   inv_temperature  finite, > 0
 *   logp       [num_rows] fp32 (written)
 *   logits     [num_rows, logits_stride] bf16, or NULL: when given, the
 *              logits are stored as well (the same bits as uattn_lm_head)
 *   workspace  device scratch of at least
 *              uattn_lm_head_logprob_workspace_bytes(num_rows, vocab) bytes,
 *              4-byte aligned, no initial contents needed; calls sharing a
 *              workspace must be ordered on one stream
 */
uattn_status uattn_lm_head_logprob(const void* hidden, int64_t hidden_stride, const void* weight,
                                   int64_t weight_stride, const int32_t* targets, int32_t num_rows, int32_t vocab,
                                   int32_t hidden_dim, float inv_temperature, float* logp, void* logits,
                                   int64_t logits_stride, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Bytes of device workspace uattn_prefill_backward needs: two fp32 values
 * per (token, q head).  Pure host arithmetic; 0 for invalid sizes.
 */
size_t uattn_prefill_backward_workspace_bytes(int32_t total_tokens, int32_t num_q_heads);

/*
 * Gradients of the full-sequence attention (the backward of uattn_prefill,
 * which the policy update runs after its forward over every trajectory,
 * Section 6 Q2).  The gradient of the Section 3.2 attention by the chain
 * rule: for each (sequence, q head), with P the causal softmax weights,
 *
 *   dV = P^T dO,  dS = P * (dO V^T - D) with D_i = dO_i . O_i,
 *   dQ = scale * dS K,  dK = scale * dS^T Q,
 *
 * dK and dV summed over the q heads of each group.  P is recomputed from the
 * forward's log-sum-exp, D from its output.
 *
 *   q, k, v, cu_seqlens, num_seqs .. softmax_scale   exactly as passed to
 *              uattn_prefill (same layouts, same clamping of cu_seqlens)
 *   out        [total_tokens, num_q_heads, head_dim] bf16, uattn_prefill's output
 *   dout       [total_tokens, num_q_heads, head_dim] bf16, upstream gradient
 *   lse        [total_tokens, num_q_heads] fp32, uattn_prefill's log-sum-exp
 *   dq         [total_tokens, num_q_heads, head_dim] bf16 (written)
 *   dk, dv     [total_tokens, num_kv_heads, head_dim] bf16 (written; every row
 *              of every sequence, zero-length sequences aside)
 *   workspace  device scratch of at least
 *              uattn_prefill_backward_workspace_bytes(total_tokens, num_q_heads)
 *              bytes, 16-byte aligned; overwritten, no initial contents needed.
 *              Calls that share a workspace must be ordered on one stream.
 *
 * Deterministic and batch-invariant: no atomics; each output row is summed by
 * one workgroup in an order fixed by its own sequence (fp32 accumulation,
 * bf16 P and dS as matrix operands, one bf16 rounding of each result), so
 * repeated calls, and the same sequence in any batch, give identical bits.
 * head_dim 64 or 128; bf16 tensors 16-byte aligned, lse 4-byte aligned.
 */
uattn_status uattn_prefill_backward(const void* q, const void* k, const void* v, const void* out, const void* dout,
                                    const float* lse, const int32_t* cu_seqlens, int32_t num_seqs,
                                    int32_t total_tokens, int32_t max_seqlen, int32_t num_q_heads,
                                    int32_t num_kv_heads, int32_t head_dim, float softmax_scale, void* dq, void* dk,
                                    void* dv, void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* UATTN_H */
