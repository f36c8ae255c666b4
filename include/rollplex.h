/*
 * rollplex.h -- C ABI of the MI355X (gfx950) prefix/suffix backbone path.
 *
 * Rollplex (arXiv 2608.14498) splits every model invocation of VLM RL at the
 * first response position (Section "Observation and Opportunity"): the prefix
 * pass (prompt prefill over visual + text tokens) depends only on the input
 * and the weights, produces boundary KV state and the prefix's log-probability
 * state, and can run while rollout still decodes; the suffix pass continues
 * from the retained boundary and scores the response tokens (Section
 * "Cross-Phase Execution", Phases 1 and 2).  This library runs both passes of
 * a Qwen2-style decoder backbone (RMSNorm, rotate-half RoPE, grouped-query
 * attention, SwiGLU MLP, untied lm_head) with hand-written HIP kernels, plus
 * the rollout-side decode step and a CU-masked stream helper for running the
 * prefix pass beside decode on one GPU (Eq. (1) and Section "Resource Sharing
 * Policy").
 *
 * Conventions shared by every entry point
 *   - Ownership: the caller owns all weights, inputs, outputs, KV buffers and
 *     workspaces.  The library keeps only the pointers given to rp_create and
 *     a few host-side constants; it never frees, reallocates or retains
 *     caller memory beyond rp_destroy.
 *   - Asynchrony: compute calls enqueue kernels on the given HIP stream
 *     (passed as void*, a hipStream_t; NULL = the null stream) and return
 *     without synchronising.  Outputs are valid once the stream reaches that
 *     point; inputs must stay alive until then.  Concurrent calls need
 *     separate workspaces; one model handle may be shared across streams.
 *   - Errors: no exception crosses the ABI.  Host-side validation runs before
 *     any HIP call and returns RP_ERR_INVALID_ARG (null/misaligned pointer,
 *     bad enum), RP_ERR_SHAPE (bad lengths or offsets), RP_ERR_UNSUPPORTED
 *     (shape outside what the kernels implement) or RP_ERR_WORKSPACE
 *     (workspace too small).  A failed launch returns RP_ERR_HIP.  The text
 *     of the last non-OK status of the calling thread is rp_last_error().
 *   - Dtypes: weights, visual embeddings and KV share rp_config.dtype (fp32,
 *     bf16 or fp16; row-major, nn.Linear layout [out, in] for projections).
 *     The 16-bit dtypes run the same kernels (MFMA with fp32 accumulation,
 *     fp32 residual stream) and differ only in the storage rounding of
 *     activations, K/V and weights: fp16 carries 3 more mantissa bits, so a
 *     bf16-trained model whose weights convert to fp16 exactly (|w| within
 *     fp16's normal range) computes its log-probabilities about 8x closer to
 *     exact arithmetic at the same speed.
 *     h_last, hidden_out, logprobs and logits are always fp32.  Token ids are
 *     int32.  Length tables (cu_seqlens) are HOST int32 arrays.
 *   - Device-side data the host cannot see (token ids, kv_len) is clamped to
 *     valid ranges inside the kernels, so bad values give unspecified numbers
 *     but never an out-of-bounds access.
 *   - Device pointers must be 16-byte aligned (workspaces 256-byte aligned).
 */
#ifndef ROLLPLEX_H
#define ROLLPLEX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RP_MAX_SEQS 256 /* sequences per prefix/suffix call */

typedef enum {
  RP_OK = 0,
  RP_ERR_INVALID_ARG = 1,
  RP_ERR_SHAPE = 2,
  RP_ERR_UNSUPPORTED = 3,
  RP_ERR_WORKSPACE = 4,
  RP_ERR_HIP = 5
} rp_status;

typedef enum { RP_F32 = 0, RP_BF16 = 1, RP_F16 = 2 } rp_dtype;

/* Backbone hyper-parameters.  head_dim must be 64 or 128; n_q_heads a
 * multiple of n_kv_heads, at most 8 q heads per kv head (q head h reads kv head
 * h / (n_q_heads/n_kv_heads)).
 * For bf16 and fp16, d_model, ffn_dim and n_q_heads*head_dim must be
 * multiples of 64.
 * rms_eps is the RMSNorm epsilon (1e-6 for the Qwen2 family); rope_theta the
 * RoPE base (1e6).  max_position bounds every position a call may use. */
/* Storage of the row-parallel projections (Section "Parallelism-Aware Weight
 * Sharing", Case 2: a logical [O, I] weight sharded along I is kept as [I, O],
 * so that every tensor-parallel shard of it is one contiguous range shared by
 * the training and rollout engines; the GEMMs read it in transpose mode and no
 * copy in the logical orientation is made).  Bits of rp_config.weight_layout;
 * others are RP_ERR_INVALID_ARG. */
#define RP_WO_TRANSPOSED 1u     /* wo stored [n_q_heads*head_dim][d_model] */
#define RP_W_DOWN_TRANSPOSED 2u /* w_down stored [ffn_dim][d_model] */
#define RP_WEIGHT_LAYOUTS 3u    /* all defined bits */

typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab, max_position;
  float rms_eps;
  double rope_theta;
  rp_dtype dtype;
  uint32_t weight_layout; /* RP_*_TRANSPOSED bits; 0 = nn.Linear layout throughout */
} rp_config;

/* One decoder layer, device pointers, nn.Linear layout [out, in]:
 * wq [Hq*Dh, d], wk/wv [Hkv*Dh, d], wo [d, Hq*Dh], w_gate/w_up [F, d],
 * w_down [d, F]; attn_norm/mlp_norm [d]; biases bq [Hq*Dh], bk/bv [Hkv*Dh]
 * are optional (NULL = none).  wo and w_down are stored transposed when
 * rp_config.weight_layout says so. */
typedef struct {
  const void *attn_norm, *wq, *wk, *wv, *bq, *bk, *bv, *wo;
  const void *mlp_norm, *w_gate, *w_up, *w_down;
} rp_layer_weights;

/* embed [V, d], final_norm [d], lm_head [V, d] (untied), layers: HOST array
 * of n_layers entries (copied by rp_create). */
typedef struct {
  const void *embed, *final_norm, *lm_head;
  const rp_layer_weights *layers;
} rp_weights;

/* Per-layer K and V buffers: layer l starts at k + l*layer_stride elements
 * (of rp_config.dtype); within a layer, rows of [n_kv_heads][head_dim].
 * K is stored after RoPE. */
typedef struct {
  void *k, *v;
  int64_t layer_stride;
} rp_kv;

typedef struct rp_model rp_model;

/* Validates cfg and weights and binds the pointers (no device memory is
 * allocated; no HIP call is made).  *out receives a handle freed by
 * rp_destroy. */
rp_status rp_create(const rp_config *cfg, const rp_weights *weights, rp_model **out);
void rp_destroy(rp_model *model);

/* ---------------------------------------------------------------------------
 * Prefix pass (Section "Observation and Opportunity": the response-independent
 * part of the invocation, prompt prefill producing boundary KV and prefix
 * log-probability state; Phase 1 of Section "Cross-Phase Execution").
 *
 * B sequences are packed: sequence b occupies rows cu_seqlens[b] ..
 * cu_seqlens[b+1]-1 (cu_seqlens[0] = 0, strictly increasing: every prefix
 * has at least one token), at positions 0 .. P_b-1.
 * token_ids  dev int32 [T]: a vocabulary id, or -1 for a visual slot; visual
 *            slots take the rows of visual_embeds in order over the packed
 *            batch (n_visual rows of [d]; slots beyond n_visual read zeros).
 * kv_out     dev, caller-allocated: K/V of every layer and prefix row, post
 *            RoPE; layer_stride >= T*n_kv_heads*head_dim.
 * h_last     dev fp32 [B, d]: the residual stream at each sequence's last
 *            prefix position after the last layer, before the final norm.
 *            It determines the boundary distribution that scores the first
 *            response token.
 * hidden_out optional dev fp32 [T, d]: the full last-layer residual stream.
 * workspace  dev, >= rp_prefix_workspace_bytes(); contents are scratch.
 * ------------------------------------------------------------------------- */
rp_status rp_prefix_workspace_bytes(const rp_model *model, int32_t B, const int32_t *cu_seqlens_host,
                                    size_t *bytes);
rp_status rp_prefix_forward(const rp_model *model, void *stream, int32_t B,
                            const int32_t *cu_seqlens_host, const int32_t *token_ids,
                            const void *visual_embeds, int64_t n_visual, rp_kv kv_out,
                            float *h_last, float *hidden_out, void *workspace,
                            size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * Prefix pass with multimodal RoPE (Qwen2.5-VL-style 3-D positions; the paper's
 * models are Qwen2.5-VL, Section "Experimental Setup", and it does not describe
 * the rotary scheme).  Identical to rp_prefix_forward except for the rotation:
 * positions is a device int32 [3][T] array (row 0 temporal, 1 height, 2 width
 * position of every prefix row; text tokens carry three equal values), 16-byte
 * aligned, values clamped to [0, max_position).  mrope_section (host int32 [3],
 * non-negative, summing to head_dim / 2, else RP_ERR_SHAPE) splits the rotary
 * pairs i < head_dim/2 into consecutive temporal, height and width sections:
 * pair i rotates by the position of its section.  Qwen2.5-VL uses {16, 24, 24}.
 * The causal rule follows token order; score the responses with
 * rp_suffix_logprob_grouped and rope_pos0 = each prefix's next rotary position.
 * Workspace: rp_prefix_workspace_bytes.
 * ------------------------------------------------------------------------- */
rp_status rp_prefix_forward_mrope(const rp_model *model, void *stream, int32_t B,
                                  const int32_t *cu_seqlens_host, const int32_t *token_ids,
                                  const void *visual_embeds, int64_t n_visual, const int32_t *positions,
                                  const int32_t *mrope_section, rp_kv kv_out, float *h_last,
                                  float *hidden_out, void *workspace, size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * Suffix pass (Phase 2 of Section "Cross-Phase Execution": the suffix
 * continues from the retained boundary and scores the response without
 * recomputing the prompt; prefix and suffix log-probabilities together form
 * the full-sequence values).
 *
 * Sequence b's response r_b,0 .. r_b,S_b-1 occupies rows suffix_cu[b] ..
 * suffix_cu[b+1]-1 (non-decreasing; S_b = 0 allowed) at positions P_b + j;
 * its prefix is rows prefix_cu[b] .. of kv (read only) and h_last[b].
 * logprobs[suffix_cu[b]+j] = log p(r_b,j | prefix_b, r_b,<j), scored with the
 * full vocabulary at temperature 1: j = 0 from h_last[b], j > 0 from the
 * hidden state of response token j-1.
 * ------------------------------------------------------------------------- */
rp_status rp_suffix_workspace_bytes(const rp_model *model, int32_t B, const int32_t *prefix_cu_host,
                                    const int32_t *suffix_cu_host, size_t *bytes);
rp_status rp_suffix_logprob(const rp_model *model, void *stream, int32_t B,
                            const int32_t *prefix_cu_host, const int32_t *suffix_cu_host, rp_kv kv,
                            const float *h_last, const int32_t *response_ids, float *logprobs,
                            void *workspace, size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * Prefix pass with options: rp_prefix_forward (positions and mrope_section
 * NULL) or rp_prefix_forward_mrope (both given), plus flags:
 *   RP_PREFIX_LAST_ROWS_ONLY  the suffix pass reads every prefix row's K/V but
 *     only the boundary state h_last (Section "Cross-Phase Execution"), so the
 *     last layer runs its K/V projection for every row and the rest (attention,
 *     o-proj, MLP) only at each sequence's last row.  kv_out is exactly that of
 *     the full pass; h_last equals it up to fp32 summation order (its GEMMs
 *     split K over the few rows).  hidden_out must be NULL (RP_ERR_INVALID_ARG).
 *     With 1-D positions (positions NULL), 16-bit models at head_dim 64 return
 *     RP_ERR_UNSUPPORTED: a GPU memory fault in a run that included that
 *     combination has no known cause, so it stays disabled until one is shown.
 * Unknown flag bits are RP_ERR_INVALID_ARG.  Workspace: rp_prefix_workspace_bytes.
 * ------------------------------------------------------------------------- */
#define RP_PREFIX_LAST_ROWS_ONLY 1u
#define RP_PREFIX_FLAGS 1u /* all defined flag bits */
rp_status rp_prefix_forward_flags(const rp_model *model, void *stream, int32_t B,
                                  const int32_t *cu_seqlens_host, const int32_t *token_ids,
                                  const void *visual_embeds, int64_t n_visual,
                                  const int32_t *positions, const int32_t *mrope_section,
                                  uint32_t flags, rp_kv kv_out, float *h_last, float *hidden_out,
                                  void *workspace, size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * Shared-prefix suffix pass (Section "Prefix Sharing": the N sampled responses
 * of a GRPO prompt group share one video-text prefix, whose prefix pass runs
 * once per group and is reused by every response).  n_suffix sequences score
 * against n_prefix prefixes: sequence s reads prefix p = prefix_of_suffix[s]
 * (host int32 [n_suffix], each in [0, n_prefix)), i.e. KV rows
 * prefix_cu[p] .. prefix_cu[p+1]-1 of kv (read only) and h_last[p]
 * (fp32 [n_prefix, d], 16-byte aligned).  Its response occupies rows
 * suffix_cu[s] .. suffix_cu[s+1]-1 of response_ids / logprobs at positions
 * P_p + j; logprobs[suffix_cu[s]+j] = log p(r_s,j | prefix_p, r_s,<j) exactly
 * as in rp_suffix_logprob, which is this call with prefix_of_suffix[s] = s.
 * Any prefix may serve any number of suffixes (also none).  n_prefix and
 * n_suffix are in [1, RP_MAX_SEQS]; P_p >= 1, S_s >= 0 and
 * P_p + S_s <= max_position, else RP_ERR_SHAPE; a prefix index out of range
 * is RP_ERR_SHAPE.  Ownership, asynchrony and workspace rules as above.
 *
 * rope_pos0_host (host int32 [n_prefix], nullable): rotary position of the first
 * response token after prefix p; response token j then rotates by
 * rope_pos0[p] + j with equal temporal, height and width positions (plain 1-D
 * RoPE; after a prefix run with multimodal positions this is the prefix's next
 * rotary position).  NULL means P_p.  The causal rule still follows token order.
 * rope_pos0[p] + S_s must not exceed max_position (RP_ERR_SHAPE).
 *
 * flags (bits; others are RP_ERR_INVALID_ARG):
 *   RP_SUFFIX_FUSED_LOGPROB  score with an lm_head whose epilogue keeps an online
 *     log-sum-exp per row and the target logit, so the [R, V] logits are never
 *     stored (the same log-probs up to fp32 summation order; the workspace
 *     holds R * 8 * 2 * ceil(V / 256) bytes of partials instead of R * V * 4
 *     bytes of logits).  16-bit models only; an fp32 model ignores the bit.
 *     The workspace size depends on flags: query it with the same flags.
 * ------------------------------------------------------------------------- */
#define RP_SUFFIX_FUSED_LOGPROB 1u
#define RP_SUFFIX_FLAGS 1u /* all defined flag bits */
rp_status rp_suffix_grouped_workspace_bytes(const rp_model *model, int32_t n_prefix,
                                            const int32_t *prefix_cu_host, int32_t n_suffix,
                                            const int32_t *prefix_of_suffix_host,
                                            const int32_t *suffix_cu_host, uint32_t flags,
                                            size_t *bytes);
rp_status rp_suffix_logprob_grouped(const rp_model *model, void *stream, int32_t n_prefix,
                                    const int32_t *prefix_cu_host, int32_t n_suffix,
                                    const int32_t *prefix_of_suffix_host,
                                    const int32_t *suffix_cu_host, const int32_t *rope_pos0_host,
                                    uint32_t flags, rp_kv kv, const float *h_last,
                                    const int32_t *response_ids, float *logprobs, void *workspace,
                                    size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * Prompt-token log-probabilities (the response-independent "prefix log-probs"
 * of Section "Observation and Opportunity", produced from the prefix pass's
 * output): teacher-forced log-probabilities of the prompt's own text tokens.
 * B, cu_seqlens_host and token_ids describe the packed prefixes exactly as in
 * rp_prefix_forward; hidden is that call's hidden_out (dev fp32 [T, d], the
 * last-layer residual stream before the final norm, 16-byte aligned).
 * positions (dev int32 [n_rows]) lists packed prompt positions t; then
 *   logprobs[i] = log p(token_ids[t] | the tokens of t's sequence before t),
 * scored like a response token from row t-1 (final norm, lm_head, log-softmax
 * over the vocabulary).  logprobs[i] is NaN when t is outside [0, T), is the
 * first token of its sequence, or is a visual slot (token_ids[t] < 0).
 * Positions may repeat and come in any order.  n_rows >= 0 (else RP_ERR_SHAPE);
 * n_rows = 0 launches nothing.  flags as in rp_suffix_logprob_grouped
 * (RP_SUFFIX_FUSED_LOGPROB: never store the [n_rows, V] logits); query the
 * workspace with the same flags.  Asynchronous on stream; inputs are read only.
 * ------------------------------------------------------------------------- */
rp_status rp_prompt_logprob_workspace_bytes(const rp_model *model, int32_t n_rows, uint32_t flags,
                                            size_t *bytes);
rp_status rp_prompt_logprob(const rp_model *model, void *stream, int32_t B,
                            const int32_t *cu_seqlens_host, const int32_t *token_ids,
                            const float *hidden, int32_t n_rows, const int32_t *positions,
                            uint32_t flags, float *logprobs, void *workspace,
                            size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * Rollout decode step (the memory-bound phase that the prefix pass overlaps
 * with; Section "Observation and Opportunity" and Eq. (1)).  One new token
 * per sequence: token_ids[b] runs at position kv_len[b], its K/V are written
 * to slot kv_len[b] of cache (layout [L][B][cap][n_kv_heads][head_dim],
 * layer_stride >= B*cap*n_kv_heads*head_dim), it attends to slots
 * 0..kv_len[b], and next_ids[b] = argmax of its logits (lowest id on ties).
 * kv_len is a device int32 [B] array, values clamped to [0, cap-1] (and to
 * max_position-1).  logits (optional) receives fp32 [B, V]; when it is NULL, a
 * 16-bit model with B <= 64 takes the argmax inside the lm_head product and the
 * logits are never formed (same next_ids as the stored-logits path).
 * bf16 models at head_dim 64 return RP_ERR_UNSUPPORTED (disabled: a GPU memory
 * fault in a run that included that combination has no known cause).
 * ------------------------------------------------------------------------- */
rp_status rp_decode_workspace_bytes(const rp_model *model, int32_t B, int32_t cap, size_t *bytes);
rp_status rp_decode_step(const rp_model *model, void *stream, int32_t B, rp_kv cache, int32_t cap,
                         const int32_t *kv_len, const int32_t *token_ids, float *logits,
                         int32_t *next_ids, void *workspace, size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * rp_decode_step without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation).  Arguments and results are those of rp_decode_step; the
 * scratch is a library-owned static device array of
 * RP_DECODE_STATIC_SCRATCH_BYTES on each GPU the library runs on (held until the
 * process ends).  The call allocates nothing; its first call on a device looks up
 * that device's copy of the array.
 * The scratch needed is rp_decode_workspace_bytes() less the [B, V] fp32 logits
 * when logits is non-NULL or the argmax is fused (about 44 MiB for the 7B slice
 * at B = 64, cap 8256); larger needs return RP_ERR_WORKSPACE before any HIP call.  No part of
 * the scratch needs to start at zero: every byte a step reads was written earlier
 * in the same step.  Every call on a GPU shares that GPU's array, so calls that
 * overlap on one GPU (concurrent streams, or a captured graph replayed while
 * another call runs) race; serialise them.
 * ------------------------------------------------------------------------- */
#define RP_DECODE_STATIC_SCRATCH_BYTES (96u << 20)
rp_status rp_decode_step_static(const rp_model *model, void *stream, int32_t B, rp_kv cache, int32_t cap,
                                const int32_t *kv_len, const int32_t *token_ids, float *logits,
                                int32_t *next_ids);

/* ---------------------------------------------------------------------------
 * Co-location helpers (Section "Resource Sharing Policy": decode and prefix
 * share one GPU; static partitions are the analog of the paper's SM
 * partitions).  mask: n_words 32-bit words, bit i = compute unit i may run
 * this stream's work.  The stream has the default priority.
 * ------------------------------------------------------------------------- */
rp_status rp_stream_create_cu_masked(int device, const uint32_t *mask, uint32_t n_words, void **out);
rp_status rp_stream_destroy(void *stream);
int rp_device_cu_count(int device);

/* ---------------------------------------------------------------------------
 * Per-launch timing (measurement aid, off by default; not thread-safe).
 * While enabled, every kernel launch of the compute entry points is bracketed
 * by two HIP events recorded on the launch stream.  rp_profile_collect waits
 * for those events and accumulates, per kernel name, the launch count and the
 * summed duration; rp_profile_read(i) returns entry i (0 <= i < count).
 * max_launches bounds the number of bracketed launches until the next collect
 * (later launches run untimed).  Enabling creates the events (a HIP call);
 * disabling destroys them.
 * ------------------------------------------------------------------------- */
rp_status rp_profile_enable(int enable, int32_t max_launches);
rp_status rp_profile_collect(void);
int32_t rp_profile_count(void);
rp_status rp_profile_read(int32_t i, const char **name, int64_t *launches, double *total_ms);
void rp_profile_reset(void);

/* ---------------------------------------------------------------------------
 * Matrix-core probe (measurement aid): launches blocks workgroups of 256
 * threads on stream; every wave issues iters x 8 independent 32x32x16 MFMAs of
 * dtype (RP_BF16 or RP_F16) on random register operands and writes one float
 * per thread to sink (device, >= blocks*256*4 bytes, else RP_ERR_WORKSPACE).
 * *flops (nullable) receives the launch's matrix flop count; the caller times
 * the launch (e.g. with events on the same stream).  Asynchronous.
 * ------------------------------------------------------------------------- */
rp_status rp_calibrate_mfma(void *stream, rp_dtype dtype, int32_t blocks, int32_t iters, float *sink,
                            size_t sink_bytes, double *flops);

/* HBM read probe (measurement aid): blocks workgroups of 256 threads stream bytes
 * (a positive multiple of 16) of device memory src once with 16-byte loads and
 * write one word per thread to sink (>= blocks*256*4 bytes).  Asynchronous; the
 * caller times it. */
rp_status rp_calibrate_read(void *stream, const void *src, int64_t bytes, int32_t blocks, uint32_t *sink,
                            size_t sink_bytes);

const char *rp_last_error(void);
const char *rp_status_string(rp_status status);
const char *rp_version(void);

#ifdef __cplusplus
}
#endif
#endif /* ROLLPLEX_H */
