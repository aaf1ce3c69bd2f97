/*
 * moa.h - C ABI of the MI355X (gfx950) Mixture-of-Attention-Spans library.
 *
 * Mixture of Attention Spans (MoA) gives every attention head (every KV head
 * under grouped-query attention) its own sliding-window length, set by an
 * elastic rule over the input length N, plus a few always-visible initial
 * "sink" tokens.  This library computes that attention on one GPU:
 *
 *   moa_plan       per-head window / cache-capacity / cache-offset tables
 *                  from the rule parameters (paper Sec. 3.2, Eq. 2; span
 *                  clipping in Appendix "Main Setup").
 *   moa_prefill    banded-plus-sink causal attention over a whole prompt
 *                  (paper Sec. 2.1, Eq. 1 with the Sec. 3.2 mask).
 *   moa_kv_append  writes new tokens into per-head static caches that keep
 *                  the sinks and the latest window tokens, replacing the
 *                  oldest non-sink entry in place (paper Appendix
 *                  "Efficiency Experiment Setup", "Memory and Throughput
 *                  Breakdown": a head's cache is exactly as long as its
 *                  span, and a new token overwrites the entry that has
 *                  left the span).
 *   moa_decode     one query token per sequence against the per-head caches
 *                  of different lengths (paper Appendix "Efficiency
 *                  Experiment Setup": decode over KV caches whose length
 *                  differs across heads).
 *   moa_kv_append_ragged, moa_decode_ragged
 *                  the same one-token append and decode with every sequence
 *                  of the batch at its own position (device position array).
 *   moa_influence  the profiling step that precedes the rule search: the
 *                  block-averaged attention influence of dense attention
 *                  (paper Sec. 3.3, Eq. 3).
 *   moa_rule_loss  the loss table of candidate rules from that profile
 *                  (paper Sec. 3.3, Eq. 4), input of the rule selection.
 *
 * Definitions used throughout (s = num_sink, w_g = window of KV head g):
 *   window    w_g = min(max(floor(alpha_g + beta_g * N), 1), N), evaluated
 *             in IEEE double without fused multiply-add.
 *   visible   query position i sees key position j iff j <= i and
 *             (j < s or i - j < w_g).  The band includes the query itself.
 *   capacity  C_g = s + w_g cache slots for KV head g.
 *   slot      position p is stored in slot p if p < s, otherwise in slot
 *             s + ((p - s) mod w_g); a later position that maps to the same
 *             slot replaces the earlier one (the earlier one is always the
 *             oldest non-sink entry).
 *   scale     scores are scale * (q . k); scale = 1/sqrt(head_dim) when the
 *             descriptor's softmax_scale is 0.
 *
 * Plan options (moa_desc_t.flags), the paper's own kernel setting:
 *   MOA_SPAN_INCLUDES_SINKS  the rule gives the whole span S including the
 *             sinks (paper Sec. 3.2 and Appendix "Attention Span": span =
 *             sliding window + initially unmasked tokens):
 *             S = min(max(floor(alpha_g + beta_g * N), 0), N) and
 *             w_g = max(S - s, 1).
 *   MOA_BLOCK_BAND  moa_prefill counts the band in blocks of MOA_BAND_BLOCK
 *             tokens (paper Appendix "Main Setup": block sliding window of 64
 *             tokens): i sees j iff j <= i and
 *             (j < s or i / 64 - j / 64 < ceil(w_g / 64)).  The caches and
 *             moa_decode keep the token-exact band (the cache replaces the
 *             oldest token one at a time), so with this option a decode step
 *             is not the last prefill row.
 *
 * Layouts (all row-major, contiguous, element type = the plan's dtype):
 *   prefill q, o         [batch, n_tokens, num_q_heads,  head_dim]
 *   prefill k, v, k_new  [batch, n_tokens, num_kv_heads, head_dim]
 *   decode q, o          [batch, num_q_heads, head_dim]
 *   k_cache, v_cache     [batch, R, head_dim] with R = offset[num_kv_heads];
 *                        KV head g owns rows [offset[g], offset[g] + C_g).
 *   pos_cache            int32 [batch, R]: position held by each slot, -1 if
 *                        empty.  The caller fills it with -1 before the
 *                        first append.
 *   Query head h uses KV head h / (num_q_heads / num_kv_heads).
 *
 * Ownership: the caller owns every device buffer (inputs, outputs, caches,
 * pos_cache, decode workspace).  A plan owns only host memory; it holds no
 * device memory and may be shared by threads for reading.  moa_prefill,
 * moa_kv_append and moa_decode allocate nothing.
 *
 * Streams: every GPU call only enqueues kernels on `hip_stream` (a
 * hipStream_t; NULL = the null stream) and returns without synchronizing.
 * Device pointers must belong to the current HIP device.
 *
 * Errors: arguments are validated on the host before anything is launched; a
 * failed validation returns MOA_ERR_INVALID_ARG / MOA_ERR_UNSUPPORTED /
 * MOA_ERR_WORKSPACE and launches nothing.  A failed launch returns
 * MOA_ERR_HIP.  moa_last_error() returns a thread-local message for the last
 * non-OK status of the calling thread.  Faults inside kernels surface at the
 * caller's next synchronization, as for any HIP kernel.
 */
#ifndef MOA_H_
#define MOA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOA_OK = 0,
  MOA_ERR_INVALID_ARG = 1,   /* null pointer, bad size, protocol violation */
  MOA_ERR_UNSUPPORTED = 2,   /* valid but not implemented (head_dim, group size, ...) */
  MOA_ERR_WORKSPACE = 3,     /* decode workspace missing or too small */
  MOA_ERR_HIP = 4            /* a HIP launch or runtime call failed */
} moa_status_t;

typedef enum {
  MOA_F32 = 0,               /* fp32 in, fp32 accumulate, fp32 out */
  MOA_BF16 = 1               /* bf16 in, fp32 accumulate, bf16 out (round to nearest even) */
} moa_dtype_t;

/* Largest supported head counts (the per-head tables travel as kernel arguments). */
#define MOA_MAX_KV_HEADS 64
#define MOA_MAX_Q_HEADS 512

/* Attention-layer descriptor.  Supported: head_dim in {64, 128};
 * num_q_heads % num_kv_heads == 0 with group size in {1, 2, 4, 8};
 * 0 <= num_sink; 1 <= n < 2^30 ("n" is the input length N at which the
 * elastic rule is evaluated; windows stay fixed afterwards, during decode). */
typedef struct {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t num_sink;
  int64_t n;
  int32_t dtype;             /* moa_dtype_t */
  float softmax_scale;       /* 0 => 1/sqrt(head_dim) */
  uint32_t flags;            /* MOA_SPAN_INCLUDES_SINKS | MOA_BLOCK_BAND, or 0 */
  uint32_t reserved;         /* must be 0 */
} moa_desc_t;

#define MOA_SPAN_INCLUDES_SINKS 1u
#define MOA_BLOCK_BAND 2u
#define MOA_BAND_BLOCK 64

typedef struct moa_plan_s moa_plan_t;

/* Builds the per-KV-head tables for one layer (paper Sec. 3.2, Eq. 2: span
 * alpha + beta * N per head; clipping per Appendix "Main Setup").
 * alpha, beta: host arrays of num_kv_heads finite doubles.  On success *out
 * receives a new plan (free it with moa_plan_free).  Host only: runs without
 * a GPU. */
moa_status_t moa_plan(const moa_desc_t* desc, const double* alpha, const double* beta,
                      moa_plan_t** out);

/* Copies the plan's tables to caller-owned host arrays (any may be NULL):
 * window[num_kv_heads], capacity[num_kv_heads], offset[num_kv_heads + 1]
 * (offset[g] = sum of capacities of heads < g; offset[num_kv_heads] = R). */
moa_status_t moa_plan_tables(const moa_plan_t* plan, int32_t* window, int32_t* capacity,
                             int64_t* offset);

/* Releases a plan (NULL is allowed). */
void moa_plan_free(moa_plan_t* plan);

/* Prefill attention (paper Sec. 2.1, Eq. 1, masked per KV head by the
 * Sec. 3.2 span): for every batch b, query head h and position i < n_tokens,
 *   o[b,i,h,:] = sum_{j visible to i} softmax_j(scale * q[b,i,h,:].k[b,j,g,:]) v[b,j,g,:]
 * with g the KV head of h.  q, k, v, o: device pointers in the layouts above;
 * o must not overlap the inputs.  Keys outside each head's sink prefix and
 * band are never read.  batch >= 1, 1 <= n_tokens < 2^30. */
moa_status_t moa_prefill(const moa_plan_t* plan, const void* q, const void* k, const void* v,
                         void* o, int32_t batch, int64_t n_tokens, void* hip_stream);

/* Appends positions start_pos .. start_pos + n_new - 1 of every sequence to
 * the per-head static caches (paper Appendix "Efficiency Experiment Setup":
 * a new token takes the slot of the entry that has just left the span).  k_new,
 * v_new: device [batch, n_new, num_kv_heads, head_dim].  Only each slot's
 * final occupant is written (K/V bits copied exactly, pos_cache set to the
 * position), so one bulk append equals n_new single appends.  Protocol:
 * appends start at 0 and are contiguous; all sequences of a batch share
 * start_pos.  1 <= batch <= 65535, start_pos >= 0, n_new >= 1,
 * start_pos + n_new < 2^31. */
moa_status_t moa_kv_append(const moa_plan_t* plan, void* k_cache, void* v_cache,
                           int32_t* pos_cache, const void* k_new, const void* v_new,
                           int32_t batch, int64_t start_pos, int64_t n_new, void* hip_stream);

/* Bytes of device workspace moa_decode needs for `batch` sequences (the
 * maximum over all positions).  Returns 0 for a NULL plan or batch < 1. */
size_t moa_decode_workspace_bytes(const moa_plan_t* plan, int32_t batch);

/* Decode attention for the token at position `pos` of every sequence (paper
 * Appendix "Efficiency Experiment Setup": one query against per-head caches
 * of different lengths).  Must follow moa_kv_append(start_pos = pos,
 * n_new = 1), so that each head's filled slots hold exactly the keys visible
 * to position pos.  q, o: device [batch, num_q_heads, head_dim].
 * workspace: device buffer of ws_bytes >= moa_decode_workspace_bytes(plan,
 * batch), 256-byte aligned, holding split-K partial results; its contents
 * need no initialisation and are meaningless after the call.  Calls that
 * share one workspace must be ordered on one stream.  Neither o nor the
 * workspace may overlap q, the caches or each other (MOA_ERR_INVALID_ARG).
 * Launches one kernel when the whole call fits one work-group, otherwise two
 * (the second merges the partial results of caches split between
 * work-groups). */
moa_status_t moa_decode(const moa_plan_t* plan, const void* q, const void* k_cache,
                        const void* v_cache, void* o, int32_t batch, int64_t pos,
                        void* workspace, size_t ws_bytes, void* hip_stream);

/* Decode for callers that cannot allocate device memory or pass a workspace
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): moa_decode with the split-K partials kept in a workspace that
 * the library owns, a fixed array of MOA_DECODE_SCRATCH_BYTES per GPU
 * (allocated when the library's code is loaded on that device and held until
 * the process ends).  Same arguments, layouts and result as moa_decode, minus
 * the workspace; the call allocates nothing (no hipMalloc, no library that
 * allocates).  Returns MOA_ERR_WORKSPACE, launching nothing, when
 * moa_decode_workspace_bytes(plan, batch) exceeds MOA_DECODE_SCRATCH_BYTES
 * (e.g. head_dim 128 with group 8 allows batch * num_kv_heads <= 7695).
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (other streams, other host threads) race and give wrong
 * results, so order them on one stream.  The array needs no clearing: each
 * partial is written before it is read within the same call. */
#define MOA_DECODE_SCRATCH_BYTES (64u << 20)
moa_status_t moa_decode_noalloc(const moa_plan_t* plan, const void* q, const void* k_cache,
                                const void* v_cache, void* o, int32_t batch, int64_t pos, void* hip_stream);

/* One-token append at per-sequence positions (paper Appendix "Efficiency
 * Experiment Setup": the newest token replaces the oldest entry beyond the
 * span; each sequence of a serving batch may be at its own position).
 * positions: device int32[batch]; sequence b appends the token
 * k_new/v_new[b] (device [batch, 1, num_kv_heads, head_dim]) at position
 * positions[b].  A negative position leaves sequence b untouched.  Each
 * sequence's appends must still be contiguous from 0.  1 <= batch <= 65535. */
moa_status_t moa_kv_append_ragged(const moa_plan_t* plan, void* k_cache, void* v_cache,
                                  int32_t* pos_cache, const void* k_new, const void* v_new,
                                  const int32_t* positions, int32_t batch, void* hip_stream);

/* Decode at per-sequence positions (paper Appendix "Efficiency Experiment
 * Setup": one query against per-head caches of different lengths).  Same as
 * moa_decode with sequence b at position positions[b] (device int32[batch]);
 * must follow moa_kv_append_ragged with the same positions.  A negative
 * position skips sequence b (its output is not written).  The workspace rules
 * of moa_decode apply (moa_decode_workspace_bytes covers any positions).
 * Launches two kernels (the second merges split-K partial results). */
moa_status_t moa_decode_ragged(const moa_plan_t* plan, const void* q, const void* k_cache,
                               const void* v_cache, void* o, const int32_t* positions, int32_t batch,
                               void* workspace, size_t ws_bytes, void* hip_stream);

/* Attention-influence profile of dense causal attention (paper Sec. 3.3
 * "Attention Influence Profiling", Eq. 3; Appendix "Derivation of Attention
 * Influence"; 64-token block granularity per Appendix "Main Setup").
 * For each calibration item b and query head h, with A = softmax(scale *
 * Q K^T) under the causal mask, O = A V and the gradient dout = dL/dO of some
 * loss L, dL/dA = dout V^T and the influence of masking A_ij is
 *   E_ij = -A_ij / (1 - A_ij) * (G_ij - sum_n G_in A_in),   G = dL/dA
 * (0 where A_ij is 0 or rounds to 1 in fp32).  Writes the mean of E over the
 * batch and over each 64 x 64 block (edge blocks: over the entries that
 * exist; blocks above the diagonal are 0):
 *   ebar  fp32 [num_q_heads, nb, nb], nb = ceil(n / 64), caller-owned device.
 * q, dout  [batch, n, num_q_heads,  head_dim]  (bf16, 16-byte aligned)
 * k, v     [batch, n, num_kv_heads, head_dim]  (bf16, 16-byte aligned)
 * desc: the layer (num_q_heads, num_kv_heads, head_dim, softmax_scale; dtype
 * must be MOA_BF16; num_sink, n and flags are ignored: the profiled
 * attention is dense).  1 <= n <= 65536, batch >= 1.  Allocates nothing;
 * one kernel launch; the result does not depend on the launch order. */
moa_status_t moa_influence(const moa_desc_t* desc, const void* q, const void* k, const void* v,
                           const void* dout, float* ebar, int32_t batch, int64_t n, void* hip_stream);

/* Rule-loss table (paper Sec. 3.3, Eq. 4): the accuracy loss of giving head h
 * candidate rule r at length n is its block-averaged influence summed over the
 * causal pairs the rule masks,
 *   dl[h][r] = sum over i, j with j <= i of M_r(i, j) * ebar[h][i / 64][j / 64],
 * M_r(i, j) = 1 iff rule r's mask (window from (alpha[r], beta[r]) at length n
 * exactly as moa_plan evaluates it under `flags`, num_sink sinks, token or
 * MOA_BLOCK_BAND band) hides key j from query i.  density[r] is rule r's
 * in-memory KV-cache length over the sequence length during decoding (paper
 * Sec. 4 "Setups"): min(num_sink + w_r, n) / n, the share of the n tokens
 * that its token-exact cache holds (the block band does not change it).
 * ebar   fp32 device [num_heads, nb, nb], nb = ceil(n / 64) (moa_influence output)
 * dl     fp64 device [num_heads, num_rules];  density fp64 device [num_rules]
 * alpha, beta: host arrays of num_rules finite doubles; 1 <= num_rules <= 64;
 * 1 <= n <= 65536.  fp64 sums (exact masked-pair counts in closed form).
 * Allocates nothing; one kernel launch. */
moa_status_t moa_rule_loss(const float* ebar, int32_t num_heads, int64_t n, int32_t num_sink, uint32_t flags,
                           const double* alpha, const double* beta, int32_t num_rules, double* dl,
                           double* density, void* hip_stream);

/* Thread-local message of the calling thread's last non-OK status ("" if none). */
const char* moa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MOA_H_ */
