/*
 * rl_kernels.h - C ABI of librlkern.so, the MI355X (gfx950) rollout hot path.
 *
 * Operations, all asynchronous on a caller-supplied HIP stream:
 *
 *  rl_decode_attn     one grouped-query decode step for a batch of prompts,
 *                     each with a group of G sampled candidates (Sec. 2.2.1,
 *                     Problem Setup: every input x gets g candidates).  The
 *                     candidates of a prompt share its prefix KV (the prompt,
 *                     including the refinement-turn feedback and summary of
 *                     Sec. 3, Structured Feedback and Iterative Refinement) and
 *                     each has its own suffix KV (its generated tokens, at most
 *                     1536 per turn in Sec. 3, Multi-turn RL Training).
 *
 *  rl_extend_attn     the prefill of a refinement turn: each candidate's new
 *                     tokens (the feedback and summary appended to its
 *                     context, Sec. 3, Structured Feedback and Iterative
 *                     Refinement) attend causally to the prompt's shared
 *                     prefix and to the candidate's suffix up to themselves.
 *
 *  rl_kv_append       writes new tokens' keys and values after each
 *                     candidate's suffix in place (the decode loop's cache
 *                     update).
 *
 *  rl_token_logprob   log pi(o_t | q, o_<t) of each sampled token under the
 *                     policy, the factor of the GRPO ratio (Sec. 3, Eq.
 *                     grpo-loss), computed from the last hidden state and the
 *                     lm-head weight over the full vocabulary without storing
 *                     the logits; masked positions (Sec. 3, Multi-turn RL
 *                     Training: masked log-probabilities) give 0.
 *
 *  rl_token_logprob_backward
 *                     d logprob / d hidden through the lm-head, scaled by
 *                     the incoming gradient per row (the policy update's
 *                     backward through the token log-probs, Sec. 3).
 *
 *  rl_sample_top_p    the next token of each row by nucleus sampling at a
 *                     per-row temperature (Sec. 3, Multi-turn RL Training),
 *                     through the lm-head.
 *
 *  rl_grpo_advantage  group-relative advantages of the candidates' rewards
 *                     (Sec. 3, the definition under Eq. grpo-loss).
 *
 *  rl_grpo_surrogate  the clipped GRPO surrogate of Eq. grpo-loss (beta = 0)
 *                     over a batch of token rows, and its gradient with
 *                     respect to the new policy's log-probs.
 *
 * Plain C: no HIP or torch types.  `stream` is a hipStream_t passed as void*
 * (NULL = the default stream).  "device" pointers must be device memory of the
 * current HIP device; "host" pointers are read only during the call.
 *
 * Ownership: the caller owns every buffer, including the workspace.  The
 * library allocates no device memory (rl_token_logprob_noalloc's static
 * array aside).  Across calls it keeps only per-thread state: the last error
 * string, a reusable planning buffer and up to 64 pinned, device-mapped host
 * buffers that a small kernel on the caller's stream copies a work list from
 * (rl_decode_attn, rl_extend_attn and rl_kv_append upload one per call).
 * Buffers are added and enlarged on demand and never freed: an outgrown
 * buffer is kept and one at least twice its size taken.  Such a call does not
 * wait for the stream unless 64 earlier ones on the same thread still wait
 * for the kernel that reads their buffer to run; it then waits for the oldest
 * of them, for at most 60 s, and returns RL_ERR_HIP if it has not run by
 * then.  Calls on different streams need distinct workspaces.
 *
 * Errors: rl_last_error() describes the problem of a failing call.  Argument
 * errors are detected on the host before any launch: a call that returns
 * any status but RL_OK or RL_ERR_HIP has enqueued nothing and written no
 * output.  RL_ERR_HIP reports a failed kernel launch; launches of the same
 * call before it may already be enqueued.  RL_OK means the work is
 * enqueued: outputs are valid after the stream is synchronised, and inputs,
 * outputs and workspace must stay alive until then.
 */
#ifndef RL_KERNELS_H
#define RL_KERNELS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RL_ABI_VERSION 13

typedef enum {
    RL_OK = 0,
    RL_ERR_NULL_POINTER = 1,   /* a required pointer is NULL */
    RL_ERR_INVALID_SHAPE = 2,  /* sizes, lengths or ranges are inconsistent */
    RL_ERR_UNSUPPORTED = 3,    /* valid, but outside what the kernels implement */
    RL_ERR_MISALIGNED = 4,     /* a device pointer is not 16-byte aligned */
    RL_ERR_WORKSPACE = 5,      /* workspace NULL or smaller than required */
    RL_ERR_HIP = 6             /* the HIP runtime reported an error */
} rl_status;

/* ------------------------------------------------------------------------ */
/* Decode attention                                                          */
/* ------------------------------------------------------------------------ */

typedef struct {
    int32_t num_prompts;   /* P >= 0: prompts (inputs x) in the batch                     */
    int32_t group_size;    /* G >= 1: candidates per prompt; sequence s = p*G + g          */
    int32_t num_q_heads;   /* Hq >= 1                                                      */
    int32_t num_kv_heads;  /* Hkv >= 1, Hq % Hkv == 0; query head h reads kv head
                              h / (Hq/Hkv) (consecutive query heads share a kv head)       */
    int32_t head_dim;      /* D: 64 or 128                                                 */
    float   softmax_scale; /* finite, > 0; scores are softmax_scale * <q, k>               */
    int32_t split_tokens;  /* 0 = automatic; else the largest number of KV tokens one
                              split-K work item covers (a multiple of 16, >= 16).  Results
                              agree across splits to rounding, and are bitwise
                              reproducible for a fixed split.                              */
    int32_t kv_layout;     /* RL_KV_TOKEN_MAJOR or RL_KV_HEAD_MAJOR (all four KV tensors)  */
} rl_decode_shape;

/* KV cache layouts.  Token-major keeps the kv heads of a token together; head-major
 * keeps each kv head's rows contiguous, so one (sequence, kv head) streams as one
 * contiguous range (the faster layout on MI355X). */
#define RL_KV_TOKEN_MAJOR 0   /* [rows, Hkv, D] */
#define RL_KV_HEAD_MAJOR 1    /* [Hkv, rows, D] */

typedef struct {
    const int64_t *prefix_start; /* host [P]:   first KV row of prompt p's prefix           */
    const int32_t *prefix_len;   /* host [P]:   Lp[p] >= 0 tokens                           */
    const int64_t *suffix_start; /* host [P*G]: first KV row of candidate s's suffix        */
    const int32_t *suffix_len;   /* host [P*G]: Ls[s] >= 0 tokens                           */
    int64_t prefix_rows;         /* rows allocated in k_prefix/v_prefix (range checks)      */
    int64_t suffix_rows;         /* rows allocated in k_suffix/v_suffix                     */
} rl_decode_lens;

typedef struct {
    const void *q;        /* device bf16 [P*G, Hq, D], contiguous                          */
    const void *k_prefix; /* device bf16 [prefix_rows, Hkv, D] or [Hkv, prefix_rows, D]    */
    const void *v_prefix; /* device bf16, same layout as k_prefix                          */
    const void *k_suffix; /* device bf16 [suffix_rows, Hkv, D] or [Hkv, suffix_rows, D]    */
    const void *v_suffix; /* device bf16, same layout as k_suffix                          */
    void  *out;           /* device bf16 [P*G, Hq, D]: softmax-weighted sum of values,
                             rounded to nearest even; 0 for an empty context               */
    float *lse;           /* device fp32 [P*G, Hq] natural-log log-sum-exp of the scaled
                             scores (-inf for an empty context), or NULL                   */
} rl_decode_ptrs;

/*
 * Attention of candidate s = p*G + g, query head h, over the concatenated
 * context: prefix rows [prefix_start[p], +Lp[p]) followed by suffix rows
 * [suffix_start[s], +Ls[s]), both at kv head h / (Hq/Hkv).  The caller appends
 * the current token's K/V to the suffix before the call; there is no causal
 * mask inside one decode step.  The prefix KV of a prompt is read once for all
 * G candidates when G*Hq/Hkv <= 64 (query rows per kv head); wider groups take
 * one work item per block of 64 such rows on the same chunk, launched side by
 * side, so the repeated reads mostly hit the last-level cache.
 *
 * Rows outside the given ranges are never read.  P*G == 0 is a valid no-op.
 * Status: NULL pointer -> RL_ERR_NULL_POINTER; negative sizes or lengths,
 * Hq % Hkv != 0, a range past prefix_rows/suffix_rows, a non-finite or
 * non-positive scale, a bad split_tokens or kv_layout -> RL_ERR_INVALID_SHAPE;
 * D not in {64, 128}, Hq/Hkv > 128, Hkv > 256, G*Hq/Hkv > 16384, or
 * prefix_rows / suffix_rows of 2^32 or more -> RL_ERR_UNSUPPORTED (the work
 * list uploaded on every call packs these into 16 bytes per item); a device
 * pointer not 16-byte aligned -> RL_ERR_MISALIGNED; workspace NULL or short ->
 * RL_ERR_WORKSPACE.  A split_tokens above 16384 acts as 16384.
 *
 * The workspace holds the work list (16 bytes per item, 8 bytes per prompt and
 * per candidate) and the split partials (max, sum and D fp32 values per
 * query row of each item).
 */
rl_status rl_decode_attn_workspace_size(const rl_decode_shape *shape,
                                        const rl_decode_lens *lens,
                                        size_t *bytes);

rl_status rl_decode_attn(const rl_decode_shape *shape, const rl_decode_lens *lens,
                         const rl_decode_ptrs *ptrs,
                         void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* Extend (prefill) attention of a refinement turn                           */
/* ------------------------------------------------------------------------ */

/*
 * Each refinement turn appends structured feedback (and a summary of the
 * earlier turns) to a candidate's context before the policy generates again
 * (Sec. 3, Structured Feedback and Iterative Refinement); the policy first
 * reads those new tokens in one pass.  Candidate s = p*G + g has the context
 * prefix(p) followed by suffix(s); the last new_len[s] tokens of its suffix
 * are new, their K/V already in the cache.  New token i (0 <= i < n = new_len[s])
 * is at suffix position Ls[s] - n + i and attends, at query head h and kv head
 * h / (Hq/Hkv), to every prefix token and to suffix positions 0 .. Ls[s] - n + i
 * (itself included): the causal mask of a prefill.  Its query and its output
 * are row q_start[s] + i of q / out ([q_rows, Hq, D] bf16, contiguous), its
 * log-sum-exp lse[(q_start[s] + i) * Hq + h] (fp32, natural log; lse may be
 * NULL).  Rows of q / out that belong to no candidate are not written.
 * With every new_len = 1 this is rl_decode_attn's result.
 *
 * The shape and the KV tensors are those of rl_decode_attn (both kv layouts;
 * split_tokens is not used).  Work is cut into blocks of 256 query rows (token
 * x query head of one candidate and kv head), each streaming its visible
 * context through LDS; blocks of one prompt run together so its prefix is read
 * from HBM about once per XCD.  The workspace holds the work list (48 bytes per
 * block).
 *
 * Status: NULL pointers -> RL_ERR_NULL_POINTER; the checks of rl_decode_attn
 * on the shape and the KV ranges, and new_len[s] < 0, new_len[s] > Ls[s], a
 * query range outside [0, q_rows), or two candidates sharing a query row ->
 * RL_ERR_INVALID_SHAPE; head_dim not in {64, 128} -> RL_ERR_UNSUPPORTED; a
 * device pointer not 16-byte aligned -> RL_ERR_MISALIGNED; workspace NULL or
 * short -> RL_ERR_WORKSPACE.  No new tokens is a valid no-op.
 */
typedef struct {
    const int64_t *prefix_start; /* host [P]:   first KV row of prompt p's prefix           */
    const int32_t *prefix_len;   /* host [P]:   Lp[p] >= 0                                  */
    const int64_t *suffix_start; /* host [P*G]: first KV row of candidate s's suffix        */
    const int32_t *suffix_len;   /* host [P*G]: Ls[s] >= 0 tokens, the new ones included     */
    const int32_t *new_len;      /* host [P*G]: 0 <= n[s] <= Ls[s] new tokens at its end     */
    const int64_t *q_start;      /* host [P*G]: row of s's first new token in q / out / lse */
    int64_t prefix_rows;         /* rows allocated in k_prefix / v_prefix                   */
    int64_t suffix_rows;         /* rows allocated in k_suffix / v_suffix                   */
    int64_t q_rows;              /* rows of q and out                                       */
} rl_extend_lens;

rl_status rl_extend_attn_workspace_size(const rl_decode_shape *shape, const rl_extend_lens *lens,
                                        size_t *bytes);

/* ptrs: q / out are [q_rows, Hq, D], lse [q_rows, Hq] or NULL; the KV pointers
 * as for rl_decode_attn. */
rl_status rl_extend_attn(const rl_decode_shape *shape, const rl_extend_lens *lens,
                         const rl_decode_ptrs *ptrs, void *workspace, size_t workspace_bytes,
                         void *stream);

/* ------------------------------------------------------------------------ */
/* Appending to the suffix KV cache                                          */
/* ------------------------------------------------------------------------ */

/*
 * A rollout adds one token per candidate per decode step (up to 1536
 * generated tokens per turn, Sec. 3, Multi-turn RL Training).  rl_kv_append
 * writes the new tokens' keys and values after each candidate's suffix in
 * place, so a cache with a region of fixed capacity per candidate grows
 * without repacking.  For candidate s and i < new_len[s], at every kv head:
 *   suffix row suffix_start[s] + suffix_len[s] + i  <-  row new_start[s] + i
 *   of k_new / v_new,
 * in the cache layout shape->kv_layout.  k_new and v_new are token-major
 * [new_rows, Hkv, D] bf16.  The suffix of s is then suffix_len[s] + new_len[s]
 * tokens long; the caller keeps the lengths.  Only num_prompts, group_size,
 * num_kv_heads, head_dim and kv_layout of the shape are used.
 */
typedef struct {
    const int64_t *suffix_start;    /* host [P*G]: first row of candidate s's region      */
    const int32_t *suffix_len;      /* host [P*G]: tokens already there                   */
    const int32_t *suffix_capacity; /* host [P*G]: rows reserved for s, or NULL (then only
                                       suffix_rows bounds the writes)                    */
    const int64_t *new_start;       /* host [P*G]: first row of s's new tokens in k_new   */
    const int32_t *new_len;         /* host [P*G] >= 0: tokens to append                  */
    int64_t suffix_rows;            /* rows allocated in k_suffix / v_suffix              */
    int64_t new_rows;               /* rows of k_new / v_new                              */
} rl_kv_append_lens;

/*
 * The workspace holds the (source, destination) row pairs, 16 bytes per new
 * token.  Status: NULL pointer -> RL_ERR_NULL_POINTER; negative lengths or
 * starts, a write past suffix_rows or past a candidate's capacity, a source
 * range past new_rows, or two candidates writing the same row ->
 * RL_ERR_INVALID_SHAPE; head_dim not in {64, 128} or a bad kv_layout ->
 * RL_ERR_UNSUPPORTED / RL_ERR_INVALID_SHAPE; a tensor not 16-byte aligned ->
 * RL_ERR_MISALIGNED; workspace NULL or short -> RL_ERR_WORKSPACE.  No new
 * tokens is a valid no-op.
 */
rl_status rl_kv_append_workspace_size(const rl_decode_shape *shape, const rl_kv_append_lens *lens,
                                      size_t *bytes);

rl_status rl_kv_append(const rl_decode_shape *shape, const rl_kv_append_lens *lens,
                       const void *k_new, const void *v_new, void *k_suffix, void *v_suffix,
                       void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* Token log-prob through the lm-head                                        */
/* ------------------------------------------------------------------------ */

/*
 * For each row r:  z_v = inv_temperature * <hidden[r, :], w_lm[v, :]>  (v < V),
 *                  lse[r] = ln sum_v exp(z_v),
 *                  logprob[r] = z_t - lse[r]  for t = target[r] in [0, V),
 *                             = 0             for t == -1 (masked position),
 *                             = NaN           for any other t (lse is still computed).
 * The [rows, V] logits are never written to memory.
 *
 *   hidden_states  device bf16 [rows, hidden], contiguous
 *   w_lm           device bf16 [vocab, hidden], contiguous (row v gives logit v)
 *   target         device int32 [rows]
 *   inv_temperature finite, > 0 (1.0 for the plain policy)
 *   logprob        device fp32 [rows]
 *   lse            device fp32 [rows], or NULL
 *
 * rows == 0 is a valid no-op.  Status: NULL pointer -> RL_ERR_NULL_POINTER;
 * rows < 0, hidden <= 0, vocab <= 0 or a bad temperature -> RL_ERR_INVALID_SHAPE;
 * hidden % 64 != 0 or hidden > 4194304 -> RL_ERR_UNSUPPORTED; a device
 * pointer not 16-byte aligned (target, logprob and lse: 4-byte) ->
 * RL_ERR_MISALIGNED; workspace NULL or short -> RL_ERR_WORKSPACE.
 *
 * The workspace holds a (max, sum) partial per (vocab tile, row) and the
 * target logit per row.  When the last round of 256 x 256 tiles would leave
 * at least half of the 256 CUs idle, those tiles run as 2-4 parts of the
 * hidden dimension and the workspace also holds their fp32 accumulators
 * (256 KB per part).  When it is more than half full and there are at most 4
 * row tiles, the vocabulary past the full rounds runs as one round of tiles
 * 128 or 192 entries wide instead (the narrower that fits; none if neither
 * does), each with its own partial slot.
 */
rl_status rl_token_logprob_workspace_size(int64_t rows, int32_t hidden, int32_t vocab,
                                          size_t *bytes);

rl_status rl_token_logprob(int64_t rows, int32_t hidden, int32_t vocab,
                           const void *hidden_states, const void *w_lm,
                           const int32_t *target, float inv_temperature,
                           float *logprob, float *lse,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * rl_token_logprob without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  It calls no hipMalloc, hipFree or other
 * allocating routine.  The workspace rl_token_logprob_workspace_size reports
 * lives instead in a static device array of RL_NOALLOC_SCRATCH_BYTES
 * (128 MiB), one per GPU the library runs on, held until the process ends;
 * its address is looked up once per device on the first call there.  Sizes
 * whose workspace exceeds it return RL_ERR_UNSUPPORTED before any launch
 * (the decode-step shapes fit; at a 151936-entry vocabulary, rows up to about
 * 28000 when no hidden-split tail is planned); the other arguments, results,
 * statuses and kernels are rl_token_logprob's.  Every call on one GPU shares
 * that GPU's array: calls whose executions overlap on one GPU (other
 * streams, or other threads) race and give wrong results; calls in order on
 * one stream are safe.  Nothing in the array needs clearing between calls.
 */
#define RL_NOALLOC_SCRATCH_BYTES (128u << 20)
rl_status rl_token_logprob_noalloc(int64_t rows, int32_t hidden, int32_t vocab,
                                   const void *hidden_states, const void *w_lm,
                                   const int32_t *target, float inv_temperature,
                                   float *logprob, float *lse, void *stream);

/*
 * Backward of rl_token_logprob with respect to the hidden rows, for the
 * policy update through a frozen lm-head (Sec. 3, Eq. grpo-loss: the token
 * ratio's gradient reaches the policy through log pi; the lm-head weight
 * itself is not trained).  With p_v = exp(z_v - lse[r]) (z as above):
 *   grad_hidden[r, :] = grad_logprob[r] * inv_temperature
 *                       * (w_lm[t, :] - sum_v p_v w_lm[v, :])   t = target[r] in [0, V),
 *                     = 0                                       t == -1,
 *                     = NaN                                     any other t.
 * The logits are recomputed; p is held in the workspace as bf16, one chunk
 * of at most 16384 rows at a time, and never returned.
 *
 *   hidden_states, w_lm, target, inv_temperature   as for rl_token_logprob
 *   lse            device fp32 [rows], the lse rl_token_logprob returned for
 *                  the same inputs (read only for rows with a valid target)
 *   grad_logprob   device fp32 [rows], d loss / d logprob[r]
 *   grad_hidden    device fp32 [rows, hidden], written (not accumulated)
 *
 * The workspace holds chunk_rows x vocab (padded to 256) bf16 probabilities
 * plus one fp32 section used in turn by the hidden-dimension parts of the
 * last round of probability tiles (when that round would leave at least
 * half of the CUs idle) and, when rows are few, by the partial sums of a
 * vocabulary split; its size depends on (rows, hidden, vocab) only.  w_lm must be finite.  rows == 0 is
 * a valid no-op.  Status: as rl_token_logprob; hidden_states, w_lm and
 * grad_hidden 16-byte aligned, target, lse and grad_logprob 4-byte aligned.
 */
rl_status rl_token_logprob_backward_workspace_size(int64_t rows, int32_t hidden, int32_t vocab,
                                                   size_t *bytes);

rl_status rl_token_logprob_backward(int64_t rows, int32_t hidden, int32_t vocab,
                                    const void *hidden_states, const void *w_lm,
                                    const int32_t *target, float inv_temperature,
                                    const float *lse, const float *grad_logprob,
                                    float *grad_hidden,
                                    void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* Nucleus (top-p) sampling head (Sec. 3, Multi-turn RL Training)            */
/* ------------------------------------------------------------------------ */

/*
 * Draws the next token of each row: candidates are sampled with nucleus
 * sampling at a temperature (the paper: p = 0.9, temperatures 0.2 and 0.7).
 * With y_v = inv_temperature[r] * <hidden[r, :], w_lm[v, :]> and p = softmax(y):
 *   - tokens are ranked by p, largest first, equal p by the smaller id;
 *   - the nucleus N is the shortest ranked prefix whose mass reaches top_p;
 *   - token[r] is the smallest id t in N whose nucleus mass in id order,
 *     sum_{v in N, v <= t} p_v, exceeds uniform[r] * sum_{v in N} p_v.
 * logprob[r] (if not NULL) is y_t - ln sum_v exp(y_v), the token's log-prob
 * under the full tempered softmax.
 *
 * Precision: the logits are fp32 (bf16 MFMA, fp32 accumulation) and the
 * probabilities are integer masses floor(2^40 exp(y_v - max y)), so all sums
 * are exact and the result is deterministic; a token whose mass rounds to 0
 * (p_v below 2^-40 of the most probable) is never drawn.
 *
 *   hidden_states, w_lm   as for rl_token_logprob
 *   inv_temperature  device fp32 [rows], 1/T per row (finite, > 0: not
 *                    checked, device memory)
 *   top_p            in (0, 1]
 *   uniform          device fp32 [rows], one draw in [0, 1) per row, from the
 *                    caller's generator (values outside are clamped into
 *                    the nucleus)
 *   token            device int32 [rows]
 *   logprob          device fp32 [rows], or NULL
 *
 * The workspace holds the tempered fp32 logits of up to 8192 rows at a time
 * (rows x vocab padded to 256) and their per-tile maxima; no logits are
 * returned.  rows == 0 is a valid no-op.  Status: NULL pointer ->
 * RL_ERR_NULL_POINTER; bad sizes or top_p -> RL_ERR_INVALID_SHAPE; hidden %
 * 64 != 0 or vocab > 2^21 -> RL_ERR_UNSUPPORTED; hidden_states, w_lm and the
 * workspace not 16-byte aligned, the other pointers not 4-byte aligned ->
 * RL_ERR_MISALIGNED; workspace NULL or short -> RL_ERR_WORKSPACE.
 */
rl_status rl_sample_top_p_workspace_size(int64_t rows, int32_t hidden, int32_t vocab, size_t *bytes);

rl_status rl_sample_top_p(int64_t rows, int32_t hidden, int32_t vocab,
                          const void *hidden_states, const void *w_lm,
                          const float *inv_temperature, float top_p, const float *uniform,
                          int32_t *token, float *logprob,
                          void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* GRPO advantages and clipped surrogate (Sec. 3, Eq. grpo-loss)             */
/* ------------------------------------------------------------------------ */

/*
 * For each prompt p's group of G candidates s = p*G + g with rewards r_s:
 *   adv[s] = (r_s - mean_g r) / std_g r,
 * std the sample standard deviation (divisor G - 1); a group whose rewards
 * are all equal, or G == 1, gets adv = 0.
 *
 *   reward, adv    device fp32 [num_prompts * group_size]
 *
 * num_prompts == 0 is a valid no-op.  Status: NULL pointer ->
 * RL_ERR_NULL_POINTER; num_prompts < 0 or group_size < 1 ->
 * RL_ERR_INVALID_SHAPE; group_size > 1024 -> RL_ERR_UNSUPPORTED; a pointer not
 * 4-byte aligned -> RL_ERR_MISALIGNED.
 */
rl_status rl_grpo_advantage(int64_t num_prompts, int32_t group_size, const float *reward, float *adv,
                            void *stream);

/*
 * Over token rows r = 0 .. rows-1, each belonging to candidate seq[r] of the
 * S = num_prompts * group_size candidates (seq[r] = -1: the row belongs to no
 * candidate and is ignored), with rho_r = exp(logp_new[r] - logp_old[r]):
 *   loss = -(1/(num_prompts * G)) * sum_s (1/|o_s|)
 *          * sum_{r: seq[r] = s} min(rho_r adv[s], clip(rho_r, 1-eps, 1+eps) adv[s]),
 * |o_s| the number of rows of candidate s.  grad[r] = dloss/dlogp_new[r]:
 * -(1/(num_prompts * G |o_s|)) rho_r adv[s] where the ratio term is the minimum
 * (ties included), 0 where the clipped term is smaller, 0 for ignored rows.
 *
 *   logp_new, logp_old  device fp32 [rows]
 *   seq                 device int32 [rows], in [-1, S)
 *   adv                 device fp32 [S]
 *   eps                 clip range, finite, in [0, 1) (the paper uses 0.2)
 *   loss                device fp32, one value
 *   grad                device fp32 [rows]
 *
 * The loss is summed in a fixed order (bitwise reproducible).  rows == 0 or
 * num_prompts == 0 writes loss 0.  Status: NULL pointer -> RL_ERR_NULL_POINTER;
 * negative sizes, group_size < 1 or a bad eps -> RL_ERR_INVALID_SHAPE; a
 * pointer not 4-byte aligned -> RL_ERR_MISALIGNED; workspace NULL or short ->
 * RL_ERR_WORKSPACE.  A seq value outside [-1, S) is not checked on the host;
 * such a row is ignored.
 */
rl_status rl_grpo_surrogate_workspace_size(int64_t rows, int64_t num_prompts, int32_t group_size,
                                           size_t *bytes);

rl_status rl_grpo_surrogate(int64_t rows, int64_t num_prompts, int32_t group_size,
                            const float *logp_new, const float *logp_old, const int32_t *seq,
                            const float *adv, float eps, float *loss, float *grad,
                            void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* Diagnostics                                                               */
/* ------------------------------------------------------------------------ */

const char *rl_status_string(rl_status status); /* static text, never NULL          */
const char *rl_last_error(void);                /* thread-local detail of the last
                                                   failing call on this thread, ""
                                                   if none; valid until the next call */
int rl_abi_version(void);                       /* RL_ABI_VERSION                     */

/*
 * Host-only view of the split-K work list rl_decode_attn would launch for
 * these arguments (no device access; for tests and tuning).  Each item covers
 * tokens [tok_begin, tok_begin + tok_count) of one unit: the prefix of prompt
 * `unit` (kind 0) or the suffix of candidate `unit` (kind 1), at one kv head.
 * Writes at most `capacity` items and sets *num_items to the full count.
 */
typedef struct {
    int32_t kind;        /* 0 = prefix of prompt `unit`, 1 = suffix of candidate `unit` */
    int32_t unit;
    int32_t kv_head;
    int32_t chunk;       /* index of this chunk within its (unit, kv_head)              */
    int64_t tok_begin;   /* first token of the chunk, relative to the unit's start      */
    int32_t tok_count;   /* >= 1                                                        */
    int32_t row_begin;   /* first query row served, of the unit's G*Hq/Hkv (prefix) or
                            Hq/Hkv (suffix) rows at this kv head                         */
    int32_t row_count;   /* query rows served: at most 64                                */
    int32_t split_variant; /* split kernel the call launches, the same in every item: 0 = one
                              KV tile in flight per workgroup, 1 = two (chosen when items of
                              more than 48 query rows hold most of the KV tokens)          */
} rl_plan_item;

rl_status rl_decode_plan_debug(const rl_decode_shape *shape, const rl_decode_lens *lens,
                               rl_plan_item *items, int64_t capacity, int64_t *num_items);

/*
 * Host-only replay of the global memory accesses that rl_token_logprob
 * (op = 0), rl_token_logprob_backward (op = 1) or rl_sample_top_p (op = 2)
 * would make for these sizes:
 * every launch of the call, every workgroup and lane, with the kernel
 * arguments the entry point builds and the kernels' own index arithmetic;
 * each load and store is checked against the allocation (or workspace
 * section) it must fall in, sized as the entry point requires.  No device
 * access; for tests.  Staged loads are checked at the first and last stage
 * (each address is affine and non-decreasing in the stage), or at every
 * stage when every_stage != 0.  shrink_region >= 0 makes that allocation or
 * section (numbered in the order listed below) 16 bytes smaller than the
 * entry point requires, to test the checker: every one that the kernels use
 * up to its last byte must then report a violation.  Regions: op 0: hidden,
 * w_lm, target, logprob, lse, workspace, and the workspace's partial max,
 * partial sum, target logit and tail part sections; op 1: hidden, w_lm,
 * target, lse, grad_logprob, grad_hidden, workspace, and the workspace's
 * probability section and (when a tail or a GEMM is split) the section of
 * tail parts and split sums; op 2: hidden, w_lm, inv_temperature, uniform,
 * token, logprob, workspace, and the workspace's logits and row-maximum
 * sections (the selection kernel's data-dependent reads are checked over
 * the whole range it may touch).  Returns the plan's
 * status for invalid sizes, RL_ERR_NULL_POINTER for a NULL report and
 * RL_ERR_INVALID_SHAPE for an unknown op; otherwise RL_OK with the counts in
 * *report.
 */
typedef struct {
    uint64_t accesses;          /* lane accesses checked                         */
    uint64_t violations;        /* accesses outside their allocation             */
    int32_t  launches;          /* kernel launches replayed                      */
    int32_t  regions;           /* allocations and sections checked              */
    char     first_violation[256]; /* the first one found, "" if none            */
} rl_bounds_report;

rl_status rl_debug_logprob_bounds(int32_t op, int64_t rows, int32_t hidden, int32_t vocab,
                                  int32_t every_stage, int32_t shrink_region, rl_bounds_report *report);

/*
 * Host-only replay of the global memory accesses that rl_extend_attn would
 * make for this shape and these lengths (Sec. 3, Structured Feedback and
 * Iterative Refinement: the extend of a refinement turn): every work block
 * of the plan, every lane, with the kernel arguments the entry point builds
 * and the kernel's own index arithmetic; each query load, K/V tile load,
 * output and lse store and the read of the block's work item is checked
 * against its allocation, sized from the lengths (q and out [q_rows, Hq, D]
 * bf16, lse [q_rows, Hq] fp32, the prefix and suffix K/V [rows, Hkv, D] bf16
 * in shape->kv_layout, the workspace as rl_extend_attn_workspace_size
 * gives it).  A block's tile loads are checked at the first and last tile of
 * its prefix and of its suffix (each lane's address grows with the tile
 * inside a range and the last tile of a range is the ragged one), or at
 * every tile when every_stage != 0.  shrink_region as for
 * rl_debug_logprob_bounds; regions: q, k_prefix, v_prefix, k_suffix,
 * v_suffix, out, lse, workspace, and the workspace's work-list section.  No
 * device access; for tests.  Returns the plan's status for invalid lengths,
 * RL_ERR_NULL_POINTER for a NULL report; otherwise RL_OK with the counts in
 * *report (all zero when the call has no work).
 */
rl_status rl_debug_extend_bounds(const rl_decode_shape *shape, const rl_extend_lens *lens, int32_t every_stage,
                                 int32_t shrink_region, rl_bounds_report *report);

/*
 * Host-only replay of the global memory accesses that rl_decode_attn would
 * make for this shape and these lengths (Sec. 2.2.1, Problem Setup: decode of
 * a group of candidates over the prompt's shared prefix): the work list's
 * upload, every work item of the split kernel (each tile's buffer descriptor,
 * whose range bounds every lane's load of that tile, the item's query rows
 * and its partial rows) and every (sequence, head) row of the combine (its
 * unit tables, the partials it merges, its output row and lse), with the
 * kernel arguments the entry point builds and the kernels' own index
 * arithmetic.  Allocations are sized from the lengths: q and out [P*G, Hq, D]
 * bf16, lse [P*G, Hq] fp32, the prefix and suffix K/V [rows, Hkv, D] bf16 in
 * shape->kv_layout, the workspace as rl_decode_attn_workspace_size gives
 * it.  shrink_region as for rl_debug_logprob_bounds; regions: q, k_prefix,
 * v_prefix, k_suffix, v_suffix, out, lse, workspace, and the workspace's
 * sections: work list and unit tables (the upload), work list, prefix units,
 * suffix units, partial max, partial sum, partial values.  No device access;
 * for tests.  Returns the plan's status for invalid lengths,
 * RL_ERR_NULL_POINTER for a NULL report; otherwise RL_OK with the counts in
 * *report (all zero when P*G = 0).
 */
rl_status rl_debug_decode_bounds(const rl_decode_shape *shape, const rl_decode_lens *lens, int32_t shrink_region,
                                 rl_bounds_report *report);

/*
 * Debug timeline of rl_token_logprob, to see where a tile's time goes: the
 * same call (arguments, plan, outputs and arithmetic), with the tile
 * launches (whole tiles, narrow tiles of a last round, hidden-dimension parts
 * of tail tiles) built with timestamps.  Each wave of each of those
 * workgroups writes one record of RL_TIMELINE_WORDS uint64 to `records`
 * (device memory, 8-byte aligned, `capacity` records):
 *   [0] HW_ID register | XCC id << 32 | launch (0 whole, 1 narrow,
 *       2 tail part) << 40 | wave << 48
 *   [1] wall clock when the workgroup starts   (s_memrealtime, 100 MHz)
 *   [2] wall clock when its first stage has landed (the loop starts)
 *   [3] wall clock at the end of the loop
 *   [4] wall clock after the epilogue
 *   [5] s_memtime cycles spent in the stage-end waits (the
 *       loads of the next stage, then the workgroup barrier) of the sampled
 *       stages, those whose index is 3 mod 8
 *   [6] s_memtime cycles of the loop (s_memtime counts at a rate of its
 *       own, not the shader clock)
 *   [7] workgroup index | hidden-dimension stages << 32 | sampled stages << 48
 * The tile workgroups have 8 waves: whole-tile workgroup b, wave w writes
 * record 8 b + w; the narrow tiles and then the tail parts follow in the same
 * way.  *num_records gets the number
 * of records the call writes; with records == NULL only that number is
 * computed (no launch, no other pointer checked).  A stamp makes the wave
 * wait for the scalar read that returns it, so the sampled stages run a
 * little slower than rl_token_logprob's.  Status: as rl_token_logprob, plus
 * RL_ERR_NULL_POINTER for a NULL num_records, RL_ERR_WORKSPACE when capacity
 * is short and RL_ERR_MISALIGNED for misaligned records.
 */
#define RL_TIMELINE_WORDS 8
rl_status rl_debug_logprob_timeline(int64_t rows, int32_t hidden, int32_t vocab, const void *hidden_states,
                                    const void *w_lm, const int32_t *target, float inv_temperature,
                                    float *logprob, float *lse, void *workspace, size_t workspace_bytes,
                                    uint64_t *records, int64_t capacity, int64_t *num_records, void *stream);

/*
 * Debug timeline of rl_decode_attn, to see where the split kernel's time
 * goes: the same call (arguments, plan, outputs and arithmetic), with the
 * split kernel built to leave one record of RL_TIMELINE_WORDS uint64 per work
 * item, item i at records + i * RL_TIMELINE_WORDS (device memory, 8-byte
 * aligned, `capacity` records):
 *   [0] HW_ID register | XCC id << 32 | kind (0 prefix item, 1 suffix item)
 *       << 40 | query rows << 48
 *   [1] wall clock when the item's workgroup starts   (s_memrealtime, 100 MHz)
 *   [2] wall clock once its first KV tile is in LDS
 *   [3] wall clock at the end of its loop over tiles
 *   [4] wall clock after its partials are written
 *   [5] KV tokens | tiles << 32
 *   [6] work-item index
 *   [7] s_memtime cycles of the loop
 * *num_records gets the number of work items; with records == NULL only that
 * number is computed (host-only planning; shape and lens are checked, no
 * pointer).  Status: as rl_decode_attn, plus RL_ERR_NULL_POINTER for a NULL
 * num_records, RL_ERR_WORKSPACE when capacity is short and
 * RL_ERR_MISALIGNED for misaligned records.
 */
rl_status rl_debug_decode_timeline(const rl_decode_shape *shape, const rl_decode_lens *lens,
                                   const rl_decode_ptrs *ptrs, void *workspace, size_t workspace_bytes,
                                   uint64_t *records, int64_t capacity, int64_t *num_records, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* RL_KERNELS_H */
