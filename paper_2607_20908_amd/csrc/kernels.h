// Launch interface between the C ABI glue (abi.cpp) and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace rlk {

// Release of the pinned staging slot an operation's work list was fetched
// from: thread 0 of block 0 of the operation's last kernel (which runs after
// the fetch) stores `value` into `flag` at system scope.  flag may be null.
struct StageRelease {
    unsigned long long *flag;
    unsigned long long value;
};

__device__ __forceinline__ void release_staging(const StageRelease &r) {
    if (r.flag && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(r.flag, r.value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// uint64 words of one debug timeline record (a work item of the decode
// split kernel, a wave of an lm-head tile kernel)
constexpr int kTimelineWords = 8;

struct DecodeArgs {
    const uint16_t *q;
    const uint16_t *k_prefix, *v_prefix, *k_suffix, *v_suffix;
    uint16_t *out;
    float *lse;                 // may be null
    const DevItem *items;       // workspace: split-K work list
    const DevUnit *prefix_units, *suffix_units;
    float *pm, *pl, *pacc;      // workspace: partial max (log2 units), sum, weighted values
    int32_t n_items;            // work items in the list
    int32_t P, G, Hq, Hkv, r, D;
    int32_t kv_layout;          // RL_KV_TOKEN_MAJOR or RL_KV_HEAD_MAJOR
    int32_t deep_prefetch;      // split kernel with two tiles in flight per workgroup
    int64_t prefix_rows, suffix_rows;
    float score_scale_log2;     // softmax_scale * log2(e)
    StageRelease release;       // stored by the combine kernel
    uint64_t *timeline;         // debug timeline only: kTimelineWords words per work item
};

// timeline: the split kernel built with one timeline record per work item
hipError_t launch_decode(const DecodeArgs &a, hipStream_t stream, bool timeline = false);

// Causal extend attention: one workgroup per ExtItem block of query rows.
struct ExtendArgs {
    const uint16_t *q;
    const uint16_t *k_prefix, *v_prefix, *k_suffix, *v_suffix;
    uint16_t *out;
    float *lse;                 // may be null
    const ExtItem *items;       // workspace: the work list
    int32_t n_items;
    int32_t Hq, Hkv, r, D;
    int32_t kv_layout;
    int64_t prefix_rows, suffix_rows;
    float score_scale_log2;     // softmax_scale * log2(e)
    StageRelease release;
};

hipError_t launch_extend(const ExtendArgs &a, hipStream_t stream);

// Copies `bytes` (a multiple of 16) from device-mapped pinned host memory to
// device memory with a kernel on `stream`, so the work list reaches the
// workspace without a hand-off between the copy engine and the compute queue.
hipError_t launch_plan_fetch(const void *host_src, void *dst, size_t bytes, hipStream_t stream);

// Appends new tokens to the suffix caches: rows[2t] is token t's row in
// k_new / v_new ([rows, Hkv, D]), rows[2t + 1] its destination suffix row.
struct KvAppendArgs {
    const uint16_t *k_new, *v_new;
    uint16_t *k_suffix, *v_suffix;
    const int64_t *rows;        // workspace: (source, destination) per new token
    int64_t n_new;
    int64_t suffix_rows;
    int32_t Hkv, D;
    int32_t kv_layout;
    StageRelease release;
};

hipError_t launch_kv_append(const KvAppendArgs &a, hipStream_t stream);

struct LogprobArgs {
    const uint16_t *hidden;     // [R, H]
    const uint16_t *w;          // [V, H]
    const int32_t *target;      // [R]
    float *logprob, *lse;       // [R], lse may be null
    float *pm, *pl, *zt;        // workspace: [n_partials, R] x2, [R]
    int64_t R;
    int32_t H, V;
    int32_t n_vocab_tiles, n_row_tiles;
    float inv_temperature;
    // forward and backward probabilities: logical tiles [0, dp_tiles) run
    // whole; the tail_tiles after them run as `splits` parts of the hidden
    // dimension each, whose fp32 accumulators go to part (256 x 256 floats
    // per part, part j*splits + s of tail tile j) for the reduce kernel.
    // tile_base and tile_count are set per launch by the launch functions.
    int64_t dp_tiles, tail_tiles;
    int32_t splits;
    float *part;
    int64_t tile_base, tile_count;
    // forward and logits only: the last round as narrow tiles of w = 64
    // narrow_tm vocab entries (narrow_tm 2 or 3), narrow tile j covering
    // [narrow_v0 + w j, + w) with its partials in slot narrow_slot0 + j; the
    // combine merges n_partials slots per row
    int64_t narrow_v0, narrow_tiles, narrow_slot0, n_partials;
    int32_t narrow_tm;
    // backward only: the forward's lse per row (input) and the probabilities
    // p = exp(inv_T z - lse) as bf16 in the blocked layout of
    // LogprobBwdArgs::probs (output); pm, pl, zt, logprob are then unused
    const float *lse_in;
    uint16_t *probs;
    // sampling head only: per-row inverse temperatures (input) and the
    // tempered logits y = inv_T[r] z, fp32 [R, ld] (output); pm then holds
    // each (vocab tile, row)'s max of y
    const float *inv_t_rows;
    float *logits;
    int64_t ld;
    // debug timeline only (launch_logprob with timeline): kTimelineWords
    // words per wave of every whole-tile, narrow-tile and tail-part
    // workgroup, the launch's first record at timeline_base (set per launch)
    uint64_t *timeline;
    int64_t timeline_base;
};

// timeline: launch the tile kernels (whole, narrow, tail parts) built with
// per-wave timeline records (same arithmetic and outputs)
hipError_t launch_logprob(const LogprobArgs &a, hipStream_t stream, bool timeline = false);

// Backward of the token log-prob with respect to the hidden rows, for one
// chunk of rows at a time (the probabilities of a chunk live in the
// workspace):
//   dh[r] = g[r] inv_T (W[t_r] - sum_v p[r, v] W[v]).
// probs: bf16, blocked: for row tile rt and vocab step ks (64 entries), a
// 256 x 64 block at element ((rt * n_vsteps) + ks) * 16384 laid out as the
// LDS stage image op_off(row, chunk); entries past the vocabulary and rows
// without a valid target hold 0.
struct LogprobBwdArgs {
    const uint16_t *w;          // [V, H]
    const int32_t *target;      // [R]  (chunk-relative pointers below)
    const float *grad;          // [R]
    float *dh;                  // [R, H] fp32
    const uint16_t *probs;      // blocked probabilities of the chunk
    float *dpart;               // [splits, rows_pad, H] fp32 partial sums
    int64_t rows;               // rows in this chunk
    int32_t H, V;
    int32_t n_vsteps;           // vocab steps of 64 (padded vocabulary / 64)
    int32_t n_row_tiles, n_h_tiles, splits, steps_per_split;
    float inv_temperature;
};

hipError_t launch_logprob_probs(const LogprobArgs &a, hipStream_t stream);
hipError_t launch_logits(const LogprobArgs &a, hipStream_t stream);

// Nucleus sampling over tempered logits already in memory (one chunk of
// rows): per row, the max from the tile maxima, the nucleus of the top_p
// most probable tokens and the inverse CDF of the renormalised nucleus in id
// order at the row's uniform draw.
struct SampleArgs {
    const float *logits;        // [rows, ld] fp32 tempered logits
    const float *pm;            // [n_partials, rows] tile maxima of the logits
    const float *uniform;       // [rows] in [0, 1)
    int32_t *token;             // [rows]
    float *logprob;             // [rows] or null
    int64_t rows, ld;
    int32_t V, n_partials;      // n_partials: row-maximum slots (whole and narrow tiles)
    float top_p;
};

hipError_t launch_sample_top_p(const SampleArgs &a, hipStream_t stream);
hipError_t launch_logprob_bwd_gemm(const LogprobBwdArgs &a, hipStream_t stream);
hipError_t launch_logprob_bwd_finish(const LogprobBwdArgs &a, hipStream_t stream);

hipError_t launch_grpo_advantage(int64_t P, int32_t G, const float *reward, float *adv, hipStream_t stream);

struct GrpoArgs {
    int64_t rows, P, S;         // token rows, prompts, candidates (P * G)
    int32_t G;
    float eps;
    const float *logp_new, *logp_old, *adv;
    const int32_t *seq;
    float *loss, *grad;
    int32_t *counts;            // workspace: rows per candidate [S]
    double *partials;           // workspace: per-workgroup term sums
};

// Workgroups of the per-row kernel (one partial sum each).
int64_t grpo_term_blocks(int64_t rows);
hipError_t launch_grpo_surrogate(const GrpoArgs &a, hipStream_t stream);

}  // namespace rlk
