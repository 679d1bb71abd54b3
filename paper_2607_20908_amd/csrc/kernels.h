// Launch interface between the C ABI glue (abi.cpp) and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace rlk {

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
    int64_t prefix_rows, suffix_rows;
    float score_scale_log2;     // softmax_scale * log2(e)
};

hipError_t launch_decode(const DecodeArgs &a, hipStream_t stream);

// Copies `bytes` (a multiple of 16) from device-mapped pinned host memory to
// device memory with a kernel on `stream`, so the work list reaches the
// workspace without a hand-off between the copy engine and the compute queue.
hipError_t launch_plan_fetch(const void *host_src, void *dst, size_t bytes, hipStream_t stream);

struct LogprobArgs {
    const uint16_t *hidden;     // [R, H]
    const uint16_t *w;          // [V, H]
    const int32_t *target;      // [R]
    float *logprob, *lse;       // [R], lse may be null
    float *pm, *pl, *zt;        // workspace: [n_vocab_tiles, R] x2, [R]
    int64_t R;
    int32_t H, V;
    int32_t n_vocab_tiles, n_row_tiles;
    float inv_temperature;
};

hipError_t launch_logprob(const LogprobArgs &a, hipStream_t stream);

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
