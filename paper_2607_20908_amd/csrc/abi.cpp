// Exported C ABI of librlkern.so (declared in include/rl_kernels.h).
#include <hip/hip_runtime.h>

#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"
#include "plan.h"
#include "rl_kernels.h"

namespace {

thread_local std::string g_last_error;

rl_status set_error(rl_status st, const std::string &msg) {
    g_last_error = msg;
    return st;
}

rl_status hip_error(hipError_t e, const char *what) {
    return set_error(RL_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" {

int rl_abi_version(void) { return RL_ABI_VERSION; }

const char *rl_status_string(rl_status status) {
    switch (status) {
        case RL_OK: return "RL_OK";
        case RL_ERR_NULL_POINTER: return "RL_ERR_NULL_POINTER";
        case RL_ERR_INVALID_SHAPE: return "RL_ERR_INVALID_SHAPE";
        case RL_ERR_UNSUPPORTED: return "RL_ERR_UNSUPPORTED";
        case RL_ERR_MISALIGNED: return "RL_ERR_MISALIGNED";
        case RL_ERR_WORKSPACE: return "RL_ERR_WORKSPACE";
        case RL_ERR_HIP: return "RL_ERR_HIP";
    }
    return "RL_ERR_UNKNOWN";
}

const char *rl_last_error(void) { return g_last_error.c_str(); }

rl_status rl_decode_attn_workspace_size(const rl_decode_shape *shape, const rl_decode_lens *lens,
                                        size_t *bytes) {
    g_last_error.clear();
    if (!bytes) return set_error(RL_ERR_NULL_POINTER, "bytes is NULL");
    rlk::DecodePlan plan;
    std::string err;
    const rl_status st = rlk::plan_decode(shape, lens, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    *bytes = plan.total_bytes;
    return RL_OK;
}

rl_status rl_decode_plan_debug(const rl_decode_shape *shape, const rl_decode_lens *lens,
                               rl_plan_item *items, int64_t capacity, int64_t *num_items) {
    g_last_error.clear();
    if (!num_items) return set_error(RL_ERR_NULL_POINTER, "num_items is NULL");
    if (capacity < 0) return set_error(RL_ERR_INVALID_SHAPE, "capacity < 0");
    if (capacity > 0 && !items) return set_error(RL_ERR_NULL_POINTER, "items is NULL");
    rlk::DecodePlan plan;
    std::string err;
    const rl_status st = rlk::plan_decode(shape, lens, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    const int64_t n = static_cast<int64_t>(plan.items.size());
    for (int64_t i = 0; i < n && i < capacity; ++i) items[i] = plan.items[i];
    *num_items = n;
    return RL_OK;
}

rl_status rl_decode_attn(const rl_decode_shape *shape, const rl_decode_lens *lens,
                         const rl_decode_ptrs *ptrs, void *workspace, size_t workspace_bytes,
                         void *stream) {
    g_last_error.clear();
    rlk::DecodePlan plan;
    std::string err;
    rl_status st = rlk::plan_decode(shape, lens, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    st = rlk::check_decode_ptrs(plan, lens, ptrs, &err);
    if (st != RL_OK) return set_error(st, err);
    const int64_t S = static_cast<int64_t>(plan.P) * plan.G;
    if (S == 0) return RL_OK;
    if (!workspace || workspace_bytes < plan.total_bytes)
        return set_error(RL_ERR_WORKSPACE, "workspace needs " + std::to_string(plan.total_bytes) +
                                               " bytes, got " + std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");

    // Work list and unit tables, uploaded in one copy on the caller's stream.
    thread_local std::vector<unsigned char> meta;
    meta.assign(plan.meta_bytes, 0);
    std::memcpy(meta.data() + plan.off_items, plan.dev_items.data(),
                plan.dev_items.size() * sizeof(rlk::DevItem));
    std::memcpy(meta.data() + plan.off_prefix_units, plan.prefix_units.data(),
                plan.prefix_units.size() * sizeof(rlk::DevUnit));
    std::memcpy(meta.data() + plan.off_suffix_units, plan.suffix_units.data(),
                plan.suffix_units.size() * sizeof(rlk::DevUnit));
    hipStream_t hs = static_cast<hipStream_t>(stream);
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    hipError_t e = hipMemcpyAsync(ws, meta.data(), plan.meta_bytes, hipMemcpyHostToDevice, hs);
    if (e != hipSuccess) return hip_error(e, "uploading the work list");

    rlk::DecodeArgs a{};
    a.q = static_cast<const uint16_t *>(ptrs->q);
    a.k_prefix = static_cast<const uint16_t *>(ptrs->k_prefix);
    a.v_prefix = static_cast<const uint16_t *>(ptrs->v_prefix);
    a.k_suffix = static_cast<const uint16_t *>(ptrs->k_suffix);
    a.v_suffix = static_cast<const uint16_t *>(ptrs->v_suffix);
    a.out = static_cast<uint16_t *>(ptrs->out);
    a.lse = ptrs->lse;
    a.items = reinterpret_cast<const rlk::DevItem *>(ws + plan.off_items);
    a.prefix_units = reinterpret_cast<const rlk::DevUnit *>(ws + plan.off_prefix_units);
    a.suffix_units = reinterpret_cast<const rlk::DevUnit *>(ws + plan.off_suffix_units);
    a.pm = reinterpret_cast<float *>(ws + plan.off_m);
    a.pl = reinterpret_cast<float *>(ws + plan.off_l);
    a.pacc = reinterpret_cast<float *>(ws + plan.off_acc);
    a.n_items = static_cast<int32_t>(plan.dev_items.size());
    a.P = plan.P;
    a.G = plan.G;
    a.Hq = plan.Hq;
    a.Hkv = plan.Hkv;
    a.r = plan.r;
    a.D = plan.D;
    a.score_scale_log2 = plan.scale * rlk::kLog2eHost;
    e = rlk::launch_decode(a, hs);
    if (e != hipSuccess) return hip_error(e, "launching decode attention");
    return RL_OK;
}

rl_status rl_token_logprob_workspace_size(int64_t rows, int32_t hidden, int32_t vocab, size_t *bytes) {
    g_last_error.clear();
    if (!bytes) return set_error(RL_ERR_NULL_POINTER, "bytes is NULL");
    rlk::LogprobPlan plan;
    std::string err;
    const rl_status st = rlk::plan_logprob(rows, hidden, vocab, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    *bytes = plan.total_bytes;
    return RL_OK;
}

rl_status rl_token_logprob(int64_t rows, int32_t hidden, int32_t vocab, const void *hidden_states,
                           const void *w_lm, const int32_t *target, float inv_temperature,
                           float *logprob, float *lse, void *workspace, size_t workspace_bytes,
                           void *stream) {
    g_last_error.clear();
    rlk::LogprobPlan plan;
    std::string err;
    rl_status st = rlk::plan_logprob(rows, hidden, vocab, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    st = rlk::check_logprob_args(plan, hidden_states, w_lm, target, inv_temperature, logprob, lse, &err);
    if (st != RL_OK) return set_error(st, err);
    if (rows == 0) return RL_OK;
    if (!workspace || workspace_bytes < plan.total_bytes)
        return set_error(RL_ERR_WORKSPACE, "workspace needs " + std::to_string(plan.total_bytes) +
                                               " bytes, got " + std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    rlk::LogprobArgs a{};
    a.hidden = static_cast<const uint16_t *>(hidden_states);
    a.w = static_cast<const uint16_t *>(w_lm);
    a.target = target;
    a.logprob = logprob;
    a.lse = lse;
    a.pm = reinterpret_cast<float *>(ws + plan.off_m);
    a.pl = reinterpret_cast<float *>(ws + plan.off_l);
    a.zt = reinterpret_cast<float *>(ws + plan.off_zt);
    a.R = rows;
    a.H = hidden;
    a.V = vocab;
    a.n_vocab_tiles = static_cast<int32_t>(plan.n_vocab_tiles);
    a.n_row_tiles = static_cast<int32_t>(plan.n_row_tiles);
    a.inv_temperature = inv_temperature;
    const hipError_t e = rlk::launch_logprob(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_error(e, "launching token log-prob");
    return RL_OK;
}

}  // extern "C"
