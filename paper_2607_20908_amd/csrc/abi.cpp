// Exported C ABI of librlkern.so (declared in include/rl_kernels.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <chrono>
#include <cstring>
#include <thread>
#include <string>
#include <vector>

#include "abi_error.h"
#include "kernels.h"
#include "decode_args.h"
#include "extend_args.h"
#include "logprob_args.h"
#include "plan.h"
#include "rl_kernels.h"
#include "tile_index.h"

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

namespace rlk {
void abi_clear_error() { g_last_error.clear(); }
rl_status abi_fail(rl_status st, const std::string &msg) { return set_error(st, msg); }
rl_status abi_hip_fail(hipError_t e, const char *what) { return hip_error(e, what); }
}  // namespace rlk

namespace {

// Pinned host staging for the work-list upload.  The slots are coherent,
// device-mapped host memory that a small kernel on the caller's stream reads
// directly (no copy-engine hand-off in front of the split kernel), so the host
// never waits for the stream.  A slot is reused once the kernel that read it
// has run: the operation's last kernel stores the slot's sequence number into
// a pinned word (no marker packet on the stream, which would hold the next
// kernel back by a few microseconds), or, if that kernel did not launch, an
// event recorded behind the fetch says so.  A call takes any slot whose
// reader has run; if there is none it adds a slot, up to kStagingSlots per
// thread, and only then waits for the oldest.  Nothing is ever freed: a slot
// that needs more room keeps its old buffer and takes one at least twice as
// large (so a slot's retired buffers total less than its current one), and
// the slots are plain thread-local storage with no destructors to run after
// the HIP runtime has shut down.  (hipHostFree could wait for the device.)
struct StagingSlot {
    unsigned char *host;
    void *dev;                 // the same memory as the device sees it
    size_t cap;
    hipEvent_t done;
    int device;
    bool pending;              // a kernel may still read the slot
    bool by_flag;              // pending until *flag reaches expect (else until `done`)
    uint64_t *flag;            // pinned word, stored into by the device
    uint64_t *flag_dev;
    uint64_t expect;
    uint64_t last_use;         // call number of the slot's last upload
};
constexpr int kStagingSlots = 64;
thread_local StagingSlot g_staging[kStagingSlots];
thread_local int g_staging_count;      // slots created so far on this thread
thread_local uint64_t g_staging_calls;

// True once the slot's reader has run (no waiting).
bool slot_released(StagingSlot &slot) {
    if (!slot.pending) return true;
    const bool done = slot.by_flag ? __atomic_load_n(slot.flag, __ATOMIC_ACQUIRE) >= slot.expect
                                   : hipEventQuery(slot.done) == hipSuccess;
    if (done) slot.pending = false;
    return done;
}

// Waits until the slot's reader has run (60 s limit).
rl_status wait_slot(StagingSlot &slot);

// One plan object per thread, reused so that planning does not allocate once
// its vectors have grown to the problem size.
thread_local rlk::DecodePlan g_plan;
thread_local rlk::ExtendPlan g_extend_plan;

struct Section {
    size_t off;
    const void *src;
    size_t n;
};

thread_local StagingSlot *g_staged_slot;     // the slot of the last upload, until committed

// Copies the sections (each followed by zeros up to the next section's
// offset, the last up to `total`) into the next staging slot and enqueues
// the fetch of `total` bytes (a multiple of 16) into `dst` on `stream`.
// The caller then enqueues the kernels that read the upload and calls
// stage_commit, which records the slot's reuse event behind them: an event
// recorded between the fetch and the next kernel would hold that kernel back
// by the few microseconds the command processor takes for the marker.
rl_status wait_slot(StagingSlot &slot) {
    if (!slot.pending) return RL_OK;
    if (slot.by_flag) {
        const auto t0 = std::chrono::steady_clock::now();
        for (uint32_t i = 1; __atomic_load_n(slot.flag, __ATOMIC_ACQUIRE) < slot.expect; ++i) {
            if (i < 256) continue;
            std::this_thread::yield();
            if ((i & 4095) == 0 && std::chrono::steady_clock::now() - t0 > std::chrono::seconds(60))
                return set_error(RL_ERR_HIP, "waiting for a staging slot: the kernel that reads it has "
                                             "not run for 60 s");
        }
    } else {
        const hipError_t e = hipEventSynchronize(slot.done);
        if (e != hipSuccess) return hip_error(e, "waiting for a staging slot");
    }
    slot.pending = false;
    return RL_OK;
}

// A slot whose reader has run: a free existing one, else a new one while
// fewer than kStagingSlots exist, else the least recently used, waited for.
rl_status next_slot(StagingSlot **out) {
    StagingSlot *lru = nullptr;
    for (int i = 0; i < g_staging_count; ++i) {
        StagingSlot &s = g_staging[i];
        if (slot_released(s)) {
            *out = &s;
            return RL_OK;
        }
        if (!lru || s.last_use < lru->last_use) lru = &s;
    }
    if (g_staging_count < kStagingSlots) {
        *out = &g_staging[g_staging_count++];
        return RL_OK;
    }
    const rl_status st = wait_slot(*lru);
    if (st != RL_OK) return st;
    *out = lru;
    return RL_OK;
}

rl_status stage_sections(const Section *sec, int nsec, size_t total, void *dst, hipStream_t stream) {
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_error(e, "hipGetDevice");
    StagingSlot *sp = nullptr;
    const rl_status st = next_slot(&sp);
    if (st != RL_OK) return st;
    StagingSlot &slot = *sp;
    slot.last_use = ++g_staging_calls;
    if (slot.done && slot.device != device) {
        (void)hipEventDestroy(slot.done);
        slot.done = nullptr;
    }
    if (!slot.done) {
        // completion only: the host reads nothing the GPU wrote, so no
        // system-scope fence (an L2 write-back) is needed when it is recorded
        e = hipEventCreateWithFlags(&slot.done, hipEventDisableTiming | hipEventDisableSystemFence);
        if (e != hipSuccess) return hip_error(e, "creating a staging event");
        if (!slot.flag) {
            e = hipHostMalloc(reinterpret_cast<void **>(&slot.flag), 64, hipHostMallocMapped | hipHostMallocCoherent);
            if (e != hipSuccess) return hip_error(e, "allocating the staging flag");
            __atomic_store_n(slot.flag, slot.expect, __ATOMIC_RELEASE);
        }
        e = hipHostGetDevicePointer(reinterpret_cast<void **>(&slot.flag_dev), slot.flag, 0);
        if (e != hipSuccess) return hip_error(e, "mapping the staging flag");
        slot.device = device;
    }
    if (slot.cap < total) {
        // the old buffer is retired, not freed (see above)
        slot.host = nullptr;
        const size_t cap = std::max<size_t>(std::max<size_t>(total, 2 * slot.cap), 1 << 16);
        slot.cap = 0;
        e = hipHostMalloc(reinterpret_cast<void **>(&slot.host), cap,
                          hipHostMallocMapped | hipHostMallocCoherent);
        if (e != hipSuccess) return hip_error(e, "allocating pinned staging memory");
        e = hipHostGetDevicePointer(&slot.dev, slot.host, 0);
        if (e != hipSuccess) return hip_error(e, "mapping pinned staging memory");
        slot.cap = cap;
    }
    for (int i = 0; i < nsec; ++i) {
        const size_t end = i + 1 < nsec ? sec[i + 1].off : total;
        if (sec[i].n) std::memcpy(slot.host + sec[i].off, sec[i].src, sec[i].n);
        std::memset(slot.host + sec[i].off + sec[i].n, 0, end - sec[i].off - sec[i].n);
    }
    e = rlk::launch_plan_fetch(slot.dev, dst, total, stream);
    if (e != hipSuccess) return hip_error(e, "uploading the work list");
    g_staged_slot = &slot;
    return RL_OK;
}

// The release word of the last upload's slot and the value that the
// operation's last kernel stores into it (system scope, thread 0 of block 0).
rlk::StageRelease stage_release() {
    StagingSlot *slot = g_staged_slot;
    if (!slot) return rlk::StageRelease{nullptr, 0};
    return rlk::StageRelease{reinterpret_cast<unsigned long long *>(slot->flag_dev),
                             static_cast<unsigned long long>(slot->expect + 1)};
}

// Marks the last upload's slot as in use until its reader has run: by the
// release word when the kernels enqueued since launched (`st` is RL_OK and
// `released_by_kernel`), otherwise by an event recorded on `stream` behind
// them.  `st` is the status of those launches and is passed through unless
// recording the event fails.
rl_status stage_commit(hipStream_t stream, rl_status st, bool released_by_kernel = false) {
    StagingSlot *slot = g_staged_slot;
    g_staged_slot = nullptr;
    if (!slot) return st;
    if (st == RL_OK && released_by_kernel) {
        slot->expect += 1;
        slot->by_flag = true;
        slot->pending = true;
        return st;
    }
    slot->by_flag = false;
    const hipError_t e = hipEventRecord(slot->done, stream);
    if (e != hipSuccess) {
        // the slot stays unguarded: drop it, so the next upload allocates afresh
        slot->host = nullptr;
        slot->cap = 0;
        slot->pending = false;
        return st != RL_OK ? st : hip_error(e, "recording the staging event");
    }
    slot->pending = true;
    return st;
}

// The decode work list: items, then the prefix and suffix unit tables.
rl_status stage_upload(const rlk::DecodePlan &plan, void *dst, hipStream_t stream) {
    const Section sec[3] = {
        {plan.off_items, plan.dev_items.data(), plan.dev_items.size() * sizeof(rlk::DevItem)},
        {plan.off_prefix_units, plan.prefix_units.data(), plan.prefix_units.size() * sizeof(rlk::DevUnit)},
        {plan.off_suffix_units, plan.suffix_units.data(), plan.suffix_units.size() * sizeof(rlk::DevUnit)}};
    return stage_sections(sec, 3, plan.meta_bytes, dst, stream);
}

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
    std::string err;
    const rl_status st = rlk::plan_decode(shape, lens, &g_plan, &err, rlk::PlanDetail::kSizes);
    if (st != RL_OK) return set_error(st, err);
    *bytes = g_plan.total_bytes;
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
    const rl_status st = rlk::plan_decode(shape, lens, &plan, &err, rlk::PlanDetail::kDebug);
    if (st != RL_OK) return set_error(st, err);
    const int64_t n = static_cast<int64_t>(plan.items.size());
    for (int64_t i = 0; i < n && i < capacity; ++i) items[i] = plan.items[i];
    *num_items = n;
    return RL_OK;
}

namespace {
// rl_decode_attn, and with num_records non-null rl_debug_decode_timeline:
// the same call with the split kernel's timeline records in `records`.
rl_status decode_call(const rl_decode_shape *shape, const rl_decode_lens *lens, const rl_decode_ptrs *ptrs,
                      void *workspace, size_t workspace_bytes, void *stream, uint64_t *records, int64_t capacity,
                      int64_t *num_records) {
    g_last_error.clear();
    rlk::DecodePlan &plan = g_plan;
    std::string err;
    rl_status st = rlk::plan_decode(shape, lens, &plan, &err, rlk::PlanDetail::kDevice);
    if (st != RL_OK) return set_error(st, err);
    const int64_t n_items = static_cast<int64_t>(plan.dev_items.size());
    if (num_records && !records) {
        *num_records = n_items;
        return RL_OK;
    }
    st = rlk::check_decode_ptrs(plan, lens, ptrs, &err);
    if (st != RL_OK) return set_error(st, err);
    if (num_records) {
        if (capacity < n_items)
            return set_error(RL_ERR_WORKSPACE, "records hold " + std::to_string(capacity) +
                                                   " entries, the call writes " + std::to_string(n_items));
        if ((reinterpret_cast<uintptr_t>(records) & 7u) != 0)
            return set_error(RL_ERR_MISALIGNED, "records are not 8-byte aligned");
    }
    const int64_t S = static_cast<int64_t>(plan.P) * plan.G;
    if (S == 0) {
        if (num_records) *num_records = 0;
        return RL_OK;
    }
    if (!workspace || workspace_bytes < plan.total_bytes)
        return set_error(RL_ERR_WORKSPACE, "workspace needs " + std::to_string(plan.total_bytes) +
                                               " bytes, got " + std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");

    // Work list and unit tables, uploaded in one copy on the caller's stream.
    hipStream_t hs = static_cast<hipStream_t>(stream);
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    st = stage_upload(plan, ws, hs);
    if (st != RL_OK) return st;

    rlk::DecodeArgs a = rlk::decode_args(plan, *ptrs, ws);
    a.release = stage_release();
    a.timeline = records;
    const hipError_t e = rlk::launch_decode(a, hs, num_records != nullptr);
    st = stage_commit(hs, e != hipSuccess ? hip_error(e, "launching decode attention") : RL_OK, true);
    if (st == RL_OK && num_records) *num_records = n_items;
    return st;
}
}  // namespace

rl_status rl_decode_attn(const rl_decode_shape *shape, const rl_decode_lens *lens,
                         const rl_decode_ptrs *ptrs, void *workspace, size_t workspace_bytes,
                         void *stream) {
    return decode_call(shape, lens, ptrs, workspace, workspace_bytes, stream, nullptr, 0, nullptr);
}

rl_status rl_debug_decode_timeline(const rl_decode_shape *shape, const rl_decode_lens *lens,
                                   const rl_decode_ptrs *ptrs, void *workspace, size_t workspace_bytes,
                                   uint64_t *records, int64_t capacity, int64_t *num_records, void *stream) {
    if (!num_records) {
        g_last_error.clear();
        return set_error(RL_ERR_NULL_POINTER, "num_records is NULL");
    }
    return decode_call(shape, lens, ptrs, workspace, workspace_bytes, stream, records, capacity, num_records);
}

rl_status rl_extend_attn_workspace_size(const rl_decode_shape *shape, const rl_extend_lens *lens,
                                        size_t *bytes) {
    g_last_error.clear();
    if (!bytes) return set_error(RL_ERR_NULL_POINTER, "bytes is NULL");
    std::string err;
    const rl_status st = rlk::plan_extend(shape, lens, &g_extend_plan, &err, false);
    if (st != RL_OK) return set_error(st, err);
    *bytes = g_extend_plan.total_bytes;
    return RL_OK;
}

rl_status rl_extend_attn(const rl_decode_shape *shape, const rl_extend_lens *lens,
                         const rl_decode_ptrs *ptrs, void *workspace, size_t workspace_bytes,
                         void *stream) {
    g_last_error.clear();
    rlk::ExtendPlan &plan = g_extend_plan;
    std::string err;
    rl_status st = rlk::plan_extend(shape, lens, &plan, &err, true);
    if (st != RL_OK) return set_error(st, err);
    st = rlk::check_extend_ptrs(plan, ptrs, &err);
    if (st != RL_OK) return set_error(st, err);
    if (plan.n_items == 0) return RL_OK;
    if (!workspace || workspace_bytes < plan.total_bytes)
        return set_error(RL_ERR_WORKSPACE, "workspace needs " + std::to_string(plan.total_bytes) +
                                               " bytes, got " + std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");
    hipStream_t hs = static_cast<hipStream_t>(stream);
    const Section sec[1] = {{0, plan.items.data(), plan.items.size() * sizeof(rlk::ExtItem)}};
    st = stage_sections(sec, 1, plan.total_bytes, workspace, hs);
    if (st != RL_OK) return st;
    rlk::ExtendArgs a = rlk::extend_args(plan, *ptrs, workspace);
    a.release = stage_release();
    const hipError_t e = rlk::launch_extend(a, hs);
    return stage_commit(hs, e != hipSuccess ? hip_error(e, "launching extend attention") : RL_OK, true);
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
    const rlk::LogprobArgs a = rlk::logprob_args(plan, hidden_states, w_lm, target, inv_temperature, logprob, lse,
                                                 static_cast<unsigned char *>(workspace));
    const hipError_t e = rlk::launch_logprob(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_error(e, "launching token log-prob");
    return RL_OK;
}

rl_status rl_debug_logprob_timeline(int64_t rows, int32_t hidden, int32_t vocab, const void *hidden_states,
                                    const void *w_lm, const int32_t *target, float inv_temperature, float *logprob,
                                    float *lse, void *workspace, size_t workspace_bytes, uint64_t *records,
                                    int64_t capacity, int64_t *num_records, void *stream) {
    g_last_error.clear();
    if (!num_records) return set_error(RL_ERR_NULL_POINTER, "num_records is NULL");
    rlk::LogprobPlan plan;
    std::string err;
    rl_status st = rlk::plan_logprob(rows, hidden, vocab, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    // one record per wave (kTileWaves per workgroup) of the whole-tile,
    // narrow-tile and tail-part launches
    const int64_t need = (plan.n_dp_tiles + plan.narrow_tiles * plan.n_row_tiles +
                          plan.n_tail_tiles * plan.tail_splits) * rlk::kTileWaves;
    if (!records) {
        *num_records = need;
        return RL_OK;
    }
    st = rlk::check_logprob_args(plan, hidden_states, w_lm, target, inv_temperature, logprob, lse, &err);
    if (st != RL_OK) return set_error(st, err);
    if (capacity < need)
        return set_error(RL_ERR_WORKSPACE, "records hold " + std::to_string(capacity) + " entries, the call writes " +
                                               std::to_string(need));
    if ((reinterpret_cast<uintptr_t>(records) & 7u) != 0)
        return set_error(RL_ERR_MISALIGNED, "records are not 8-byte aligned");
    if (rows == 0) {
        *num_records = 0;
        return RL_OK;
    }
    if (!workspace || workspace_bytes < plan.total_bytes)
        return set_error(RL_ERR_WORKSPACE, "workspace needs " + std::to_string(plan.total_bytes) +
                                               " bytes, got " + std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");
    rlk::LogprobArgs a = rlk::logprob_args(plan, hidden_states, w_lm, target, inv_temperature, logprob, lse,
                                           static_cast<unsigned char *>(workspace));
    a.timeline = records;
    const hipError_t e = rlk::launch_logprob(a, static_cast<hipStream_t>(stream), true);
    if (e != hipSuccess) return hip_error(e, "launching token log-prob (timeline)");
    *num_records = need;
    return RL_OK;
}

static bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

namespace {
// Validates an append and builds its (source, destination) row pairs.
thread_local std::vector<int64_t> g_append_rows;
thread_local std::vector<std::pair<int64_t, int64_t>> g_append_ranges;

rl_status plan_append(const rl_decode_shape *shape, const rl_kv_append_lens *lens, bool build, int64_t *n_new) {
    if (!shape || !lens) return set_error(RL_ERR_NULL_POINTER, "shape and lens must not be NULL");
    const int64_t P = shape->num_prompts, G = shape->group_size;
    if (P < 0 || G < 1) return set_error(RL_ERR_INVALID_SHAPE, "num_prompts >= 0 and group_size >= 1 required");
    if (shape->num_kv_heads < 1) return set_error(RL_ERR_INVALID_SHAPE, "num_kv_heads must be >= 1");
    if (shape->head_dim != 64 && shape->head_dim != 128) return set_error(RL_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
    if (shape->kv_layout != RL_KV_TOKEN_MAJOR && shape->kv_layout != RL_KV_HEAD_MAJOR)
        return set_error(RL_ERR_INVALID_SHAPE, "kv_layout must be RL_KV_TOKEN_MAJOR or RL_KV_HEAD_MAJOR");
    const int64_t S = P * G;
    if (S > 0 && (!lens->suffix_start || !lens->suffix_len || !lens->new_start || !lens->new_len))
        return set_error(RL_ERR_NULL_POINTER, "suffix_start, suffix_len, new_start and new_len must not be NULL");
    if (lens->suffix_rows < 0 || lens->new_rows < 0) return set_error(RL_ERR_INVALID_SHAPE, "negative row counts");
    int64_t total = 0;
    g_append_ranges.clear();
    for (int64_t s = 0; s < S; ++s) {
        const int64_t st = lens->suffix_start[s], len = lens->suffix_len[s];
        const int64_t ns = lens->new_start[s], nl = lens->new_len[s];
        if (st < 0 || len < 0 || ns < 0 || nl < 0)
            return set_error(RL_ERR_INVALID_SHAPE, "negative start or length at candidate " + std::to_string(s));
        if (nl == 0) continue;
        const int64_t end = st + len + nl;
        if (end > lens->suffix_rows)
            return set_error(RL_ERR_INVALID_SHAPE, "candidate " + std::to_string(s) + " writes past suffix_rows");
        if (lens->suffix_capacity && len + nl > lens->suffix_capacity[s])
            return set_error(RL_ERR_INVALID_SHAPE, "candidate " + std::to_string(s) + " exceeds its capacity");
        if (ns + nl > lens->new_rows)
            return set_error(RL_ERR_INVALID_SHAPE, "candidate " + std::to_string(s) + " reads past new_rows");
        g_append_ranges.emplace_back(st + len, end);
        total += nl;
    }
    std::sort(g_append_ranges.begin(), g_append_ranges.end());
    for (size_t i = 1; i < g_append_ranges.size(); ++i)
        if (g_append_ranges[i].first < g_append_ranges[i - 1].second)
            return set_error(RL_ERR_INVALID_SHAPE, "two candidates write the same suffix rows");
    *n_new = total;
    if (build) {
        g_append_rows.resize(static_cast<size_t>(2 * total));
        int64_t t = 0;
        for (int64_t s = 0; s < S; ++s) {
            const int64_t nl = lens->new_len[s];
            const int64_t dst0 = lens->suffix_start[s] + lens->suffix_len[s];
            for (int64_t i = 0; i < nl; ++i, ++t) {
                g_append_rows[2 * t] = lens->new_start[s] + i;
                g_append_rows[2 * t + 1] = dst0 + i;
            }
        }
    }
    return RL_OK;
}
}  // namespace

rl_status rl_kv_append_workspace_size(const rl_decode_shape *shape, const rl_kv_append_lens *lens, size_t *bytes) {
    g_last_error.clear();
    if (!bytes) return set_error(RL_ERR_NULL_POINTER, "bytes is NULL");
    int64_t n = 0;
    const rl_status st = plan_append(shape, lens, false, &n);
    if (st != RL_OK) return st;
    *bytes = rlk::align_up(static_cast<size_t>(n) * 16, 256);
    return RL_OK;
}

rl_status rl_kv_append(const rl_decode_shape *shape, const rl_kv_append_lens *lens, const void *k_new,
                       const void *v_new, void *k_suffix, void *v_suffix, void *workspace, size_t workspace_bytes,
                       void *stream) {
    g_last_error.clear();
    int64_t n = 0;
    rl_status st = plan_append(shape, lens, true, &n);
    if (st != RL_OK) return st;
    if (n == 0) return RL_OK;
    if (!k_new || !v_new || !k_suffix || !v_suffix)
        return set_error(RL_ERR_NULL_POINTER, "k_new, v_new, k_suffix and v_suffix must not be NULL");
    if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_suffix) || !aligned16(v_suffix))
        return set_error(RL_ERR_MISALIGNED, "the KV tensors must be 16-byte aligned");
    const size_t need = rlk::align_up(static_cast<size_t>(n) * 16, 256);
    if (!workspace || workspace_bytes < need)
        return set_error(RL_ERR_WORKSPACE,
                         "workspace needs " + std::to_string(need) + " bytes, got " + std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    const Section sec[1] = {{0, g_append_rows.data(), static_cast<size_t>(n) * 16}};
    st = stage_sections(sec, 1, need, workspace, hs);
    if (st != RL_OK) return st;
    rlk::KvAppendArgs a{};
    a.k_new = static_cast<const uint16_t *>(k_new);
    a.v_new = static_cast<const uint16_t *>(v_new);
    a.k_suffix = static_cast<uint16_t *>(k_suffix);
    a.v_suffix = static_cast<uint16_t *>(v_suffix);
    a.rows = static_cast<const int64_t *>(workspace);
    a.n_new = n;
    a.suffix_rows = lens->suffix_rows;
    a.Hkv = shape->num_kv_heads;
    a.D = shape->head_dim;
    a.kv_layout = shape->kv_layout;
    a.release = stage_release();
    const hipError_t e = rlk::launch_kv_append(a, hs);
    return stage_commit(hs, e != hipSuccess ? hip_error(e, "launching the KV append") : RL_OK, true);
}

rl_status rl_token_logprob_backward_workspace_size(int64_t rows, int32_t hidden, int32_t vocab, size_t *bytes) {
    g_last_error.clear();
    if (!bytes) return set_error(RL_ERR_NULL_POINTER, "bytes is NULL");
    rlk::LogprobBwdPlan plan;
    std::string err;
    const rl_status st = rlk::plan_logprob_bwd(rows, hidden, vocab, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    *bytes = plan.total_bytes;
    return RL_OK;
}

rl_status rl_token_logprob_backward(int64_t rows, int32_t hidden, int32_t vocab, const void *hidden_states,
                                    const void *w_lm, const int32_t *target, float inv_temperature,
                                    const float *lse, const float *grad_logprob, float *grad_hidden,
                                    void *workspace, size_t workspace_bytes, void *stream) {
    g_last_error.clear();
    rlk::LogprobBwdPlan plan;
    std::string err;
    rl_status st = rlk::plan_logprob_bwd(rows, hidden, vocab, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    if (!(std::isfinite(inv_temperature) && inv_temperature > 0.f))
        return set_error(RL_ERR_INVALID_SHAPE, "inv_temperature must be finite and > 0");
    if (rows == 0) return RL_OK;
    if (!hidden_states || !w_lm || !target || !lse || !grad_logprob || !grad_hidden)
        return set_error(RL_ERR_NULL_POINTER,
                         "hidden_states, w_lm, target, lse, grad_logprob and grad_hidden must not be NULL");
    if (!aligned16(hidden_states) || !aligned16(w_lm) || !aligned16(grad_hidden))
        return set_error(RL_ERR_MISALIGNED, "hidden_states, w_lm and grad_hidden must be 16-byte aligned");
    if (!aligned4(target) || !aligned4(lse) || !aligned4(grad_logprob))
        return set_error(RL_ERR_MISALIGNED, "target, lse and grad_logprob must be 4-byte aligned");
    if (!workspace || workspace_bytes < plan.total_bytes)
        return set_error(RL_ERR_WORKSPACE, "workspace needs " + std::to_string(plan.total_bytes) +
                                               " bytes, got " + std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    const uint16_t *hid = static_cast<const uint16_t *>(hidden_states);
    const uint16_t *w = static_cast<const uint16_t *>(w_lm);
    for (int64_t c0 = 0; c0 < rows; c0 += plan.chunk_rows) {
        rlk::LogprobArgs f;
        rlk::LogprobBwdArgs b;
        rlk::logprob_bwd_chunk_args(plan, c0, hid, w, target, inv_temperature, lse, grad_logprob, grad_hidden, ws, &f,
                                    &b);
        hipError_t e = rlk::launch_logprob_probs(f, hs);
        if (e != hipSuccess) return hip_error(e, "launching the log-prob backward (probabilities)");
        e = rlk::launch_logprob_bwd_gemm(b, hs);
        if (e != hipSuccess) return hip_error(e, "launching the log-prob backward (GEMM)");
        e = rlk::launch_logprob_bwd_finish(b, hs);
        if (e != hipSuccess) return hip_error(e, "launching the log-prob backward (finish)");
    }
    return RL_OK;
}

rl_status rl_sample_top_p_workspace_size(int64_t rows, int32_t hidden, int32_t vocab, size_t *bytes) {
    g_last_error.clear();
    if (!bytes) return set_error(RL_ERR_NULL_POINTER, "bytes is NULL");
    rlk::SamplePlan plan;
    std::string err;
    const rl_status st = rlk::plan_sample(rows, hidden, vocab, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    *bytes = plan.total_bytes;
    return RL_OK;
}

rl_status rl_sample_top_p(int64_t rows, int32_t hidden, int32_t vocab, const void *hidden_states,
                          const void *w_lm, const float *inv_temperature, float top_p, const float *uniform,
                          int32_t *token, float *logprob, void *workspace, size_t workspace_bytes,
                          void *stream) {
    g_last_error.clear();
    rlk::SamplePlan plan;
    std::string err;
    rl_status st = rlk::plan_sample(rows, hidden, vocab, &plan, &err);
    if (st != RL_OK) return set_error(st, err);
    if (!(std::isfinite(top_p) && top_p > 0.f && top_p <= 1.f))
        return set_error(RL_ERR_INVALID_SHAPE, "top_p must be in (0, 1]");
    if (rows == 0) return RL_OK;
    if (!hidden_states || !w_lm || !inv_temperature || !uniform || !token)
        return set_error(RL_ERR_NULL_POINTER, "hidden_states, w_lm, inv_temperature, uniform and token must not be NULL");
    if (!aligned16(hidden_states) || !aligned16(w_lm))
        return set_error(RL_ERR_MISALIGNED, "hidden_states and w_lm must be 16-byte aligned");
    if (!aligned4(inv_temperature) || !aligned4(uniform) || !aligned4(token) || (logprob && !aligned4(logprob)))
        return set_error(RL_ERR_MISALIGNED, "inv_temperature, uniform, token and logprob must be 4-byte aligned");
    if (!workspace || workspace_bytes < plan.total_bytes)
        return set_error(RL_ERR_WORKSPACE, "workspace needs " + std::to_string(plan.total_bytes) +
                                               " bytes, got " + std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    const uint16_t *hid = static_cast<const uint16_t *>(hidden_states);
    for (int64_t c0 = 0; c0 < rows; c0 += plan.chunk_rows) {
        rlk::LogprobArgs f;
        rlk::SampleArgs s;
        rlk::sample_chunk_args(plan, c0, hid, static_cast<const uint16_t *>(w_lm), inv_temperature, top_p, uniform,
                               token, logprob, ws, &f, &s);
        hipError_t e = rlk::launch_logits(f, hs);
        if (e != hipSuccess) return hip_error(e, "launching the sampling head (logits)");
        e = rlk::launch_sample_top_p(s, hs);
        if (e != hipSuccess) return hip_error(e, "launching the sampling head (selection)");
    }
    return RL_OK;
}

rl_status rl_grpo_advantage(int64_t num_prompts, int32_t group_size, const float *reward, float *adv,
                            void *stream) {
    g_last_error.clear();
    if (num_prompts < 0) return set_error(RL_ERR_INVALID_SHAPE, "num_prompts < 0");
    if (group_size < 1) return set_error(RL_ERR_INVALID_SHAPE, "group_size < 1");
    if (group_size > 1024) return set_error(RL_ERR_UNSUPPORTED, "group_size must be <= 1024");
    if (num_prompts == 0) return RL_OK;
    if (!reward || !adv) return set_error(RL_ERR_NULL_POINTER, "reward and adv must not be NULL");
    if (!aligned4(reward) || !aligned4(adv)) return set_error(RL_ERR_MISALIGNED, "reward/adv not 4-byte aligned");
    const hipError_t e = rlk::launch_grpo_advantage(num_prompts, group_size, reward, adv,
                                                    static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_error(e, "launching the GRPO advantages");
    return RL_OK;
}

namespace {
struct GrpoLayout {
    size_t off_counts = 0, off_partials = 0, total = 0;
};

rl_status grpo_layout(int64_t rows, int64_t num_prompts, int32_t group_size, GrpoLayout *lay) {
    if (rows < 0) return set_error(RL_ERR_INVALID_SHAPE, "rows < 0");
    if (num_prompts < 0) return set_error(RL_ERR_INVALID_SHAPE, "num_prompts < 0");
    if (group_size < 1) return set_error(RL_ERR_INVALID_SHAPE, "group_size < 1");
    const int64_t S = num_prompts * group_size;
    if (S > INT32_MAX) return set_error(RL_ERR_UNSUPPORTED, "too many candidates");
    lay->off_counts = 0;
    lay->off_partials = rlk::align_up(static_cast<size_t>(S) * 4, 256);
    lay->total = rlk::align_up(lay->off_partials + static_cast<size_t>(rlk::grpo_term_blocks(rows)) * 8, 256);
    if (lay->total == 0) lay->total = 256;
    return RL_OK;
}
}  // namespace

rl_status rl_grpo_surrogate_workspace_size(int64_t rows, int64_t num_prompts, int32_t group_size,
                                           size_t *bytes) {
    g_last_error.clear();
    if (!bytes) return set_error(RL_ERR_NULL_POINTER, "bytes is NULL");
    GrpoLayout lay;
    const rl_status st = grpo_layout(rows, num_prompts, group_size, &lay);
    if (st != RL_OK) return st;
    *bytes = lay.total;
    return RL_OK;
}

rl_status rl_grpo_surrogate(int64_t rows, int64_t num_prompts, int32_t group_size,
                            const float *logp_new, const float *logp_old, const int32_t *seq,
                            const float *adv, float eps, float *loss, float *grad,
                            void *workspace, size_t workspace_bytes, void *stream) {
    g_last_error.clear();
    GrpoLayout lay;
    const rl_status st = grpo_layout(rows, num_prompts, group_size, &lay);
    if (st != RL_OK) return st;
    if (!(std::isfinite(eps) && eps >= 0.f && eps < 1.f))
        return set_error(RL_ERR_INVALID_SHAPE, "eps must be finite and in [0, 1)");
    if (!loss) return set_error(RL_ERR_NULL_POINTER, "loss is NULL");
    if (rows > 0 && (!logp_new || !logp_old || !seq || !grad))
        return set_error(RL_ERR_NULL_POINTER, "logp_new, logp_old, seq and grad must not be NULL");
    if (num_prompts > 0 && !adv) return set_error(RL_ERR_NULL_POINTER, "adv is NULL");
    const void *ptrs[] = {logp_new, logp_old, seq, adv, loss, grad};
    for (const void *p : ptrs)
        if (p && !aligned4(p)) return set_error(RL_ERR_MISALIGNED, "a pointer is not 4-byte aligned");
    if (!workspace || workspace_bytes < lay.total)
        return set_error(RL_ERR_WORKSPACE, "workspace needs " + std::to_string(lay.total) + " bytes, got " +
                                               std::to_string(workspace_bytes));
    if (!aligned16(workspace)) return set_error(RL_ERR_MISALIGNED, "workspace is not 16-byte aligned");
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    rlk::GrpoArgs a{};
    a.rows = rows;
    a.P = num_prompts;
    a.G = group_size;
    a.S = num_prompts * group_size;
    a.eps = eps;
    a.logp_new = logp_new;
    a.logp_old = logp_old;
    a.adv = adv;
    a.seq = seq;
    a.loss = loss;
    a.grad = grad;
    a.counts = reinterpret_cast<int32_t *>(ws + lay.off_counts);
    a.partials = reinterpret_cast<double *>(ws + lay.off_partials);
    const hipError_t e = rlk::launch_grpo_surrogate(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_error(e, "launching the GRPO surrogate");
    return RL_OK;
}

}  // extern "C"
