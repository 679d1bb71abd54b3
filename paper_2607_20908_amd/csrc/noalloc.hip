// rl_token_logprob_noalloc: the token log-prob with its workspace (the
// forward's (max, sum) partials, target logits and tail parts) in a static
// device array of this file instead of a caller buffer, for callers that
// cannot allocate.  The kernels and the plan are rl_token_logprob's.
//
// `scratch` below is a host-side stand-in in host code, not a device address:
// the address of each device's copy comes from hipGetSymbolAddress, looked up
// once per device and kept, and only that address reaches the kernels.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "abi_error.h"
#include "kernels.h"
#include "logprob_args.h"
#include "plan.h"
#include "rl_kernels.h"

namespace rlk {
namespace {

constexpr size_t kNoAllocScratchBytes = size_t(RL_NOALLOC_SCRATCH_BYTES);
static_assert(kNoAllocScratchBytes % 256 == 0, "scratch size");

// One copy per GPU the library runs on, held until the process ends.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up on the first call on
// that device.
rl_status scratch_of_current_device(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return abi_hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return abi_fail(RL_ERR_UNSUPPORTED, "rl_token_logprob_noalloc supports devices 0-63");
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return abi_hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return abi_fail(RL_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return RL_OK;
}

}  // namespace
}  // namespace rlk

extern "C" rl_status rl_token_logprob_noalloc(int64_t rows, int32_t hidden, int32_t vocab, const void *hidden_states,
                                              const void *w_lm, const int32_t *target, float inv_temperature,
                                              float *logprob, float *lse, void *stream) {
    using namespace rlk;
    abi_clear_error();
    LogprobPlan plan;
    std::string err;
    rl_status st = plan_logprob(rows, hidden, vocab, &plan, &err);
    if (st != RL_OK) return abi_fail(st, err);
    st = check_logprob_args(plan, hidden_states, w_lm, target, inv_temperature, logprob, lse, &err);
    if (st != RL_OK) return abi_fail(st, err);
    if (rows == 0) return RL_OK;
    if (plan.total_bytes > kNoAllocScratchBytes)
        return abi_fail(RL_ERR_UNSUPPORTED, "rl_token_logprob_noalloc: these sizes need " +
                                                std::to_string(plan.total_bytes) + " bytes of scratch, more than its " +
                                                std::to_string(kNoAllocScratchBytes) +
                                                "; call rl_token_logprob with a workspace");
    void *ws = nullptr;
    st = scratch_of_current_device(&ws);
    if (st != RL_OK) return st;
    // every partial, target logit and tail part is written before it is read,
    // so nothing in the scratch needs clearing between calls
    const LogprobArgs a = logprob_args(plan, hidden_states, w_lm, target, inv_temperature, logprob, lse,
                                       static_cast<unsigned char *>(ws));
    const hipError_t e = launch_logprob(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return abi_hip_fail(e, "launching token log-prob");
    return RL_OK;
}
