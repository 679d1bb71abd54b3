// Kernel arguments of the extend attention, built from a plan and the
// caller's pointers.  rl_extend_attn launches with exactly these arguments,
// and the host bounds replay (bounds.cpp) replays the same ones.
#pragma once

#include "kernels.h"
#include "plan.h"
#include "rl_kernels.h"

namespace rlk {

// The staging release (where the kernel reports that it has read the work
// list) is the caller's to set.
inline ExtendArgs extend_args(const ExtendPlan &plan, const rl_decode_ptrs &ptrs, const void *workspace) {
    ExtendArgs a{};
    a.q = static_cast<const uint16_t *>(ptrs.q);
    a.k_prefix = static_cast<const uint16_t *>(ptrs.k_prefix);
    a.v_prefix = static_cast<const uint16_t *>(ptrs.v_prefix);
    a.k_suffix = static_cast<const uint16_t *>(ptrs.k_suffix);
    a.v_suffix = static_cast<const uint16_t *>(ptrs.v_suffix);
    a.out = static_cast<uint16_t *>(ptrs.out);
    a.lse = ptrs.lse;
    a.items = static_cast<const ExtItem *>(workspace);
    a.n_items = static_cast<int32_t>(plan.n_items);
    a.Hq = plan.Hq;
    a.Hkv = plan.Hkv;
    a.r = plan.r;
    a.D = plan.D;
    a.kv_layout = plan.kv_layout;
    a.prefix_rows = plan.prefix_rows;
    a.suffix_rows = plan.suffix_rows;
    a.score_scale_log2 = plan.scale * kLog2eHost;
    return a;
}

}  // namespace rlk
