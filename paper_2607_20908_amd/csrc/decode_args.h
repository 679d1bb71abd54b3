// Kernel arguments of the decode attention, built from a plan and the
// caller's pointers.  rl_decode_attn launches with exactly these arguments,
// and the host bounds replay (bounds.cpp) replays the same ones.
#pragma once

#include "kernels.h"
#include "plan.h"
#include "rl_kernels.h"

namespace rlk {

// The staging release and the debug timeline are the caller's to set.
inline DecodeArgs decode_args(const DecodePlan &plan, const rl_decode_ptrs &ptrs, unsigned char *ws) {
    DecodeArgs a{};
    a.q = static_cast<const uint16_t *>(ptrs.q);
    a.k_prefix = static_cast<const uint16_t *>(ptrs.k_prefix);
    a.v_prefix = static_cast<const uint16_t *>(ptrs.v_prefix);
    a.k_suffix = static_cast<const uint16_t *>(ptrs.k_suffix);
    a.v_suffix = static_cast<const uint16_t *>(ptrs.v_suffix);
    a.out = static_cast<uint16_t *>(ptrs.out);
    a.lse = ptrs.lse;
    a.items = reinterpret_cast<const DevItem *>(ws + plan.off_items);
    a.prefix_units = reinterpret_cast<const DevUnit *>(ws + plan.off_prefix_units);
    a.suffix_units = reinterpret_cast<const DevUnit *>(ws + plan.off_suffix_units);
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
    a.kv_layout = plan.kv_layout;
    a.deep_prefetch = plan.deep_prefetch;
    a.prefix_rows = plan.prefix_rows;
    a.suffix_rows = plan.suffix_rows;
    a.score_scale_log2 = plan.scale * kLog2eHost;
    return a;
}

}  // namespace rlk
