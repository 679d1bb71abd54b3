// The C ABI's per-thread error state (rl_last_error), for entry points
// defined outside abi.cpp.
#pragma once

#include <hip/hip_runtime.h>

#include <string>

#include "rl_kernels.h"

namespace rlk {

void abi_clear_error();
rl_status abi_fail(rl_status st, const std::string &msg);
rl_status abi_hip_fail(hipError_t e, const char *what);

}  // namespace rlk
