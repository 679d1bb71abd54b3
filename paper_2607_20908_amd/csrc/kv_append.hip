// In-place append of new tokens' keys and values to the suffix KV cache, for
// gfx950: one thread per 16-byte chunk of (new token, kv head), K and V.
// The (source row, destination row) pair of each new token comes from the
// workspace; consecutive threads cover consecutive chunks of one row, so both
// the reads and the writes are coalesced in either cache layout.
#include "device_common.h"
#include "kernels.h"

namespace rlk {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void kv_append_kernel(KvAppendArgs a) {
    release_staging(a.release);
    const int chunks = a.D / 8;
    const int64_t per_tok = static_cast<int64_t>(a.Hkv) * chunks;
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (idx >= a.n_new * per_tok) return;
    const int64_t t = idx / per_tok;
    const int kh = static_cast<int>((idx % per_tok) / chunks);
    const int c = static_cast<int>(idx % chunks);
    const int64_t src = a.rows[2 * t], dst = a.rows[2 * t + 1];
    const int64_t soff = (src * a.Hkv + kh) * a.D + c * 8;
    const int64_t doff = (a.kv_layout == RL_KV_HEAD_MAJOR ? (kh * a.suffix_rows + dst) * a.D
                                                          : (dst * a.Hkv + kh) * a.D) + c * 8;
    *reinterpret_cast<u32x4 *>(a.k_suffix + doff) = *reinterpret_cast<const u32x4 *>(a.k_new + soff);
    *reinterpret_cast<u32x4 *>(a.v_suffix + doff) = *reinterpret_cast<const u32x4 *>(a.v_new + soff);
}

}  // namespace

hipError_t launch_kv_append(const KvAppendArgs &a, hipStream_t stream) {
    const int64_t n = a.n_new * a.Hkv * (a.D / 8);
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(kv_append_kernel, dim3(static_cast<uint32_t>((n + kThreads - 1) / kThreads)), dim3(kThreads),
                       0, stream, a);
    return hipGetLastError();
}

}  // namespace rlk
