// Group-relative advantages and the clipped GRPO surrogate (beta = 0) for
// gfx950 (Sec. 3, Eq. grpo-loss and the advantage definition under it).
//
// Advantages: one wave per prompt group; mean and sample variance in fp64.
// Surrogate: the rows of each candidate are counted with integer atomics
// (order-independent), then each row's clipped term and gradient are
// computed and the terms are summed in a fixed order (a tree per workgroup,
// then the workgroup sums in index order), so the loss is bitwise
// reproducible.
#include "device_common.h"
#include "kernels.h"

namespace rlk {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// One wave per group of G candidates.
__global__ __launch_bounds__(kThreads) void grpo_advantage_kernel(int64_t P, int32_t G, const float *reward,
                                                                  float *adv) {
    const int lane = threadIdx.x & 63;
    const int64_t p = static_cast<int64_t>(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
    if (p >= P) return;
    const float *r = reward + p * G;
    float *a = adv + p * G;
    double s = 0.0;
    for (int i = lane; i < G; i += 64) s += r[i];
    const double mean = wave_sum_f64(s) / G;
    double ss = 0.0;
    for (int i = lane; i < G; i += 64) {
        const double d = r[i] - mean;
        ss += d * d;
    }
    ss = wave_sum_f64(ss);
    const double sd = G > 1 ? sqrt(ss / (G - 1)) : 0.0;
    for (int i = lane; i < G; i += 64) a[i] = sd > 0.0 ? static_cast<float>((r[i] - mean) / sd) : 0.f;
}

__global__ __launch_bounds__(kThreads) void grpo_zero_counts_kernel(int32_t *counts, int64_t S) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i < S) counts[i] = 0;
}

// A candidate's rows are usually contiguous, so one atomic per row would
// pile onto a few counters.  Each wave splits its 64 rows into runs of equal
// candidate id; the first lane of a run adds the run's length.  Any row order
// gives the same counts (every row belongs to exactly one run).
__global__ __launch_bounds__(kThreads) void grpo_count_kernel(GrpoArgs a) {
    const int64_t r = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    const int lane = threadIdx.x & 63;
    int32_t s = -1;
    if (r < a.rows) {
        s = a.seq[r];
        if (s < 0 || s >= a.S) s = -1;
    }
    const int32_t prev = __shfl_up(s, 1, 64);
    const bool head = lane == 0 || prev != s;
    const uint64_t heads = __ballot(head);
    if (head && s >= 0) {
        const uint64_t later = lane == 63 ? 0 : heads >> (lane + 1);
        const int next = later ? lane + 1 + __builtin_ctzll(later) : 64;
        atomicAdd(a.counts + s, next - lane);
    }
}

// Per row: the clipped term (weighted) and the gradient; per workgroup: the
// sum of its rows' terms (a fixed-shape tree).
__global__ __launch_bounds__(kThreads) void grpo_term_kernel(GrpoArgs a) {
    __shared__ double part[kThreads / 64];
    const int64_t r = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    double term = 0.0;
    if (r < a.rows) {
        const int32_t s = a.seq[r];
        float g = 0.f;
        if (s >= 0 && s < a.S) {
            const double A = a.adv[s];
            const double rho = exp(static_cast<double>(a.logp_new[r]) - static_cast<double>(a.logp_old[r]));
            const double lo = 1.0 - a.eps, hi = 1.0 + a.eps;
            const double clipped = rho < lo ? lo : (rho > hi ? hi : rho);
            const double u = rho * A, c = clipped * A;
            const double w = 1.0 / (static_cast<double>(a.P) * a.G * static_cast<double>(a.counts[s]));
            term = (u <= c ? u : c) * w;
            g = u <= c ? static_cast<float>(-w * rho * A) : 0.f;
        }
        a.grad[r] = g;
    }
    const double ws = wave_sum_f64(term);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ws;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) t += part[w];
        a.partials[blockIdx.x] = t;
    }
}

// One workgroup: the workgroup sums in index order, strided over the threads
// and then a fixed tree.
__global__ __launch_bounds__(kThreads) void grpo_loss_kernel(GrpoArgs a, int64_t nparts) {
    __shared__ double part[kThreads];
    double t = 0.0;
    for (int64_t i = threadIdx.x; i < nparts; i += kThreads) t += a.partials[i];
    part[threadIdx.x] = t;
    __syncthreads();
    for (int o = kThreads / 2; o >= 1; o >>= 1) {
        if (threadIdx.x < o) part[threadIdx.x] += part[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) *a.loss = static_cast<float>(-part[0]);
}

}  // namespace

hipError_t launch_grpo_advantage(int64_t P, int32_t G, const float *reward, float *adv, hipStream_t stream) {
    if (P == 0) return hipSuccess;
    const int64_t blocks = (P + kThreads / 64 - 1) / (kThreads / 64);
    hipLaunchKernelGGL(grpo_advantage_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0, stream, P,
                       G, reward, adv);
    return hipGetLastError();
}

int64_t grpo_term_blocks(int64_t rows) { return (rows + kThreads - 1) / kThreads; }

hipError_t launch_grpo_surrogate(const GrpoArgs &a, hipStream_t stream) {
    const int64_t nparts = grpo_term_blocks(a.rows);
    if (a.S > 0) {
        const int64_t zb = (a.S + kThreads - 1) / kThreads;
        hipLaunchKernelGGL(grpo_zero_counts_kernel, dim3(static_cast<uint32_t>(zb)), dim3(kThreads), 0, stream,
                           a.counts, a.S);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (a.rows > 0) {
        hipLaunchKernelGGL(grpo_count_kernel, dim3(static_cast<uint32_t>(nparts)), dim3(kThreads), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(grpo_term_kernel, dim3(static_cast<uint32_t>(nparts)), dim3(kThreads), 0, stream, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(grpo_loss_kernel, dim3(1), dim3(kThreads), 0, stream, a, nparts);
    return hipGetLastError();
}

}  // namespace rlk
