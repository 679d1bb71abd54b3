// Nucleus (top-p) sampling over tempered logits, one workgroup per row, for
// gfx950 (the rollout's sampling step, Sec. 3, Multi-turn RL Training).
//
// Probabilities are handled as integer masses q(y) = floor(2^40 exp(y - m)),
// m the row max, so every sum below is exact and independent of the order in
// which threads add: the sample is deterministic.  Tokens are ranked by the
// order-preserving 32-bit key of their fp32 logit (larger first), equal keys
// by the smaller id.  With Z the total mass and T = ceil(top_p Z), the nucleus
// is the shortest ranked prefix whose mass reaches T; it is described by the
// last member's key tau and how many tokens with key tau it holds (the k
// smallest ids among them).  The sample is the first id, in id order, at
// which the nucleus mass passes floor(u * Z_N).
//
// Passes over the row's logits:
//   1. mass histogram over b = floor(64 (m - y)) (4096 buckets of 1/64 logit
//      unit; the last also holds everything further below m, whose mass is
//      at most 2^40 e^-64 < 1, i.e. 0) -> the bucket B where the ranked mass
//      crosses T;
//   2. per chunk of 2048 ids the mass of the buckets above B, and the tokens
//      of B gathered, sorted by (key desc, id asc) in LDS and their masses
//      walked to tau and k; if B holds more than kCap tokens, further passes
//      refine it by 8-bit key digits first and recount each chunk's nucleus
//      mass and key-tau tokens;
//   3. the chunk holding the sample is rescanned in id order.
#include "device_common.h"
#include "kernels.h"

namespace rlk {
namespace {

constexpr int kThreads = 1024;          // 16 waves per row: the passes are issue-bound
constexpr int kWaves = kThreads / 64;
constexpr int kBuckets = 4096;
constexpr float kBucketScale = 64.f;
constexpr int kCap = 4096;              // candidates sorted in LDS
constexpr int kChunk = 2048;            // ids per chunk of the CDF pass
constexpr int kMaxChunks = 1024;        // vocabulary up to 2M entries
constexpr float kMassScale = 1099511627776.f;   // 2^40

// Order-preserving map of a float to uint32 (-0 and +0 arrive as +0).
__device__ __forceinline__ uint32_t fkey(float y) {
    const uint32_t b = __float_as_uint(y);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float key_to_float(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ uint64_t qmass(float y, float m) {
    return __float2ull_rz(fast_exp2((y - m) * kLog2e) * kMassScale);
}

// Bucket of a logit below the row max; a NaN lands in the last bucket and a
// logit above m (impossible: m is the max of the same values) in the first.
__device__ __forceinline__ int bucket_of(float y, float m) {
    const float d = (m - y) * kBucketScale;
    if (d >= 0.f) return d < static_cast<float>(kBuckets - 1) ? static_cast<int>(d) : kBuckets - 1;
    return d < 0.f ? 0 : kBuckets - 1;
}

template <typename T>
__device__ __forceinline__ T wave_sum_int(T v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Inclusive prefix sum over the 64 lanes of a wave.
template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const T x = __shfl_up(v, o, 64);
        if (lane >= o) v += x;
    }
    return v;
}

struct SelShared {
    union {
        uint64_t hist[kBuckets];                    // bucket masses; later digit masses
        struct {
            uint64_t mass[kMaxChunks];              // nucleus mass above tau per chunk of ids
            uint32_t ties[kMaxChunks];              // tokens with key tau per chunk
        } chunk;                                    // (once the histograms are no longer read)
    } a;
    union {
        uint64_t cand[kCap];                        // (key << 32) | ~id of the candidates
    } b;
    uint32_t dcount[256];                           // tokens per key digit
    uint64_t part[kThreads];                        // block scans
    uint64_t zsum[kWaves];
    float fred[kWaves];
    uint32_t ncand;
};

// Exclusive scan of one value per thread; returns the total.
__device__ uint64_t block_excl_scan(SelShared &sh, uint64_t v, uint64_t *excl) {
    const int tid = threadIdx.x;
    sh.part[tid] = v;
    __syncthreads();
    if (tid < 64) {
        constexpr int kPerLane = kThreads / 64;
        uint64_t sl = 0;
#pragma unroll
        for (int j = 0; j < kPerLane; ++j) sl += sh.part[kPerLane * tid + j];
        const uint64_t inc = wave_incl_scan(sl, tid);
        uint64_t run = inc - sl;
#pragma unroll
        for (int j = 0; j < kPerLane; ++j) {
            const uint64_t x = sh.part[kPerLane * tid + j];
            sh.part[kPerLane * tid + j] = run;
            run += x;
        }
        if (tid == 63) sh.zsum[0] = inc;
    }
    __syncthreads();
    *excl = sh.part[tid];
    const uint64_t total = sh.zsum[0];
    __syncthreads();
    return total;
}

// Calls f(v, y_v) for the ids of float4 groups g0, g0 + step, ... below g1
// (ids < V only), with DEPTH groups' loads in flight: the passes are bound by
// how many bytes each CU keeps in flight against the HBM latency.
template <int DEPTH, typename F>
__device__ __forceinline__ void scan_groups(const float *y, int V, int g0, int g1, int step, F &&f) {
    auto visit = [&](const float4 q4, int g) {
        const float yy[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (4 * g + e < V) f(4 * g + e, yy[e]);
    };
    int g = g0;
    for (; g + (DEPTH - 1) * step < g1; g += DEPTH * step) {
        float4 q[DEPTH];
#pragma unroll
        for (int j = 0; j < DEPTH; ++j) q[j] = *reinterpret_cast<const float4 *>(y + 4 * (g + j * step));
#pragma unroll
        for (int j = 0; j < DEPTH; ++j) visit(q[j], g + j * step);
    }
    for (; g < g1; g += step) visit(*reinterpret_cast<const float4 *>(y + 4 * g), g);
}

// Sorts the ncand gathered candidates by (key desc, id asc) and walks their
// masses from `above` to the first position reaching T: its key is tau and k
// counts the key-tau candidates up to it.
__device__ void sort_and_walk(SelShared &sh, uint32_t ncand, uint64_t above, uint64_t T, float m, uint32_t *tau,
                              uint64_t *k) {
    const int tid = threadIdx.x;
    int n2 = 1;
    while (n2 < static_cast<int>(ncand)) n2 <<= 1;
    for (int i = static_cast<int>(ncand) + tid; i < n2; i += kThreads) sh.b.cand[i] = 0;   // sorts last
    __syncthreads();
    for (int size = 2; size <= n2; size <<= 1) {                   // bitonic, descending
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < n2 / 2; i += kThreads) {
                const int lo = 2 * i - (i & (stride - 1));
                const int hi = lo + stride;
                const bool desc = (lo & size) == 0;
                const uint64_t x = sh.b.cand[lo], z = sh.b.cand[hi];
                if ((x < z) == desc) {
                    sh.b.cand[lo] = z;
                    sh.b.cand[hi] = x;
                }
            }
            __syncthreads();
        }
    }
    const int per = (static_cast<int>(ncand) + kThreads - 1) / kThreads;
    const int i0 = tid * per, i1 = min(static_cast<int>(ncand), i0 + per);
    uint64_t seg = 0;
    for (int i = i0; i < i1; ++i) seg += qmass(key_to_float(static_cast<uint32_t>(sh.b.cand[i] >> 32)), m);
    uint64_t segb;
    block_excl_scan(sh, seg, &segb);
    if (tid == 0) {                                                // defaults for a degenerate row
        sh.part[0] = ncand ? static_cast<uint32_t>(sh.b.cand[ncand - 1] >> 32) : 0u;
        sh.part[1] = 0;
    }
    __syncthreads();
    if (i0 < i1 && above + segb < T && above + segb + seg >= T) {
        uint64_t acc = above + segb;
        int i = i0;
        for (;; ++i) {
            acc += qmass(key_to_float(static_cast<uint32_t>(sh.b.cand[i] >> 32)), m);
            if (acc >= T || i == i1 - 1) break;
        }
        const uint32_t kt = static_cast<uint32_t>(sh.b.cand[i] >> 32);
        int f = i;
        while (f > 0 && static_cast<uint32_t>(sh.b.cand[f - 1] >> 32) == kt) --f;
        sh.part[0] = kt;
        sh.part[1] = static_cast<uint64_t>(i - f + 1);
    }
    __syncthreads();
    *tau = static_cast<uint32_t>(sh.part[0]);
    *k = sh.part[1];
    __syncthreads();
}

// DEPTH: float4 loads in flight per lane in the passes; WPE: waves per SIMD
// the build allows.  More than 256 rows: 8 waves per SIMD, so two rows share
// a CU (the LDS fits two workgroups) and one row's serial steps overlap the
// other's passes, at 64 registers and 4 loads per lane.  Up to 256 rows each
// CU holds one row anyway, so its lanes keep 8 loads in flight instead.
template <int DEPTH, int WPE>
__global__ __launch_bounds__(kThreads, WPE) void sample_top_p_kernel(SampleArgs a) {
    __shared__ SelShared sh;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t r = blockIdx.x;
    const float *y = a.logits + r * a.ld;
    const int V = a.V;
    const int nvec = (V + 3) / 4;                 // float4 groups (the row is padded past V)
    const int nchunks = (V + kChunk - 1) / kChunk;

    // ---- row max from the tile maxima
    float m = -INFINITY;
    for (int t = tid; t < a.n_partials; t += kThreads) m = fmaxf(m, a.pm[static_cast<int64_t>(t) * a.rows + r]);
    m = wave_max(m);
    if (lane == 0) sh.fred[wave] = m;
    for (int i = tid; i < kBuckets; i += kThreads) sh.a.hist[i] = 0;
    __syncthreads();
    for (int w = 0; w < kWaves; ++w) m = fmaxf(m, sh.fred[w]);

    // ---- pass 1: bucket masses (a bucket's token count is not needed: pass 2
    // gathers the tokens of one bucket and counts them as it goes)
    scan_groups<DEPTH>(y, V, tid, nvec, kThreads, [&](int, float yv) {
        const uint64_t q = qmass(yv, m);
        if (q)
            atomicAdd(reinterpret_cast<unsigned long long *>(&sh.a.hist[bucket_of(yv, m)]),
                      static_cast<unsigned long long>(q));
    });
    __syncthreads();

    // ---- the total mass Z (the histogram's sum) and the bucket where the
    // ranked mass reaches T (buckets run from the max down)
    constexpr int kPer = kBuckets / kThreads;
    uint64_t mine = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) mine += sh.a.hist[tid * kPer + j];
    uint64_t before;
    const uint64_t Z = block_excl_scan(sh, mine, &before);
    uint64_t T = a.top_p >= 1.f ? Z : static_cast<uint64_t>(ceil(static_cast<double>(a.top_p) * static_cast<double>(Z)));
    if (T < 1) T = 1;
    if (T > Z) T = Z;
    if (tid == 0) {                              // defaults, in range, for a degenerate row
        sh.part[0] = 0;
        sh.zsum[0] = kBuckets - 1;
    }
    __syncthreads();
    if (before < T && before + mine >= T) {
        uint64_t acc = before;
        int b = tid * kPer;
        while (acc + sh.a.hist[b] < T) acc += sh.a.hist[b++];
        sh.part[0] = acc;                        // mass above the bucket
        sh.zsum[0] = static_cast<uint64_t>(b);
    }
    __syncthreads();
    uint64_t above = sh.part[0];
    const int B = static_cast<int>(sh.zsum[0]);
    if (tid == 0) sh.ncand = 0;
    __syncthreads();                             // the histogram is free from here

    // ---- pass 2: per chunk of ids the mass of the buckets above B, and the
    // tokens of B gathered for sorting (at most kCap of them stored; the
    // counter keeps counting past kCap)
    for (int c = wave; c < nchunks; c += kWaves) {
        uint64_t ms = 0;
        scan_groups<DEPTH>(y, V, c * (kChunk / 4) + lane, min(nvec, (c + 1) * (kChunk / 4)), 64, [&](int v, float yv) {
            const int b = bucket_of(yv, m);
            if (b < B) {
                ms += qmass(yv, m);
            } else if (b == B) {
                const uint32_t slot = atomicAdd(&sh.ncand, 1u);
                if (slot < kCap)
                    sh.b.cand[slot] = (static_cast<uint64_t>(fkey(yv)) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(v));
            }
        });
        ms = wave_sum_int(ms);
        if (lane == 0) {
            sh.a.chunk.mass[c] = ms;
            sh.a.chunk.ties[c] = 0;
        }
    }
    __syncthreads();
    uint32_t ncand = sh.ncand;                   // tokens in bucket B
    __syncthreads();

    uint32_t tau;
    uint64_t k;
    if (ncand <= kCap) {
        // ---- fast path: sort the gathered tokens
        sort_and_walk(sh, ncand, above, T, m, &tau, &k);
        // the candidates complete the chunk masses (key above tau) and tie counts
        for (int i = tid; i < static_cast<int>(ncand); i += kThreads) {
            const uint32_t kk = static_cast<uint32_t>(sh.b.cand[i] >> 32);
            const int c = static_cast<int>(~static_cast<uint32_t>(sh.b.cand[i])) / kChunk;
            if (kk > tau)
                atomicAdd(reinterpret_cast<unsigned long long *>(&sh.a.chunk.mass[c]),
                          static_cast<unsigned long long>(qmass(key_to_float(kk), m)));
            else if (kk == tau)
                atomicAdd(&sh.a.chunk.ties[c], 1u);
        }
        __syncthreads();
    } else {
        // ---- B holds more than kCap tokens: refine the set (bucket B, key >>
        // shift == prefix) by 8-bit key digits until it fits or is one key
        int shift = 32;
        uint32_t prefix = 0;
        bool ties_only = false;
        for (;;) {
            if (shift == 0) {
                ties_only = true;                // more than kCap tokens share one key
                break;
            }
            const int s2 = shift - 8;
            for (int i = tid; i < 256; i += kThreads) {
                sh.a.hist[i] = 0;
                sh.dcount[i] = 0;
            }
            __syncthreads();
            scan_groups<DEPTH>(y, V, tid, nvec, kThreads, [&](int, float yv) {
                const uint32_t kk = fkey(yv);
                if (bucket_of(yv, m) == B && (shift == 32 || (kk >> shift) == prefix)) {
                    const int d = (kk >> s2) & 255;
                    atomicAdd(reinterpret_cast<unsigned long long *>(&sh.a.hist[d]),
                              static_cast<unsigned long long>(qmass(yv, m)));
                    atomicAdd(&sh.dcount[d], 1u);
                }
            });
            __syncthreads();
            if (tid == 0) {
                // digits from the largest key down
                uint64_t acc = above;
                int d = 255;
                while (d > 0 && (acc + sh.a.hist[d] < T || sh.dcount[d] == 0)) acc += sh.a.hist[d--];
                sh.part[0] = acc;
                sh.zsum[0] = static_cast<uint64_t>(d);
            }
            __syncthreads();
            above = sh.part[0];
            const uint32_t d = static_cast<uint32_t>(sh.zsum[0]);
            prefix = (shift == 32 ? 0u : (prefix << 8)) | d;
            shift = s2;
            ncand = sh.dcount[d];
            __syncthreads();
            if (ncand <= kCap) break;
        }
        if (ties_only) {
            tau = prefix;
            const uint64_t qt = qmass(key_to_float(tau), m);
            k = qt ? (T - above + qt - 1) / qt : ncand;
            if (k > ncand) k = ncand;
        } else {
            if (tid == 0) sh.ncand = 0;
            __syncthreads();
            scan_groups<DEPTH>(y, V, tid, nvec, kThreads, [&](int v, float yv) {
                const uint32_t kk = fkey(yv);
                if (bucket_of(yv, m) == B && (kk >> shift) == prefix) {
                    const uint32_t slot = atomicAdd(&sh.ncand, 1u);
                    sh.b.cand[slot] = (static_cast<uint64_t>(kk) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(v));
                }
            });
            __syncthreads();
            sort_and_walk(sh, ncand, above, T, m, &tau, &k);
        }
        // per chunk: mass of members above tau and count of key-tau tokens
        for (int c = wave; c < nchunks; c += kWaves) {
            uint64_t ms = 0;
            uint32_t nt = 0;
            scan_groups<DEPTH>(y, V, c * (kChunk / 4) + lane, min(nvec, (c + 1) * (kChunk / 4)), 64, [&](int, float yv) {
                const uint32_t kk = fkey(yv);
                if (kk > tau) ms += qmass(yv, m);
                nt += kk == tau;
            });
            ms = wave_sum_int(ms);
            nt = wave_sum_int(nt);
            if (lane == 0) {
                sh.a.chunk.mass[c] = ms;
                sh.a.chunk.ties[c] = nt;
            }
        }
        __syncthreads();
    }

    const uint64_t qt = qmass(key_to_float(tau), m);
    // ---- the nucleus mass per chunk of ids: its members above tau plus the
    // key-tau tokens among the first k of them in id order; then the chunk
    // where the running mass passes U = floor(u Z_N).  Wave 0, 64 chunks at
    // a time, with wave scans of the tie counts and masses.
    if (wave == 0) {
        auto chunk_mass = [&](int c0, uint64_t tb, uint64_t *ti, uint64_t *tbx, uint64_t *mc) {
            const int c = c0 + lane;
            const uint64_t t = c < nchunks ? sh.a.chunk.ties[c] : 0;
            *ti = wave_incl_scan(t, lane);
            *tbx = tb + *ti - t;                                   // key-tau tokens in earlier chunks
            const uint64_t inc = min(t, k > *tbx ? k - *tbx : 0);
            *mc = c < nchunks ? sh.a.chunk.mass[c] + inc * qt : 0;
        };
        uint64_t zn = 0, tb = 0;
        for (int c0 = 0; c0 < nchunks; c0 += 64) {
            uint64_t ti, tbx, mc;
            chunk_mass(c0, tb, &ti, &tbx, &mc);
            zn += wave_sum_int(mc);
            tb += __shfl(ti, 63, 64);
        }
        uint64_t U = static_cast<uint64_t>(floor(static_cast<double>(a.uniform[r]) * static_cast<double>(zn)));
        if (!(U < zn)) U = zn ? zn - 1 : 0;
        uint64_t cum = 0;
        tb = 0;
        int cs = -1;
        uint64_t tb_cs = 0, cum_cs = 0;
        for (int c0 = 0; c0 < nchunks; c0 += 64) {
            uint64_t ti, tbx, mc;
            chunk_mass(c0, tb, &ti, &tbx, &mc);
            const uint64_t mi = wave_incl_scan(mc, lane);
            const uint64_t hits = __ballot(c0 + lane < nchunks && cum + mi > U);   // the running mass passes U
            if (hits) {
                const int src = __builtin_ctzll(hits);
                cs = c0 + src;
                tb_cs = __shfl(tbx, src, 64);
                cum_cs = cum + __shfl(mi - mc, src, 64);
                break;
            }
            cum += __shfl(mi, 63, 64);
            tb += __shfl(ti, 63, 64);
        }
        if (cs < 0) {                            // no chunk passes U (a row without mass)
            cs = nchunks - 1;
            tb_cs = tb;
            cum_cs = cum;
        }
        if (lane == 0) {
            sh.part[0] = static_cast<uint64_t>(cs);
            sh.part[1] = tb_cs;
            sh.part[2] = U - min(U, cum_cs);
            sh.part[3] = zn;
        }
    }
    __syncthreads();

    // ---- rescan the chunk in id order (wave 0)
    if (wave == 0) {
        const int cs = static_cast<int>(sh.part[0]);
        uint64_t tie_base = sh.part[1];
        const uint64_t need = sh.part[2];        // the sample is where the running mass passes this
        uint64_t run = 0;
        int found = -1, last = -1;
        for (int g0 = cs * (kChunk / 4); g0 < min(nvec, (cs + 1) * (kChunk / 4)); g0 += 64) {
            const int g = g0 + lane;
            uint64_t qe[4] = {0, 0, 0, 0};
            uint32_t te[4] = {0, 0, 0, 0};
            uint32_t kk[4] = {0, 0, 0, 0};
            if (g < nvec) {
                const float4 y4 = *reinterpret_cast<const float4 *>(y + 4 * g);
                const float yy[4] = {y4.x, y4.y, y4.z, y4.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (4 * g + e < V) {
                        kk[e] = fkey(yy[e]);
                        te[e] = kk[e] == tau;
                        qe[e] = (kk[e] > tau || kk[e] == tau) ? qmass(yy[e], m) : 0;
                    }
                }
            }
            // tie ranks in id order decide which key-tau tokens are members
            const uint32_t tl = te[0] + te[1] + te[2] + te[3];
            const uint32_t tinc = wave_incl_scan(tl, lane);
            uint64_t rank = tie_base + (tinc - tl);
            uint64_t mq[4];
            uint64_t ml = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                bool member = kk[e] > tau;
                if (te[e]) {
                    member = rank < k;
                    ++rank;
                }
                mq[e] = member ? qe[e] : 0;
                if (member && 4 * g + e < V) last = 4 * g + e;
                ml += mq[e];
            }
            const uint64_t minc = wave_incl_scan(ml, lane);
            uint64_t acc = run + (minc - ml);
            int hit = -1;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (hit < 0 && mq[e] && acc + mq[e] > need) hit = 4 * g + e;
                acc += mq[e];
            }
            const uint64_t hits = __ballot(hit >= 0);
            if (hits) {
                const int src = __builtin_ctzll(hits);
                found = __shfl(hit, src, 64);
                break;
            }
            run += __shfl(minc, 63, 64);
            tie_base += __shfl(tinc, 63, 64);
        }
        // a member always holds the sample; the last member covers rounding
        if (found < 0) {
            int lm = last;
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) lm = max(lm, __shfl_xor(lm, o, 64));
            found = lm;
        }
        if (lane == 0) {
            const int t = found < 0 ? 0 : found;
            a.token[r] = t;
            if (a.logprob) {
                const double zn_full = static_cast<double>(Z) / static_cast<double>(kMassScale);   // sum exp(y - m)
                a.logprob[r] = static_cast<float>(static_cast<double>(y[t] - m) - log(zn_full));
            }
        }
    }
}

}  // namespace

hipError_t launch_sample_top_p(const SampleArgs &a, hipStream_t stream) {
    if (a.rows == 0) return hipSuccess;
    if (a.rows > 256)
        hipLaunchKernelGGL((sample_top_p_kernel<4, 8>), dim3(static_cast<uint32_t>(a.rows)), dim3(kThreads), 0, stream,
                           a);
    else
        hipLaunchKernelGGL((sample_top_p_kernel<8, 4>), dim3(static_cast<uint32_t>(a.rows)), dim3(kThreads), 0, stream,
                           a);
    return hipGetLastError();
}

}  // namespace rlk
