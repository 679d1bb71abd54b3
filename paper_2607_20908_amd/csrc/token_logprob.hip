// Fused lm-head token log-prob for gfx950.
//
// Tile kernel: one workgroup (8 wave64s, 2 x 4, two per SIMD) computes the
// 256 x 256 logit tile  Z^T = W_tile * hidden_tile^T  (vocab entries on the M
// side, token rows on the N side); each wave owns 128 vocab x 64 rows as
// 4 x 2 MFMA 32x32x16 bf16 tiles with fp32 accumulation.  Both operands are
// hidden-contiguous.  The hidden dimension streams through two LDS stages of
// 64 entries (XOR-swizzled 16-byte chunks); global loads run two stages ahead
// in two alternating register sets, so each load has two compute phases to
// land.  Rows past the vocabulary or the batch re-read the last valid row:
// their logits are masked (vocab) or never written (rows).
// The epilogue never stores the logits: per token row it
// takes the max and the sum of exp2 over the tile's vocab entries (the vocab
// index lives in the accumulator registers, so the reduction is in-lane plus
// one cross-half shuffle), picks out the target's logit when the target falls
// in the tile, and writes one (max, sum) partial per (vocab tile, row).
// Combine kernel: per row, merge the partials of all vocab tiles into the
// log-sum-exp and subtract it from the target logit.
#include "device_common.h"
#include "kernels.h"

namespace rlk {
namespace {

constexpr int kThreads = 256;
constexpr int kK = kHiddenStep;                 // 64 hidden entries per LDS stage
constexpr int kTileElems = kVocabTile * kK;     // bf16 elements per operand per stage
static_assert(kVocabTile == kRowTile, "square tiles assumed below");

// Element offset of 16-byte chunk c (0..7) of tile row `row` in a stage buffer.
// Rows are 128 bytes, so two rows share one 256-byte window of the 64 LDS
// banks; XOR-ing the chunk with row bits 1..3 gives the 16 rows that one
// ds_read_b128 pass serves (same chunk, consecutive rows) 16 distinct 16-byte
// slots of that window, and keeps the register-to-LDS stores conflict-free.
__device__ __forceinline__ int op_off(int row, int c) { return row * kK + ((c ^ ((row >> 1) & 7)) << 3); }

// Maps the launch index to a (vocab tile, row tile).  The hardware hands
// consecutive workgroups to the 8 XCDs in turn; renumbering gives each XCD a
// contiguous run of logical tiles, and inside a run 4 row tiles sweep the
// vocabulary together, so a weight tile is fetched into an XCD's L2 once for
// 4 row tiles and the row tiles stay resident in L2 / the MALL.
__device__ __forceinline__ void tile_of(int64_t b, int64_t nvt, int64_t nrt, int64_t *vt, int64_t *rt) {
    const int64_t total = nvt * nrt;
    const int64_t full = total / 8 * 8;
    const int64_t L = b < full ? (b % 8) * (total / 8) + b / 8 : b;
    constexpr int64_t GR = 4;
    const int64_t group = L / (GR * nvt);
    const int64_t in = L % (GR * nvt);
    const int64_t rows_in_group = min(GR, nrt - group * GR);
    *rt = group * GR + in % rows_in_group;
    *vt = in / rows_in_group;
}

constexpr int kTileThreads = 512;
constexpr int kLoadsPerOperand = kTileElems / 8 / kTileThreads;   // 16-byte chunks per thread
static_assert(kLoadsPerOperand == 4, "staging layout");

__global__ __launch_bounds__(kTileThreads, 1) void logprob_tile_kernel(LogprobArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t smem[2 * 2 * kTileElems];   // [buf][W, hidden]
    __shared__ float red[2][kRowTile][2];                                        // [vocab half][row][m, l]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wv = wave & 1, wr = wave >> 1;     // vocab half (128 entries), row quarter (64 rows)
    const int l32 = lane & 31, h2 = lane >> 5;
    int64_t vt, rt;
    tile_of(blockIdx.x, a.n_vocab_tiles, a.n_row_tiles, &vt, &rt);
    const int64_t v0 = vt * kVocabTile, r0 = rt * kRowTile;
    const int64_t H = a.H;

    // ---- staging: per stage, 4 chunks of W and 4 of hidden per thread -------
    // Rows past the vocabulary / the batch re-read the last valid row (the
    // bounds are uniform; full tiles never clamp).
    const uint16_t *wg = a.w + v0 * H;
    const uint16_t *hg = a.hidden + r0 * H;
    const int wlast = static_cast<int>(min(static_cast<int64_t>(kVocabTile - 1), a.V - 1 - v0));
    const int hlast = static_cast<int>(min(static_cast<int64_t>(kRowTile - 1), a.R - 1 - r0));
    u32x4 ra0[kLoadsPerOperand], rb0[kLoadsPerOperand], ra1[kLoadsPerOperand], rb1[kLoadsPerOperand];
    auto load_stage = [&](int ks, u32x4 *ra, u32x4 *rb) {
        const int k0 = ks * kK;
#pragma unroll
        for (int j = 0; j < kLoadsPerOperand; ++j) {
            const int idx = tid + j * kTileThreads;
            const int row = idx >> 3, c = idx & 7;
            ra[j] = *reinterpret_cast<const u32x4 *>(wg + min(row, wlast) * H + k0 + c * 8);
            rb[j] = *reinterpret_cast<const u32x4 *>(hg + min(row, hlast) * H + k0 + c * 8);
        }
    };
    auto store_stage = [&](int buf, const u32x4 *ra, const u32x4 *rb) {
        uint16_t *as = smem + buf * 2 * kTileElems;
        uint16_t *bs = as + kTileElems;
#pragma unroll
        for (int j = 0; j < kLoadsPerOperand; ++j) {
            const int idx = tid + j * kTileThreads;
            const int row = idx >> 3, c = idx & 7;
            *reinterpret_cast<u32x4 *>(as + op_off(row, c)) = ra[j];
            *reinterpret_cast<u32x4 *>(bs + op_off(row, c)) = rb[j];
        }
    };

    f32x16 acc[4][2];
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) acc[tm][tn] = f32x16{};

    auto compute_stage = [&](int buf) {
        const uint16_t *as = smem + buf * 2 * kTileElems;
        const uint16_t *bs = as + kTileElems;
#pragma unroll
        for (int kq = 0; kq < kK / 16; ++kq) {
            const int c = kq * 2 + h2;
            bf16x8 af[4], bf[2];
#pragma unroll
            for (int tm = 0; tm < 4; ++tm)
                af[tm] = *reinterpret_cast<const bf16x8 *>(as + op_off(wv * 128 + tm * 32 + l32, c));
#pragma unroll
            for (int tn = 0; tn < 2; ++tn)
                bf[tn] = *reinterpret_cast<const bf16x8 *>(bs + op_off(wr * 64 + tn * 32 + l32, c));
#pragma unroll
            for (int tm = 0; tm < 4; ++tm)
#pragma unroll
                for (int tn = 0; tn < 2; ++tn)
                    acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[tm], bf[tn], acc[tm][tn], 0, 0, 0);
        }
    };

    // Stage ks lives in LDS buffer ks % 2; odd stages pass through register set
    // 0, even stages >= 2 through set 1, each loaded two stages ahead.
    const int nk = a.H / kK;
    load_stage(0, ra0, rb0);
    store_stage(0, ra0, rb0);
    if (nk > 1) load_stage(1, ra0, rb0);
    if (nk > 2) load_stage(2, ra1, rb1);
    __syncthreads();
    for (int ks = 0; ks < nk; ks += 2) {
        compute_stage(0);
        if (ks + 1 < nk) {
            store_stage(1, ra0, rb0);
            if (ks + 3 < nk) load_stage(ks + 3, ra0, rb0);
        }
        __syncthreads();
        if (ks + 1 < nk) {
            compute_stage(1);
            if (ks + 2 < nk) {
                store_stage(0, ra1, rb1);
                if (ks + 4 < nk) load_stage(ks + 4, ra1, rb1);
            }
            __syncthreads();
        }
    }

    // ---- epilogue: per token row, max / sum of exp2 / target logit ---------
    // acc[tm][tn][i] holds vocab v0 + wv*128 + tm*32 + 8*(i/4) + 4*h2 + i%4
    // for token row r0 + wr*64 + tn*32 + l32.
    const float c2 = a.inv_temperature * kLog2e;
    const int64_t vbase = v0 + wv * 128;
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
        const int64_t rr = r0 + wr * 64 + tn * 32 + l32;
        // target logit, if the target lies in this wave's 128 vocab entries
        if (rr < a.R) {
            const int64_t local = static_cast<int64_t>(a.target[rr]) - vbase;
            if (local >= 0 && local < 128) {
                const int tmt = static_cast<int>(local >> 5), rem = static_cast<int>(local & 31);
                const int it = ((rem >> 3) << 2) | (rem & 3);
                if (((rem >> 2) & 1) == h2) {
                    float val = 0.f;
#pragma unroll
                    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            if (tm == tmt && i == it) val = acc[tm][tn][i];
                    a.zt[rr] = val * a.inv_temperature;
                }
            }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int tm = 0; tm < 4; ++tm)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int64_t v = vbase + tm * 32 + 8 * (i >> 2) + 4 * h2 + (i & 3);
                const float x = v < a.V ? acc[tm][tn][i] * c2 : -INFINITY;
                acc[tm][tn][i] = x;
                mx = fmaxf(mx, x);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float mu = mx == -INFINITY ? 0.f : mx;
        float sum = 0.f;
#pragma unroll
        for (int tm = 0; tm < 4; ++tm)
#pragma unroll
            for (int i = 0; i < 16; ++i) sum += fast_exp2(acc[tm][tn][i] - mu);
        sum += __shfl_xor(sum, 32, 64);
        if (h2 == 0) {
            red[wv][wr * 64 + tn * 32 + l32][0] = mx;
            red[wv][wr * 64 + tn * 32 + l32][1] = sum;
        }
    }
    __syncthreads();
    if (tid < kRowTile) {
        const int row = tid;
        const int64_t rr = r0 + row;
        if (rr < a.R) {
            const float m0 = red[0][row][0], m1 = red[1][row][0];
            const float Mx = fmaxf(m0, m1);
            const float L = red[0][row][1] * fast_exp2(m0 - Mx) + red[1][row][1] * fast_exp2(m1 - Mx);
            a.pm[vt * a.R + rr] = Mx;
            a.pl[vt * a.R + rr] = L;
        }
    }
}

// Online log-sum-exp merge of (max, sum) partials, both in log2 units.
__device__ __forceinline__ void lse_merge(float &M, float &L, float m, float l) {
    if (m > M) {
        L = L * fast_exp2(M - m) + l;
        M = m;
    } else {
        L += l * fast_exp2(m - M);
    }
}

__device__ __forceinline__ void finish_row(const LogprobArgs &a, int64_t r, float M, float L) {
    const float lse = (M + fast_log2(L)) * kLn2;
    const int32_t t = a.target[r];
    float lp;
    if (t == -1) lp = 0.f;
    else if (t >= 0 && t < a.V) lp = a.zt[r] - lse;
    else lp = __builtin_nanf("");
    a.logprob[r] = lp;
    if (a.lse) a.lse[r] = lse;
}

// Few rows: one wave per row, lanes stride over the vocab tiles.
__global__ __launch_bounds__(kThreads) void logprob_combine_wave_kernel(LogprobArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t r = static_cast<int64_t>(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
    if (r >= a.R) return;
    float M = -INFINITY, L = 0.f;
    for (int64_t vt = lane; vt < a.n_vocab_tiles; vt += 64) lse_merge(M, L, a.pm[vt * a.R + r], a.pl[vt * a.R + r]);
    const float Mw = wave_max(M);
    const float Lw = wave_sum(M == -INFINITY ? 0.f : L * fast_exp2(M - Mw));
    if (lane == 0) finish_row(a, r, Mw, Lw);
}

// Many rows: one thread per row; neighbouring threads read neighbouring rows
// of each vocab tile's partials (coalesced).
__global__ __launch_bounds__(kThreads) void logprob_combine_row_kernel(LogprobArgs a) {
    const int64_t r = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (r >= a.R) return;
    float M = -INFINITY, L = 0.f;
    int64_t vt = 0;
    for (; vt + 4 <= a.n_vocab_tiles; vt += 4) {
        float m[4], l[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            m[j] = a.pm[(vt + j) * a.R + r];
            l[j] = a.pl[(vt + j) * a.R + r];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) lse_merge(M, L, m[j], l[j]);
    }
    for (; vt < a.n_vocab_tiles; ++vt) lse_merge(M, L, a.pm[vt * a.R + r], a.pl[vt * a.R + r]);
    finish_row(a, r, M, L);
}

}  // namespace

hipError_t launch_logprob(const LogprobArgs &a, hipStream_t stream) {
    const int64_t tiles = static_cast<int64_t>(a.n_vocab_tiles) * a.n_row_tiles;
    hipLaunchKernelGGL(logprob_tile_kernel, dim3(static_cast<uint32_t>(tiles)), dim3(kTileThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.R < 32768) {
        const int64_t blocks = (a.R + 3) / 4;
        hipLaunchKernelGGL(logprob_combine_wave_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0,
                           stream, a);
    } else {
        const int64_t blocks = (a.R + kThreads - 1) / kThreads;
        hipLaunchKernelGGL(logprob_combine_row_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0,
                           stream, a);
    }
    return hipGetLastError();
}

}  // namespace rlk
