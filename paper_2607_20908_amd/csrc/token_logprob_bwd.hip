// Backward of the lm-head token log-prob with respect to the hidden rows, for
// gfx950.  With z = W h, p = softmax(inv_T z) and logprob = inv_T z_t - lse:
//   d logprob / d h = inv_T (W[t] - sum_v p_v W[v]),
// scaled per row by the incoming gradient g.  The lm-head weight is frozen
// (only adapters train), so no weight gradient is formed.
//
// Per chunk of rows:
//   1. the forward tile kernel recomputes the logits and writes p as bf16 in a
//      blocked layout (one 32 KB block per 256 rows x 64 vocab entries, in the
//      LDS image the GEMM below stages), given the forward's lse;
//   2. this file's GEMM forms  S = P W  (rows x hidden, contraction over the
//      vocabulary) on bf16 MFMA with fp32 accumulation, split over the
//      vocabulary when the chunk has too few output tiles to fill the GPU;
//   3. the finish kernel sums the splits and writes
//      dh = g inv_T (W[t] - S)  (0 for masked rows, NaN for invalid targets).
//
// The GEMM's B operand is W[v][h] with the contraction index v as the row:
// a 64 x 256 band of W is copied row-contiguous into LDS and read with the
// transposing ds_read_b64_tr_b16, which hands each lane 4 consecutive v of one
// column h.
#include "device_common.h"
#include "kernels.h"
#include "lds_stage.h"

namespace rlk {
namespace {

constexpr int kThreads = 256;                   // finish kernel
constexpr int kTileElems = 256 * 64;            // one stage of one operand, bf16 elements
constexpr int kGemmThreads = 64 * kBwdGemmWaves;   // 8 waves, two per SIMD
constexpr int kBlocksPerWave = kTileElems / 512 / kBwdGemmWaves;   // 1 KB blocks per wave per operand per stage
static_assert(kBlocksPerWave == 4, "staging layout");

// gfx950 transposing LDS read: in each group of 16 lanes, lane s supplies the
// address of 4 consecutive bf16; seen as a 4 x 16 block whose row k holds the
// values of lanes 4k..4k+3 in order, lane n receives column n (rows 0..3).
__device__ __forceinline__ bf16x4 lds_read_tr16(const uint16_t *p) {
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    typedef s16x4 __attribute__((address_space(3))) *lds_s16x4;
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(p));
    return __builtin_bit_cast(bf16x4, v);
}

// S[rows, h] over one vocabulary range; one workgroup of 8 waves (two per
// SIMD) per 256 x 256 output tile, each wave 128 rows x 64 hidden entries as
// 4 x 2 MFMA 32x32x16 tiles, so one wave of a SIMD issues its loads and LDS
// reads while the other runs MFMAs.
template <int WS>
__global__ __launch_bounds__(kGemmThreads, 1) void logprob_bwd_gemm_kernel(LogprobBwdArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t bring[WS * kTileElems];   // W bands [64 v][256 h]
    __shared__ __attribute__((aligned(16))) uint16_t aring[2 * kTileElems];    // probabilities [256 rows][64 v]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1, wn = wave >> 1;     // row half, hidden quarter
    const int l32 = lane & 31, h2 = lane >> 5;
    int split, ht, rt;
    gemm_tile_of(blockIdx.x, a.n_h_tiles, a.n_row_tiles, a.splits, &split, &ht, &rt);
    const int H = a.H;
    const int h0 = ht * 256;
    const int ks0 = split * a.steps_per_split;
    const int nks = min(a.steps_per_split, a.n_vsteps - ks0);

    // ---- staging.  Probabilities: the blocked buffer already holds the LDS
    // image, so block j of a stage is a plain 1 KB copy.  W: block blk holds
    // band rows 2 blk and 2 blk + 1; lane i fills slot i % 32 of row
    // 2 blk + i / 32 with chunk slot ^ (4 * (row % 4)).  Rows past the
    // vocabulary re-read the last row (their probabilities are 0); columns
    // past the hidden size re-read the last chunk (never stored).
    const int clast = bwd_clast(H, h0);
    auto abuf = [&](int s) { return aring + (s & 1) * kTileElems; };
    auto bbuf = [&](int s) { return bring + (s % WS) * kTileElems; };
    // saddr-form loads: wave-uniform bases (scalar arithmetic only) and
    // per-lane byte offsets fixed for the whole loop; for W, one table for
    // blocks whose second row exists and one for the last rows
    const uint32_t aring_l = lds_addr(aring), bring_l = lds_addr(bring);
    const uint32_t avoff = bwd_a_voff(lane);
    uint32_t bvoff_pair[kBlocksPerWave], bvoff_same[kBlocksPerWave];
#pragma unroll
    for (int j = 0; j < kBlocksPerWave; ++j) {
        const int row = bwd_b_row(wave * kBlocksPerWave + j, lane);
        const int c = bwd_b_chunk(row, lane);
        bvoff_pair[j] = bwd_b_voff(lane, true, c, clast, H);
        bvoff_same[j] = bwd_b_voff(lane, false, c, clast, H);
    }
    auto issue_a = [&](int slot, int j) {
        const int blk = wave * kBlocksPerWave + j;
        load_lds16_s(a.probs + bwd_a_base(rt, a.n_vsteps, ks0, slot, nks, blk), avoff,
                     aring_l + ((slot & 1) * kTileElems + blk * 512) * 2);
    };
    auto issue_b = [&](int slot, int j) {
        const int blk = wave * kBlocksPerWave + j;
        const int64_t first = bwd_b_first(ks0, slot, nks, blk);
        load_lds16_s(a.w + bwd_b_base_row(first, a.V) * H + h0, bwd_b_pair(first, a.V) ? bvoff_pair[j] : bvoff_same[j],
                     bring_l + ((slot % WS) * kTileElems + blk * 512) * 2);
    };

    f32x16 acc[4][2];
#pragma unroll
    for (int tm = 0; tm < 4; ++tm)
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) acc[tm][tn] = f32x16{};

    // transposing-read address of this lane, relative to a band and k-step:
    // lanes 16q..16q+15 read rows 8 (q/2) + 4 e + s/4 at hidden entries
    // 16 (q%2) + 4 (s%4) of the 32-wide block j
    const int q = lane >> 4, s = lane & 15;
    const int brow = 8 * (q >> 1) + (s >> 2);
    int boff[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int hl = wn * 64 + j * 32 + 16 * (q & 1) + 4 * (s & 3);
        boff[j] = band_off(brow, hl >> 3) + (hl & 7);
    }
    bf16x8 fa[2][4], fb[2][2];
    auto read_frags = [&](int ks, int kq, int p) {
        const uint16_t *as = abuf(ks);
        const uint16_t *bs = bbuf(ks) + kq * 16 * 256;
        const int c = kq * 2 + h2;
#pragma unroll
        for (int i = 0; i < 4; ++i) fa[p][i] = *reinterpret_cast<const bf16x8 *>(as + op_off(wm * 128 + i * 32 + l32, c));
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const bf16x4 lo = lds_read_tr16(bs + boff[j]);
            const bf16x4 hi = lds_read_tr16(bs + boff[j] + 4 * 256);
            fb[p][j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
    };
    auto mfma_step = [&](int p) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[p][i], fb[p][j], acc[i][j], 0, 0, 0);
    };

    // Same ring discipline as the forward tile kernel: stage s lives in
    // probability buffer s % 2 and W buffer s % WS; at the end of stage s the
    // loads of stage s + 2 (probabilities) and s + WS (W) are issued.
#pragma unroll
    for (int j = 0; j < kBlocksPerWave; ++j) issue_a(0, j);
#pragma unroll
    for (int j = 0; j < kBlocksPerWave; ++j) issue_b(0, j);
#pragma unroll
    for (int j = 0; j < kBlocksPerWave; ++j) issue_a(1, j);
#pragma unroll
    for (int j = 0; j < kBlocksPerWave; ++j) issue_b(1, j);
    if (WS == 3) {
#pragma unroll
        for (int j = 0; j < kBlocksPerWave; ++j) issue_b(2, j);
    }
    wait_vm<(WS == 3 ? 3 : 2) * kBlocksPerWave>();
    barrier();
    read_frags(0, 0, 0);
    for (int ks = 0; ks < nks; ++ks) {
#pragma unroll
        for (int kq = 0; kq < 3; ++kq) {
            read_frags(ks, kq + 1, (kq + 1) & 1);
            mfma_step(kq & 1);
        }
        wait_vm<(WS == 3 ? 1 : 0) * kBlocksPerWave>();
        wait_lds();
        barrier();
        // one load, one MFMA of this k-step's last quarter and one fragment
        // read of stage ks + 1 per group (the B fragments in groups 4 and 5)
        {
            const uint16_t *as = abuf(ks + 1);
            const uint16_t *bs = bbuf(ks + 1);
#pragma unroll
            for (int g = 0; g < 8; ++g) {
                if (g < 4) issue_a(ks + 2, g);
                else issue_b(ks + WS, g - 4);
                acc[g >> 1][g & 1] =
                    __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][g >> 1], fb[1][g & 1], acc[g >> 1][g & 1], 0, 0, 0);
                if (g < 4) {
                    fa[0][g] = *reinterpret_cast<const bf16x8 *>(as + op_off(wm * 128 + g * 32 + l32, h2));
                } else if (g < 6) {
                    const bf16x4 lo = lds_read_tr16(bs + boff[g - 4]);
                    const bf16x4 hi = lds_read_tr16(bs + boff[g - 4] + 4 * 256);
                    fb[0][g - 4] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
    wait_vm<0>();

    // ---- epilogue: acc[tm][tn][i] is S at row wm*128 + tm*32 + 8*(i/4) +
    // 4*h2 + i%4 of the tile, hidden entry wn*64 + tn*32 + l32.
    const int64_t rows_pad = static_cast<int64_t>(a.n_row_tiles) * 256;
    float *out = a.dpart + bwd_out_base(split, rows_pad, rt, H, h0);
    const int64_t rlim = a.rows - static_cast<int64_t>(rt) * 256;
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
        const int h = wn * 64 + tn * 32 + l32;
        if (h0 + h >= H) continue;
#pragma unroll
        for (int tm = 0; tm < 4; ++tm)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int row = wm * 128 + tm * 32 + 8 * (i >> 2) + 4 * h2 + (i & 3);
                if (row < rlim) out[bwd_out_off(row, H, h)] = acc[tm][tn][i];
            }
    }
}

// dh = g inv_T (W[t] - sum over splits of S); 4 hidden entries per thread.
__global__ __launch_bounds__(kThreads) void logprob_bwd_finish_kernel(LogprobBwdArgs a) {
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    const int64_t per_row = a.H / 4;
    if (idx >= a.rows * per_row) return;
    const int64_t r = idx / per_row;
    const int h = static_cast<int>(idx % per_row) * 4;
    const int32_t t = a.target[r];
    float4 o;
    if (t == -1) {
        o = make_float4(0.f, 0.f, 0.f, 0.f);
    } else if (t < 0 || t >= a.V) {
        const float nan = __builtin_nanf("");
        o = make_float4(nan, nan, nan, nan);
    } else {
        const int64_t rows_pad = static_cast<int64_t>(a.n_row_tiles) * 256;
        float4 sacc = *reinterpret_cast<const float4 *>(a.dpart + bwd_part_elem(0, rows_pad, r, a.H, h));
        for (int sp = 1; sp < a.splits; ++sp) {
            const float4 x = *reinterpret_cast<const float4 *>(a.dpart + bwd_part_elem(sp, rows_pad, r, a.H, h));
            sacc.x += x.x;
            sacc.y += x.y;
            sacc.z += x.z;
            sacc.w += x.w;
        }
        const uint2 wb = *reinterpret_cast<const uint2 *>(a.w + static_cast<int64_t>(t) * a.H + h);
        const float w0 = __uint_as_float(wb.x << 16), w1 = __uint_as_float(wb.x & 0xffff0000u);
        const float w2 = __uint_as_float(wb.y << 16), w3 = __uint_as_float(wb.y & 0xffff0000u);
        const float sc = a.grad[r] * a.inv_temperature;
        o = make_float4(sc * (w0 - sacc.x), sc * (w1 - sacc.y), sc * (w2 - sacc.z), sc * (w3 - sacc.w));
    }
    *reinterpret_cast<float4 *>(a.dh + r * a.H + h) = o;
}

}  // namespace

hipError_t launch_logprob_bwd_gemm(const LogprobBwdArgs &a, hipStream_t stream) {
    const int64_t blocks = bwd_gemm_blocks(a);
    if (tile_weight_stages(a.n_row_tiles) == 3)
        hipLaunchKernelGGL(logprob_bwd_gemm_kernel<3>, dim3(static_cast<uint32_t>(blocks)), dim3(kGemmThreads), 0,
                           stream, a);
    else
        hipLaunchKernelGGL(logprob_bwd_gemm_kernel<2>, dim3(static_cast<uint32_t>(blocks)), dim3(kGemmThreads), 0,
                           stream, a);
    return hipGetLastError();
}

hipError_t launch_logprob_bwd_finish(const LogprobBwdArgs &a, hipStream_t stream) {
    const int64_t blocks = bwd_finish_blocks(a);
    if (blocks == 0) return hipSuccess;
    static_assert(kBwdFinishThreads == kThreads, "finish launch shape");
    hipLaunchKernelGGL(logprob_bwd_finish_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace rlk
