// Fused lm-head token log-prob for gfx950.
//
// Tile kernel: one workgroup (8 wave64s, two per SIMD) computes the 256 x 256
// logit tile  Z^T = W_tile * hidden_tile^T  (vocab entries on the M side,
// token rows on the N side); each wave owns 128 vocab x 64 rows as 4 x 2
// MFMA 32x32x16 bf16 tiles (fp32 accumulators: 128 registers), so while one
// wave of a SIMD waits on LDS or issues loads the other keeps the matrix
// core busy.  Both operands are hidden-contiguous.  The hidden dimension streams through two
// LDS stages of 64 entries, filled by direct global->LDS loads (no register
// staging): the loads for stage s+2 are issued right after the barrier that
// frees stage s's buffer, interleaved with the MFMAs of stage s's last k-step,
// and the fragments of k-step q+1 are read from LDS while the MFMAs of k-step
// q run.  Rows past the vocabulary or the batch re-read the last valid row:
// their logits are masked (vocab) or never written (rows).
// The epilogue never stores the logits: per token row it takes the max and
// the sum of exp2 over the tile's vocab entries (the vocab index lives in the
// accumulator registers, so the reduction is in-lane plus one cross-half
// shuffle), picks out the target's logit when the target falls in the tile,
// and writes one (max, sum) partial per (vocab tile, row).
// A last round of tiles runs either as hidden-dimension parts summed by a
// reduce kernel (at most half the CUs busy) or as tiles 128 or 192 vocab
// entries wide (at most 4 row tiles; more than half busy in the forward, any
// partial round for the sampling head's logits), each with a partial slot
// of its own.
// Combine kernel: per row, merge the partials of all slots into the
// log-sum-exp and subtract it from the target logit.
#include "device_common.h"
#include "kernels.h"
#include "lds_stage.h"

namespace rlk {
namespace {

constexpr int kThreads = 256;
constexpr int kK = kHiddenStep;                 // 64 hidden entries per LDS stage
constexpr int kTileElems = kVocabTile * kK;     // bf16 elements per operand per stage
static_assert(kVocabTile == kRowTile, "square tiles assumed below");
constexpr int kTileThreads = 64 * kTileWaves;  // 8 waves
constexpr int kBlocksPerWave = kTileElems / 512 / kTileWaves;   // 1 KB hidden load blocks per wave per stage
static_assert(kBlocksPerWave == 4, "staging layout");

// WS: weight-ring depth.  With few row tiles the hidden rows stay in L2 and
// only the weights stream from HBM; a third weight stage gives them two
// stages to arrive (WS = 3 fills the whole 160 KB of LDS).  With many row
// tiles both operands miss and WS = 2 measures better.
// The epilogue modes (kFwd, kBwdProbs, kLogits, kPartialK, kNarrow) and
// the tile each workgroup computes are defined with the index arithmetic.

// Forward epilogue of one 32-row column of a (64 TM) x 256 logit tile, as one
// lane of a wave holds it: z(tm)[i] is vocab vbase + tm*32 + 8*(i/4) + 4*h2 +
// i%4 for token row rr (vbase = v0 + 32 TM * the wave's vocab half).  Returns
// the row's max and sum of exp2 over the wave's 32 TM vocab entries (both lane
// halves merged) and writes the target's logit if it falls among them.
template <int TM, class Z>
__device__ __forceinline__ void row_partial(const LogprobArgs &a, Z z, int64_t rr, int64_t vbase, int h2,
                                            float &mx_out, float &sum_out) {
    constexpr int SPAN = 32 * TM;                // vocab entries per wave
    const float c2 = a.inv_temperature * kLog2e;
    const bool full_vocab = vbase + SPAN <= a.V;  // only the last vocab tile is masked
    // the target's index among the wave's vocab entries, shifted so that
    // it compares against compile-time constants; -1 unless this lane's half
    // of the accumulator rows (bit 2 of the index) holds it
    int tsel = -1;
    if (rr < a.R) {
        const int64_t local = static_cast<int64_t>(a.target[rr]) - vbase;
        if (local >= 0 && local < SPAN && ((local >> 2) & 1) == h2) tsel = static_cast<int>(local) - 4 * h2;
    }
    // one pass per 32-entry block: block max and sum, merged online into the
    // row's (mx, sum); each accumulator register is read once.  Only the last
    // vocab tile masks entries past the vocabulary: the other tiles take a
    // path without per-entry compares (the branch is uniform over the wave).
    float mx = -INFINITY, sum = 0.f;
    auto merge = [&](float bm, float bs) {
        const float nm = fmaxf(mx, bm);
        const float nmu = nm == -INFINITY ? 0.f : nm;
        sum = sum * fast_exp2(mx - nmu) + bs * fast_exp2(bm - nmu);
        mx = nm;
    };
    if (full_vocab) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
            const f32x16 zz = z(tm);
            float bm = fmaxf(fmaxf(zz[0], zz[1]), zz[2]);
#pragma unroll
            for (int i = 3; i < 15; i += 2) bm = fmaxf(fmaxf(bm, zz[i]), zz[i + 1]);
            bm = fmaxf(bm, zz[15]) * c2;         // c2 > 0: scaling commutes with max
            const float bmu = bm == -INFINITY ? 0.f : bm;
            float bs = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) bs += fast_exp2(zz[i] * c2 - bmu);
            merge(bm, bs);
            __builtin_amdgcn_sched_barrier(0);
        }
    } else {
        const int vlim = static_cast<int>(a.V - vbase) - 4 * h2;
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
            const f32x16 zz = z(tm);
            float bm = -INFINITY;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int loc = tm * 32 + 8 * (i >> 2) + (i & 3);
                bm = fmaxf(bm, loc < vlim ? zz[i] : -INFINITY);
            }
            bm *= c2;
            const float bmu = bm == -INFINITY ? 0.f : bm;
            float bs = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int loc = tm * 32 + 8 * (i >> 2) + (i & 3);
                bs += loc < vlim ? fast_exp2(zz[i] * c2 - bmu) : 0.f;
            }
            merge(bm, bs);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // the target's logit: a tile holds a given row's target with probability
    // 256 / V, so the search runs only when some lane of the wave needs it
    if (__any(tsel >= 0)) {
        float zsel = 0.f;
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
            const f32x16 zz = z(tm);
#pragma unroll
            for (int i = 0; i < 16; ++i) zsel = tm * 32 + 8 * (i >> 2) + (i & 3) == tsel ? zz[i] : zsel;
        }
        if (tsel >= 0) a.zt[rr] = zsel * a.inv_temperature;
    }
    // merge the two lane halves (same row, disjoint vocab entries)
    const float om = __shfl_xor(mx, 32, 64), os = __shfl_xor(sum, 32, 64);
    const float nm = fmaxf(mx, om);
    const float nmu = nm == -INFINITY ? 0.f : nm;
    sum_out = sum * fast_exp2(mx - nmu) + os * fast_exp2(om - nmu);
    mx_out = nm;
}

// Writes the (max, sum) partial of (partial slot vt, row rr) from the two vocab
// halves' partials.
__device__ __forceinline__ void write_partial(const LogprobArgs &a, int64_t vt, int64_t rr, float m0, float l0,
                                              float m1, float l1) {
    const float Mx = fmaxf(m0, m1);
    a.pm[vt * a.R + rr] = Mx;
    a.pl[vt * a.R + rr] = l0 * fast_exp2(m0 - Mx) + l1 * fast_exp2(m1 - Mx);
}

// Backward epilogue of one 32-row column of a wave's 128 x 128 block, as one
// lane holds it: z(tm)[i] is vocab v0 + wm*128 + tm*32 + 8*(i/4) + 4*h2 + i%4
// for tile row `row` of row tile rt.  p = exp(inv_T z - lse) (0 for masked
// or invalid targets and past the vocabulary) goes to the blocked
// probability buffer as bf16: the 4 consecutive entries i%4 are one 8-byte
// store into vocab step vt*4 + wm*2 + tm/2, chunk (tm%2)*4 + i/4.
template <class Z>
__device__ __forceinline__ void probs_column(const LogprobArgs &a, Z z, int64_t v0, int64_t vt, int64_t rt, int wm,
                                             int row, int h2) {
    const float c2 = a.inv_temperature * kLog2e;
    const int64_t vbase = v0 + wm * 128;
    const int vlim = vbase + 128 <= a.V ? 128 : static_cast<int>(a.V - vbase) - 4 * h2;
    uint16_t *pb = a.probs + probs_block(rt, a.n_vocab_tiles * 4LL, vt * 4 + wm * 2);
    const int64_t rr = rt * kRowTile + row;
    bool live = false;
    float l2 = 0.f;
    if (rr < a.R) {
        const int32_t t = a.target[rr];
        live = t >= 0 && t < a.V;
        l2 = a.lse_in[rr] * kLog2e;
    }
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) {
        const f32x16 zz = z(tm);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t w2[2];
#pragma unroll
            for (int e = 0; e < 4; e += 2) {
                const int loc = tm * 32 + 8 * q + e;
                const float p0 = live && loc < vlim ? fast_exp2(zz[4 * q + e] * c2 - l2) : 0.f;
                const float p1 = live && loc + 1 < vlim ? fast_exp2(zz[4 * q + e + 1] * c2 - l2) : 0.f;
                w2[e >> 1] = static_cast<uint32_t>(f32_to_bf16_bits(p0)) |
                             (static_cast<uint32_t>(f32_to_bf16_bits(p1)) << 16);
            }
            *reinterpret_cast<uint2 *>(pb + probs_store_off(tm, q, row, h2)) = make_uint2(w2[0], w2[1]);
        }
    }
}

// Forward epilogue of one (64 TM) x 256 logit tile held in the registers of
// the workgroup's 8 waves (acc[tm][tn][i] of wave (wm, wn), lane (h2, l32)
// holds vocab v0 + wm*32*TM + tm*32 + 8*(i/4) + 4*h2 + i%4 for token row
// r0 + wn*64 + tn*32 + l32): per token row the max and the sum of exp2 over
// the tile's vocab entries and, if the target falls in the tile, its logit.
// The partial goes to slot `slot`.  `red` is 4 KB of LDS that the caller no
// longer uses.
template <int TM>
__device__ __forceinline__ void fwd_epilogue(const LogprobArgs &a, const f32x16 (&acc)[TM][2], int64_t v0,
                                             int64_t slot, int64_t rt, float (*red)[kRowTile][2]) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1, wn = wave >> 1;
    const int l32 = lane & 31, h2 = lane >> 5;
    const int64_t r0 = rt * kRowTile;
    const int64_t vbase = v0 + wm * 32 * TM;
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
        const int row = wn * 64 + tn * 32 + l32;
        float mx, sum;
        row_partial<TM>(a, [&](int tm) -> const f32x16 & { return acc[tm][tn]; }, r0 + row, vbase, h2, mx, sum);
        if (h2 == 0) {
            red[wm][row][0] = mx;
            red[wm][row][1] = sum;
        }
        // keep each row block's accumulator copies local
        __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    if (tid < kRowTile) {                        // one thread per row of the tile
        const int64_t rr = r0 + tid;
        if (rr < a.R) write_partial(a, slot, rr, red[0][tid][0], red[0][tid][1], red[1][tid][0], red[1][tid][1]);
    }
}

// TM: 32-entry vocab blocks per wave; a tile spans 64 TM vocab entries (4:
// the 256 x 256 tiles; 2, 3: the narrow tiles of a last round, for the
// forward (kNarrow) and the sampling head's logits (kLogits)).
// TL: debug build with a timeline record per wave (forward modes only): wall
// clock at the start, at the loop's start and end and after the epilogue,
// s_memtime cycles of the loop, and the cycles of the stage-end wait in one
// stage of every 8 (a sample: each stamp makes the wave wait for the scalar
// read that returns it).  The same arithmetic as TL = false.
template <int WS, int MODE, int TM = 4, bool TL = false>
__global__ __launch_bounds__(kTileThreads, 1) void logprob_tile_kernel(LogprobArgs a) {
    static_assert(TM == 4 || MODE == kNarrow || MODE == kLogits, "narrow tiles: forward and logits only");
    static_assert(!TL || MODE == kFwd || MODE == kNarrow || MODE == kPartialK, "timeline: forward tiles only");
    [[maybe_unused]] uint64_t tl_start = 0, tl_loop0 = 0, tl_loop1 = 0, tl_c0 = 0, tl_c1 = 0, tl_wait = 0;
    [[maybe_unused]] uint32_t tl_samples = 0;
    if constexpr (TL) tl_start = __builtin_amdgcn_s_memrealtime();
    constexpr int VW = 64 * TM;                  // vocab entries per tile
    constexpr int WELEMS = VW * kK;              // bf16 elements of one weight stage
    constexpr int WBLK = VW / 64;                // 1 KB weight blocks per wave per stage (= TM)
    constexpr int HBLK = kBlocksPerWave;         // 1 KB hidden blocks per wave per stage
    constexpr int HS = tile_hidden_stages(TM);   // hidden-row stages
    static_assert(HS == 2 || WS == 3, "a third hidden stage goes with the 3-stage weight ring");
    // WS weight stages + HS x 32 KB hidden stages; the epilogue's reduction
    // area reuses the weight ring once the loop is done
    __shared__ __attribute__((aligned(16))) uint16_t wring[WS * WELEMS];
    __shared__ __attribute__((aligned(16))) uint16_t hring[HS * kTileElems];
    float (*red)[kRowTile][2] = reinterpret_cast<float (*)[kRowTile][2]>(wring);   // [vocab half][row][m, l]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1, wn = wave >> 1;     // vocab half (32 TM entries), row quarter (64 rows)
    const int l32 = lane & 31, h2 = lane >> 5;
    const TileCoord tc = tile_coord(MODE, TM, blockIdx.x, a);
    const int64_t vt = uniform64(tc.vt), rt = uniform64(tc.rt), v0 = uniform64(tc.v0);   // vt: the tile's partial slot
    const int kb = tc.kb, nks = tc.nks;                 // hidden steps [kb, kb + nks)
    const int64_t r0 = rt * kRowTile;
    const int64_t H = a.H;

    // ---- staging: each wave fills TM blocks of 8 weight rows and 4 blocks
    // of 8 hidden rows per stage (wave w: blocks w TM .. and 4 w ..).
    // Lane i of a block covers row 8*block + i/8 and LDS slot i%8 of that row,
    // which holds chunk (i%8) ^ swizzle(row), so the LDS image is op_off's.
    // Rows past the vocabulary / the batch re-read the last valid row.
    const uint16_t *wg = a.w + v0 * H;
    const uint16_t *hg = a.hidden + r0 * H;
    const int wlast = stage_last(VW, a.V, v0);
    const int hlast = stage_last(kRowTile, a.R, r0);
    // Block j of stage `slot`'s buffer gets the data of stage min(slot, nks-1):
    // past the last stage the loads refill a buffer nobody reads any more.
    auto wbuf = [&](int ks) { return wring + (ks % WS) * WELEMS; };
    auto hbuf = [&](int ks) { return hring + (ks % HS) * kTileElems; };
    const uint32_t wring_l = lds_addr(wring), hring_l = lds_addr(hring);
    auto issue_block = [&](const uint16_t *g, int last, uint32_t st, int slot, int blk) {
        const int row = stage_row(blk, lane);
        // wave-uniform base (SGPRs) plus a per-lane byte offset that stays
        // the same from stage to stage
        load_lds16_s(g + stage_k0(kb, slot, nks), stage_voff(row, last, H, stage_chunk(row, lane)), st + blk * 1024);
    };
    auto wbuf_l = [&](int ks) { return wring_l + (ks % WS) * (WELEMS * 2); };
    auto hbuf_l = [&](int ks) { return hring_l + (ks % HS) * (kTileElems * 2); };
    auto issue_w = [&](int slot) {
        const uint32_t st = wbuf_l(slot);
#pragma unroll
        for (int j = 0; j < WBLK; ++j) issue_block(wg, wlast, st, slot, wave * WBLK + j);
    };
    auto issue_h = [&](int slot) {
        const uint32_t st = hbuf_l(slot);
#pragma unroll
        for (int j = 0; j < HBLK; ++j) issue_block(hg, hlast, st, slot, wave * HBLK + j);
    };

    f32x16 acc[TM][2];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) acc[tm][tn] = f32x16{};
    bf16x8 fa[2][TM], fb[2][2];
    auto read_frags = [&](int ks, int kq, int p) {
        const uint16_t *as = wbuf(ks);
        const uint16_t *bs = hbuf(ks);
        const int c = kq * 2 + h2;
#pragma unroll
        for (int i = 0; i < TM; ++i)
            fa[p][i] = *reinterpret_cast<const bf16x8 *>(as + op_off(wm * 32 * TM + i * 32 + l32, c));
#pragma unroll
        for (int j = 0; j < 2; ++j) fb[p][j] = *reinterpret_cast<const bf16x8 *>(bs + op_off(wn * 64 + j * 32 + l32, c));
    };
    auto mfma_step = [&](int p) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[p][i], fb[p][j], acc[i][j], 0, 0, 0);
    };

    // Stage ks lives in weight buffer ks % WS and hidden buffer ks % HS.  At
    // the end of stage ks (once every wave is done reading it) the hidden rows
    // of stage ks+HS and then the weights of stage ks+WS are issued, so they
    // have HS-1 and WS-1 stages to arrive; the one wait per stage leaves only
    // the newest stage in flight: the weights (HS = 2, WS = 3), both operands
    // (HS = WS = 3) or nothing (WS = 2).  Loads past the last stage refill a
    // buffer nobody reads any more (so the loop body has no branch); the
    // final wait makes sure none of them is still writing LDS when the
    // epilogue starts.
    issue_h(0);
    issue_w(0);
    issue_h(1);
    issue_w(1);
    if (HS == 3) issue_h(2);
    if (WS == 3) issue_w(2);
    wait_vm<(HS - 1) * HBLK + (WS - 1) * WBLK>();   // stage 0 has landed
    barrier();
    if constexpr (TL) {
        tl_loop0 = __builtin_amdgcn_s_memrealtime();
        tl_c0 = __builtin_amdgcn_s_memtime();
    }
    read_frags(0, 0, 0);
    for (int ks = 0; ks < nks; ++ks) {
#pragma unroll
        for (int kq = 0; kq < kK / 16 - 1; ++kq) {
            read_frags(ks, kq + 1, (kq + 1) & 1);
            mfma_step(kq & 1);
#pragma unroll
            for (int i = 0; i < TM + 2; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read
            }
            if constexpr (TM > 2) __builtin_amdgcn_sched_group_barrier(0x008, 2 * TM - (TM + 2), 0);
        }
        // last k-step: stage ks+1 has landed (only stage ks+2's loads may
        // still be in flight) and every wave is done reading stage ks
        [[maybe_unused]] uint64_t tl_w0 = 0;
        if constexpr (TL)
            if ((ks & 7) == 3) tl_w0 = __builtin_amdgcn_s_memtime();
        wait_vm<(HS - 2) * HBLK + (WS - 2) * WBLK>();
        wait_lds();
        barrier();
        if constexpr (TL)
            if ((ks & 7) == 3) {
                tl_wait += __builtin_amdgcn_s_memtime() - tl_w0;
                ++tl_samples;
            }
        // eight groups of: one global->LDS load (hidden rows of stage ks+HS
        // in groups 0-3, weights of stage ks+WS in groups 4-7), one MFMA of
        // this k-step, one fragment read of stage ks+1 (kept in this order:
        // the loads are opaque to the scheduler)
        {
            const uint16_t *as = wbuf(ks + 1);
            const uint16_t *bs = hbuf(ks + 1);
#pragma unroll
            for (int g = 0; g < 8; ++g) {
                if (g < HBLK) issue_block(hg, hlast, hbuf_l(ks + HS), ks + HS, wave * HBLK + g);
                else if (g - HBLK < WBLK) issue_block(wg, wlast, wbuf_l(ks + WS), ks + WS, wave * WBLK + (g - HBLK));
                if (g < 2 * TM)
                    acc[g >> 1][g & 1] =
                        __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][g >> 1], fb[1][g & 1], acc[g >> 1][g & 1], 0, 0, 0);
                if (g < TM)
                    fa[0][g] = *reinterpret_cast<const bf16x8 *>(as + op_off(wm * 32 * TM + g * 32 + l32, h2));
                else if (g >= 4 && g < 6)
                    fb[0][g - 4] = *reinterpret_cast<const bf16x8 *>(bs + op_off(wn * 64 + (g - 4) * 32 + l32, h2));
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
    wait_vm<0>();
    barrier();                                   // the reduction area aliases the weight ring
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (TL) {
        tl_loop1 = __builtin_amdgcn_s_memrealtime();
        tl_c1 = __builtin_amdgcn_s_memtime();
    }
    // the timeline record of this wave (lane 0 stores it)
    [[maybe_unused]] auto tl_record = [&]() {
        const uint64_t tl_end = __builtin_amdgcn_s_memrealtime();
        const uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);    // HW_ID
        const uint32_t xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20);  // XCC_ID
        if (lane == 0) {
            uint64_t *rec =
                a.timeline + (a.timeline_base + static_cast<int64_t>(blockIdx.x) * kTileWaves + wave) * kTimelineWords;
            const uint64_t kind = MODE == kFwd ? 0 : MODE == kNarrow ? 1 : 2;
            rec[0] = hw | (static_cast<uint64_t>(xcc & 0xff) << 32) | (kind << 40) | (static_cast<uint64_t>(wave) << 48);
            rec[1] = tl_start;
            rec[2] = tl_loop0;
            rec[3] = tl_loop1;
            rec[4] = tl_end;
            rec[5] = tl_wait;
            rec[6] = tl_c1 - tl_c0;
            rec[7] = blockIdx.x | (static_cast<uint64_t>(nks) << 32) | (static_cast<uint64_t>(tl_samples) << 48);
        }
    };

    if constexpr (MODE == kBwdProbs) {
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) {
            probs_column(a, [&](int tm) -> const f32x16 & { return acc[tm][tn]; }, v0, vt, rt, wm,
                         wn * 64 + tn * 32 + l32, h2);
            __builtin_amdgcn_sched_barrier(0);
        }
        return;
    }
    if constexpr (MODE == kLogits) {
        // acc[tm][tn][i]: vocab v0 + wm*32*TM + tm*32 + 8*(i/4) + 4*h2 + i%4,
        // row r0 + wn*64 + tn*32 + l32: 4 consecutive entries per store
        const int64_t vbase = v0 + wm * 32 * TM;
        const int vlim = vbase + 32 * TM <= a.V ? 32 * TM : static_cast<int>(a.V - vbase) - 4 * h2;
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) {
            const int row = wn * 64 + tn * 32 + l32;
            const int64_t rr = r0 + row;
            const bool live = rr < a.R;
            const float it = live ? a.inv_t_rows[rr] : 0.f;
            float *yrow = a.logits + (live ? rr : 0) * a.ld + vbase + 4 * h2;
            float mx = -INFINITY;
#pragma unroll
            for (int tm = 0; tm < TM; ++tm) {
                const f32x16 z = acc[tm][tn];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float y[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        y[e] = z[4 * q + e] * it;
                        y[e] = y[e] == 0.f ? 0.f : y[e];   // one key for +0 and -0
                        if (tm * 32 + 8 * q + e < vlim) mx = fmaxf(mx, y[e]);
                    }
                    if (live)
                        *reinterpret_cast<float4 *>(yrow + tm * 32 + 8 * q) = make_float4(y[0], y[1], y[2], y[3]);
                }
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            if (h2 == 0) red[wm][row][0] = mx;
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();
        if (tid < kRowTile) {
            const int64_t rr = r0 + tid;
            if (rr < a.R) a.pm[vt * a.R + rr] = fmaxf(red[0][tid][0], red[1][tid][0]);
        }
        return;
    }

    if constexpr (MODE == kPartialK) {
        // one part of a tail tile: its fp32 accumulators, in register order
        // (each store writes 1 KB contiguously), for the reduce kernel
#pragma unroll
        for (int tm = 0; tm < 4; ++tm)
#pragma unroll
            for (int tn = 0; tn < 2; ++tn)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const f32x4 v = {acc[tm][tn][4 * q], acc[tm][tn][4 * q + 1], acc[tm][tn][4 * q + 2],
                                     acc[tm][tn][4 * q + 3]};
                    *reinterpret_cast<f32x4 *>(a.part + part_elem(blockIdx.x, wm, wn * 2 + tn, tm, q, lane)) = v;
                }
        if constexpr (TL) tl_record();
        return;
    }
    fwd_epilogue<TM>(a, acc, v0, vt, rt, red);
    if constexpr (TL) tl_record();
}

// Sum, in part order, of the hidden-dimension parts of tail tile j (its
// logical tile a.tile_base + j): what lane `lane` held in the accumulators
// (tm = 0..3) of vocab half wm and 32-row block rb.
__device__ __forceinline__ void sum_parts(const LogprobArgs &a, int64_t j, int wm, int rb, int lane, f32x16 (&z)[4]) {
#pragma unroll
    for (int tm = 0; tm < 4; ++tm) z[tm] = f32x16{};
    for (int sp = 0; sp < a.splits; ++sp) {
        f32x4 v[4][4];
#pragma unroll
        for (int tm = 0; tm < 4; ++tm)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                v[tm][q] = *reinterpret_cast<const f32x4 *>(a.part + part_elem(j * a.splits + sp, wm, rb, tm, q, lane));
#pragma unroll
        for (int tm = 0; tm < 4; ++tm)
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int e = 0; e < 4; ++e) z[tm][4 * q + e] += v[tm][q][e];
    }
}

// The reduce kernels of a hidden-split tail: one workgroup of 2 waves per
// (tail tile, 32-row block rb), 8 workgroups per tile, so the parts are read
// by many CUs at once.  Wave wm holds what lane (h2, l32) of the tile
// kernel's wave of vocab half wm held for that block.
//
// Forward: the forward epilogue on the sums.
__global__ __launch_bounds__(128) void logprob_tail_reduce_kernel(LogprobArgs a) {
    __shared__ float red[2][32][2];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wm = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t j = blockIdx.x >> 3;
    const int rb = blockIdx.x & 7;
    const int l32 = lane & 31, h2 = lane >> 5;
    int64_t vt, rt;
    tile_of_logical(a.tile_base + j, a.n_vocab_tiles, a.n_row_tiles, &vt, &rt);
    f32x16 z[4];
    sum_parts(a, j, wm, rb, lane, z);
    const int64_t rr = rt * kRowTile + rb * 32 + l32;
    float mx, sum;
    row_partial<4>(a, [&](int tm) -> const f32x16 & { return z[tm]; }, rr, vt * kVocabTile + wm * 128, h2, mx, sum);
    if (h2 == 0) {
        red[wm][l32][0] = mx;
        red[wm][l32][1] = sum;
    }
    __syncthreads();
    if (tid < 32) {
        const int64_t r = rt * kRowTile + rb * 32 + tid;
        if (r < a.R) write_partial(a, vt, r, red[0][tid][0], red[0][tid][1], red[1][tid][0], red[1][tid][1]);
    }
}

// Backward: the probabilities of the sums.
__global__ __launch_bounds__(128) void logprob_probs_tail_reduce_kernel(LogprobArgs a) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wm = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t j = blockIdx.x >> 3;
    const int rb = blockIdx.x & 7;
    const int l32 = lane & 31, h2 = lane >> 5;
    int64_t vt, rt;
    tile_of_logical(a.tile_base + j, a.n_vocab_tiles, a.n_row_tiles, &vt, &rt);
    f32x16 z[4];
    sum_parts(a, j, wm, rb, lane, z);
    probs_column(a, [&](int tm) -> const f32x16 & { return z[tm]; }, vt * kVocabTile, vt, rt, wm, rb * 32 + l32, h2);
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

// Very few rows (a decode step): one workgroup per row, each thread merging
// at most a few of the row's partial slots, so all of the row's loads are in
// flight at once; the (max, sum) pairs then merge across the waves in LDS.
__global__ __launch_bounds__(kThreads) void logprob_combine_block_kernel(LogprobArgs a) {
    __shared__ float ml[kThreads / 64][2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t r = blockIdx.x;
    float M = -INFINITY, L = 0.f;
    for (int64_t vt = tid; vt < a.n_partials; vt += kThreads) lse_merge(M, L, a.pm[vt * a.R + r], a.pl[vt * a.R + r]);
    const float Mw = wave_max(M);
    const float Lw = wave_sum(M == -INFINITY ? 0.f : L * fast_exp2(M - Mw));
    if (lane == 0) {
        ml[wave][0] = Mw;
        ml[wave][1] = Lw;
    }
    __syncthreads();
    if (tid == 0) {
        float Mb = -INFINITY, Lb = 0.f;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w)
            if (ml[w][0] != -INFINITY) lse_merge(Mb, Lb, ml[w][0], ml[w][1]);
        finish_row(a, r, Mb, Lb);
    }
}

// Few rows: one wave per row, lanes stride over the vocab tiles.
__global__ __launch_bounds__(kThreads) void logprob_combine_wave_kernel(LogprobArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t r = static_cast<int64_t>(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
    if (r >= a.R) return;
    float M = -INFINITY, L = 0.f;
    for (int64_t vt = lane; vt < a.n_partials; vt += 64) lse_merge(M, L, a.pm[vt * a.R + r], a.pl[vt * a.R + r]);
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
    for (; vt + 4 <= a.n_partials; vt += 4) {
        float m[4], l[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            m[j] = a.pm[(vt + j) * a.R + r];
            l[j] = a.pl[(vt + j) * a.R + r];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) lse_merge(M, L, m[j], l[j]);
    }
    for (; vt < a.n_partials; ++vt) lse_merge(M, L, a.pm[vt * a.R + r], a.pl[vt * a.R + r]);
    finish_row(a, r, M, L);
}

}  // namespace

hipError_t launch_logprob(const LogprobArgs &a, hipStream_t stream, bool timeline) {
    // whole tiles [0, dp_tiles)
    LogprobArgs d = a;
    d.tile_base = 0;
    d.tile_count = a.dp_tiles;
    d.timeline_base = 0;
    const uint32_t whole = static_cast<uint32_t>(d.tile_count);
    if (tile_weight_stages(a.n_row_tiles) == 3) {
        if (timeline)
            hipLaunchKernelGGL((logprob_tile_kernel<3, kFwd, 4, true>), dim3(whole), dim3(kTileThreads), 0, stream, d);
        else
            hipLaunchKernelGGL((logprob_tile_kernel<3, kFwd>), dim3(whole), dim3(kTileThreads), 0, stream, d);
    } else {
        if (timeline)
            hipLaunchKernelGGL((logprob_tile_kernel<2, kFwd, 4, true>), dim3(whole), dim3(kTileThreads), 0, stream, d);
        else
            hipLaunchKernelGGL((logprob_tile_kernel<2, kFwd>), dim3(whole), dim3(kTileThreads), 0, stream, d);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.narrow_tiles > 0) {
        // the last round as narrow tiles, 128 or 192 vocab entries wide (the
        // plan allows them only for at most 4 row tiles, so the 3-stage
        // weight ring applies)
        static_assert(kNarrowMinTM == 2 && kNarrowMaxTM == 3, "narrow tile widths");
        const uint32_t blocks = static_cast<uint32_t>(a.narrow_tiles * a.n_row_tiles);
        LogprobArgs n = a;
        n.timeline_base = a.dp_tiles * kTileWaves;
        if (a.narrow_tm == 2) {
            if (timeline)
                hipLaunchKernelGGL((logprob_tile_kernel<3, kNarrow, 2, true>), dim3(blocks), dim3(kTileThreads), 0,
                                   stream, n);
            else
                hipLaunchKernelGGL((logprob_tile_kernel<3, kNarrow, 2>), dim3(blocks), dim3(kTileThreads), 0, stream,
                                   n);
        } else {
            if (timeline)
                hipLaunchKernelGGL((logprob_tile_kernel<3, kNarrow, 3, true>), dim3(blocks), dim3(kTileThreads), 0,
                                   stream, n);
            else
                hipLaunchKernelGGL((logprob_tile_kernel<3, kNarrow, 3>), dim3(blocks), dim3(kTileThreads), 0, stream,
                                   n);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (a.tail_tiles > 0) {
        // the tail: `splits` hidden-dimension parts per tile, then their sum
        LogprobArgs t = a;
        t.tile_base = a.dp_tiles;
        t.tile_count = a.tail_tiles;
        t.timeline_base = (a.dp_tiles + a.narrow_tiles * a.n_row_tiles) * kTileWaves;
        const uint32_t parts = static_cast<uint32_t>(a.tail_tiles * a.splits);
        if (tile_weight_stages(a.n_row_tiles) == 3) {
            if (timeline)
                hipLaunchKernelGGL((logprob_tile_kernel<3, kPartialK, 4, true>), dim3(parts), dim3(kTileThreads), 0,
                                   stream, t);
            else
                hipLaunchKernelGGL((logprob_tile_kernel<3, kPartialK>), dim3(parts), dim3(kTileThreads), 0, stream, t);
        } else {
            if (timeline)
                hipLaunchKernelGGL((logprob_tile_kernel<2, kPartialK, 4, true>), dim3(parts), dim3(kTileThreads), 0,
                                   stream, t);
            else
                hipLaunchKernelGGL((logprob_tile_kernel<2, kPartialK>), dim3(parts), dim3(kTileThreads), 0, stream, t);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(logprob_tail_reduce_kernel, dim3(static_cast<uint32_t>(a.tail_tiles * 8)), dim3(128), 0,
                           stream, t);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int combine = logprob_combine_kind(a.R);
    if (combine == kCombineBlock) {
        hipLaunchKernelGGL(logprob_combine_block_kernel, dim3(static_cast<uint32_t>(a.R)), dim3(kThreads), 0, stream,
                           a);
    } else if (combine == kCombineWave) {
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

hipError_t launch_logprob_probs(const LogprobArgs &a, hipStream_t stream) {
    // whole tiles [0, dp_tiles), then the tail's hidden-dimension parts and
    // their sums, which give the tail tiles' probabilities
    LogprobArgs d = a;
    d.tile_base = 0;
    d.tile_count = a.dp_tiles;
    const bool ws3 = tile_weight_stages(a.n_row_tiles) == 3;
    if (ws3)
        hipLaunchKernelGGL((logprob_tile_kernel<3, kBwdProbs>), dim3(static_cast<uint32_t>(d.tile_count)),
                           dim3(kTileThreads), 0, stream, d);
    else
        hipLaunchKernelGGL((logprob_tile_kernel<2, kBwdProbs>), dim3(static_cast<uint32_t>(d.tile_count)),
                           dim3(kTileThreads), 0, stream, d);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.tail_tiles == 0) return e;
    LogprobArgs t = a;
    t.tile_base = a.dp_tiles;
    t.tile_count = a.tail_tiles;
    const uint32_t parts = static_cast<uint32_t>(a.tail_tiles * a.splits);
    if (ws3)
        hipLaunchKernelGGL((logprob_tile_kernel<3, kPartialK>), dim3(parts), dim3(kTileThreads), 0, stream, t);
    else
        hipLaunchKernelGGL((logprob_tile_kernel<2, kPartialK>), dim3(parts), dim3(kTileThreads), 0, stream, t);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(logprob_probs_tail_reduce_kernel, dim3(static_cast<uint32_t>(a.tail_tiles * 8)), dim3(128), 0,
                       stream, t);
    return hipGetLastError();
}

hipError_t launch_logits(const LogprobArgs &a, hipStream_t stream) {
    // whole tiles [0, dp_tiles), then the last round's narrow tiles if any
    LogprobArgs d = a;
    d.tile_base = 0;
    d.tile_count = a.dp_tiles;
    if (d.tile_count > 0) {
        if (tile_weight_stages(a.n_row_tiles) == 3)
            hipLaunchKernelGGL((logprob_tile_kernel<3, kLogits>), dim3(static_cast<uint32_t>(d.tile_count)),
                               dim3(kTileThreads), 0, stream, d);
        else
            hipLaunchKernelGGL((logprob_tile_kernel<2, kLogits>), dim3(static_cast<uint32_t>(d.tile_count)),
                               dim3(kTileThreads), 0, stream, d);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (a.narrow_tiles > 0) {
        static_assert(kNarrowMinTM == 2 && kNarrowMaxTM == 3, "narrow tile widths");
        const uint32_t blocks = static_cast<uint32_t>(a.narrow_tiles * a.n_row_tiles);
        if (a.narrow_tm == 2)
            hipLaunchKernelGGL((logprob_tile_kernel<3, kLogits, 2>), dim3(blocks), dim3(kTileThreads), 0, stream, a);
        else
            hipLaunchKernelGGL((logprob_tile_kernel<3, kLogits, 3>), dim3(blocks), dim3(kTileThreads), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace rlk
