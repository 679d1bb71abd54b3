// Prefix-shared split-K decode attention for gfx950.
//
// One workgroup (4 wave64s) runs one work item: a chunk of KV tokens of one
// unit at one kv head, serving up to 64 query rows:
//   prefix item: the prompt's KV, for the G*r query rows of its candidates
//                (r = Hq/Hkv; wider groups take one item per 64 rows), so the
//                chunk crosses HBM once per group of up to 64 rows;
//   suffix item: one candidate's own KV, for its r query rows.
// The KV chunk streams through LDS in tiles of 64 tokens: coalesced 16-byte
// buffer loads (rows past the chunk read as zeros through the descriptor's
// range) into registers one tile ahead and a single LDS stage, so three
// workgroups fit on a CU, each with a tile's loads in flight.  Per 16-token
// sub-tile a wave computes scores S^T = K Q^T on MFMA 16x16x32 (tokens on the
// M side, query rows on the N side), keeps an online softmax per query row in
// fp32, rounds the probabilities to bf16 and accumulates O^T = V^T P^T on
// MFMA 16x16x16, whose B operand is exactly the score tile's C layout.
// Each item leaves, per query row, a partial (max m, sum l, weighted value
// sum acc[D]) in log2 units; the combine kernel merges the partials of each
// (sequence, head) by log-sum-exp and writes the bf16 output and fp32 lse.
#include <algorithm>

#include "decode_index.h"
#include "device_common.h"
#include "kernels.h"

namespace rlk {
namespace {

constexpr int kThreads = 256;
// Three workgroups per CU (LDS: one ~36 KB stage each; registers: at most 168
// per lane), each with one tile's loads in flight; with two tiles in flight
// (two register sets) two workgroups fit.
constexpr int kSplitBlocksPerCU = 3;
constexpr int kSplitBlocksPerCUDeep = 2;
constexpr int kSub = 16;                          // tokens per MFMA sub-tile
constexpr int kSubPerTile = kTileTokens / kSub;   // 4

template <int D>
struct DCfg {
    static constexpr int CH = D / 8;             // 16-byte chunks per token row
    static constexpr int KK = D / 32;            // k-steps of S^T = K Q^T
    static constexpr int DT = D / 16;            // 16-wide d tiles of O^T
    static constexpr int LDR = D + 8;            // K row pitch in bf16 (16-byte pad)
    static constexpr int LDRV = D + 16;          // V row pitch in bf16 (32-byte pad)
    static constexpr int TILE = kTileTokens * LDR;   // bf16 elements of one K tile
    static constexpr int TILEV = kTileTokens * LDRV; // bf16 elements of one V tile
    static constexpr int STAGE = TILE + TILEV;       // one K tile followed by one V tile
    static constexpr int LD = kTileTokens * CH / kThreads;  // 16-byte chunks per thread per tensor
    static constexpr int RED_STRIDE = D + 4;     // fp32 row stride of the merge area (16-byte rows, bank spread)
    static constexpr int KV_BYTES = STAGE * 2;                         // one LDS stage (K, V)
    static constexpr int RED_BYTES = 4 * 16 * RED_STRIDE * 4;          // waves x 16 rows
    static constexpr int MAIN_BYTES = KV_BYTES > RED_BYTES ? KV_BYTES : RED_BYTES;
    static constexpr int ML_BYTES = 4 * 16 * 2 * 4;
};

// Element offset of 16-byte chunk c of token t inside a K tile.  Rows are
// padded by 16 bytes, so the 16 lanes that read one chunk of 16 consecutive
// tokens (K operand) hit 16 disjoint groups of 4 banks, and every read of a
// lane sits at a constant offset from one base address.
template <int D>
__device__ __forceinline__ int kv_off(int t, int c) {
    return t * DCfg<D>::LDR + (c << 3);
}

// Element offset of 16-byte chunk c of token t inside a V tile.  V rows are
// padded by 32 bytes: the transposing reads of the V^T operand fetch 8 bytes
// at 4 d-offsets of 8 consecutive tokens per half-wave, and a pitch of 8 banks
// (mod 64) puts those 8 rows on disjoint banks.
template <int D>
__device__ __forceinline__ int v_off(int t, int c) {
    return t * DCfg<D>::LDRV + (c << 3);
}

// Items serve at most 64 query rows: 4 MFMA column tiles of 16, one per wave.
// Items of up to 16 rows split each tile's 4 sub-tiles over the 4 waves, items
// of up to 32 rows over 2; those waves' partials are merged through LDS.
// PF: tiles whose loads are in flight while a tile is computed (1 or 2).
// TL: debug build that leaves one timeline record per work item (wall clock
// at the start, once the first tile is in LDS, at the loop's end and after
// the partials; s_memtime cycles of the loop); the same arithmetic.
template <int D, int PF, bool TL = false>
__global__ __launch_bounds__(kThreads, PF == 2 ? kSplitBlocksPerCUDeep : kSplitBlocksPerCU) void decode_split_kernel(
    DecodeArgs a) {
    using C = DCfg<D>;
    [[maybe_unused]] uint64_t tl_start = 0, tl_first = 0, tl_loop1 = 0, tl_c0 = 0, tl_c1 = 0;
    if constexpr (TL) tl_start = __builtin_amdgcn_s_memrealtime();
    __shared__ __attribute__((aligned(16))) unsigned char smem[C::MAIN_BYTES + C::ML_BYTES];
    uint16_t *kv = reinterpret_cast<uint16_t *>(smem);
    float *red_acc = reinterpret_cast<float *>(smem);
    float *red_ml = reinterpret_cast<float *>(smem + C::MAIN_BYTES);

    const DevItem it = a.items[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g4 = lane >> 4, l16 = lane & 15;
    const int kh = dec_kh(it.meta);
    const bool is_suffix = dec_is_suffix(it.meta);
    const int row_begin = dec_row_begin(it.meta);
    const int M = dec_unit_rows(a, is_suffix);
    const int rows = dec_item_rows(M, row_begin);
    const int n_ct = (rows + 15) >> 4;
    const int Wc = n_ct == 1 ? 1 : (n_ct == 2 ? 2 : 4);
    const int Wt = 4 / Wc;
    const int nst = kSubPerTile / Wt;            // sub-tiles per wave per tile
    const int wc = wave % Wc, wt = wave / Wc;
    const bool mine = wc < n_ct;                 // this wave has a column tile
    const int ntok = dec_ntok(it.meta);
    const int64_t tok_stride = dec_tok_stride(a, D);
    const int64_t base = dec_kv_base(a, it, DecItem{kh, is_suffix}, D);
    const uint16_t *kg = (is_suffix ? a.k_suffix : a.k_prefix) + base;
    const uint16_t *vg = (is_suffix ? a.v_suffix : a.v_prefix) + base;

    // ---- query rows of this wave as MFMA B operands (Q^T, k = d) ----------
    bf16x8 qb[C::KK];
    {
        const int i = wc * 16 + l16;                 // row within the item
        const bool ok = mine && i < rows;
        int64_t qoff = 0;
        if (ok) {
            const int ig = row_begin + i;            // row within the unit
            qoff = dec_q_off(a, it, DecItem{kh, is_suffix}, ig, D);
        }
#pragma unroll
        for (int kk = 0; kk < C::KK; ++kk) {
            if (ok) qb[kk] = *reinterpret_cast<const bf16x8 *>(a.q + qoff + kk * 32 + g4 * 8);
            else    qb[kk] = bf16x8{};
        }
    }

    // ---- online softmax state --------------------------------------------
    float m_run = -INFINITY, l_run = 0.f;        // l_run: this lane's share of the row sum
    f32x4 acc[C::DT];
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // ---- tile staging -----------------------------------------------------
    u32x4 kA[C::LD], vA[C::LD], kB[C::LD], vB[C::LD];
    // Buffer loads: a descriptor per tile covers the chunk's rows from the
    // tile's first token to the end of the chunk's last row, so rows past the
    // chunk fall outside it and read as zeros; each lane's byte offset inside
    // a tile is fixed (tokens x row pitch < 2^23 bytes, ranges < 2^31).
    uint32_t voff[C::LD];
#pragma unroll
    for (int j = 0; j < C::LD; ++j) {
        voff[j] = dec_load_off(tid + j * kThreads, C::CH, tok_stride);
    }
    auto load_tile = [&](int tile, u32x4 (&kr)[C::LD], u32x4 (&vr)[C::LD]) {
        // a tile past the chunk gets an empty range: its loads touch no memory
        // and return zeros, so every step issues the same loads
        const int t0 = tile * kTileTokens;
        const int64_t first = dec_tile_first(t0, ntok, tok_stride);
        const int range = dec_tile_range(t0, ntok, tok_stride, D);
        const __amdgpu_buffer_rsrc_t rk =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(kg + first), 0, range, 0x00020000);
        const __amdgpu_buffer_rsrc_t rv =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(vg + first), 0, range, 0x00020000);
#pragma unroll
        for (int j = 0; j < C::LD; ++j) {
            kr[j] = __builtin_amdgcn_raw_buffer_load_b128(rk, voff[j], 0, 0);
            vr[j] = __builtin_amdgcn_raw_buffer_load_b128(rv, voff[j], 0, 0);
        }
    };
    auto store_tile = [&](const u32x4 (&kr)[C::LD], const u32x4 (&vr)[C::LD]) {
        uint16_t *kl = kv;
        uint16_t *vl = kl + C::TILE;
#pragma unroll
        for (int j = 0; j < C::LD; ++j) {
            const int idx = tid + j * kThreads;
            const int t = idx / C::CH, ch = idx % C::CH;
            *reinterpret_cast<u32x4 *>(kl + kv_off<D>(t, ch)) = kr[j];
            *reinterpret_cast<u32x4 *>(vl + v_off<D>(t, ch)) = vr[j];
        }
    };

    const int ntiles = (ntok + kTileTokens - 1) / kTileTokens;

    const uint16_t *kl = kv;
    const uint16_t *vl = kl + C::TILE;
    auto step = [&](int tile, u32x4 (&kc)[C::LD], u32x4 (&vc)[C::LD]) {
        const int t0 = tile * kTileTokens;
        if (mine) {
            // scores of my sub-tiles, log2 units, masked past the chunk end
            float sc[kSubPerTile][4];
#pragma unroll
            for (int k = 0; k < kSubPerTile; ++k) {
                if (k < nst) {
                    const int st = wt + k * Wt;
                    f32x4 sv = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int kk = 0; kk < C::KK; ++kk) {
                        const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(
                            kl + kv_off<D>(st * kSub + l16, kk * 4 + g4));
                        sv = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qb[kk], sv, 0, 0, 0);
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const bool valid = t0 + st * kSub + g4 * 4 + i < ntok;
                        sc[k][i] = valid ? sv[i] * a.score_scale_log2 : -INFINITY;
                    }
                }
            }
            // online softmax update, probabilities to bf16
            bf16x4 pb[kSubPerTile];
            float mx = -INFINITY;
#pragma unroll
            for (int k = 0; k < kSubPerTile; ++k)
                if (k < nst)
#pragma unroll
                    for (int i = 0; i < 4; ++i) mx = fmaxf(mx, sc[k][i]);
            mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const float m_new = fmaxf(m_run, mx);
            const float m_use = m_new == -INFINITY ? 0.f : m_new;
            const float alpha = fast_exp2(m_run - m_use);
            m_run = m_new;
            // only the wave's own sub-tiles (one of four in a 4-row suffix item)
            float psum = 0.f;
#pragma unroll
            for (int k = 0; k < kSubPerTile; ++k) {
                if (k >= nst) continue;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float p = fast_exp2(sc[k][i] - m_use);
                    psum += p;
                    pb[k][i] = static_cast<__bf16>(p);
                }
            }
            l_run = l_run * alpha + psum;
            // the running max rarely moves after the first tiles: skip the
            // rescale when it stayed put for every row of the wave
            if (__any(alpha != 1.f)) {
#pragma unroll
                for (int dt = 0; dt < C::DT; ++dt) acc[dt] *= alpha;
            }
            // O^T += V^T P^T; lane (g4, l16) needs the 4 tokens st*16 + 4*g4 + 0..3
            // at d = dt*16 + l16, which one transposing read delivers when source
            // lane s of the 16-lane group points at token +s/4, d-offset 4*(s%4).
#pragma unroll
            for (int k = 0; k < kSubPerTile; ++k) {
                if (k < nst) {
                    const int st = wt + k * Wt;
                    const uint16_t *vsrc = vl + (st * kSub + g4 * 4 + (l16 >> 2)) * C::LDRV + 4 * (l16 & 3);
                    bf16x4 vt[C::DT];
#pragma unroll
                    for (int dt = 0; dt < C::DT; ++dt) vt[dt] = lds_read_tr16(vsrc + dt * 16);
#pragma unroll
                    for (int dt = 0; dt < C::DT; ++dt)
                        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt[dt], pb[k], acc[dt], 0, 0, 0);
                }
            }
        }
        // one LDS stage: once every wave has read it, the next tile moves in
        // from its register set, which then takes the loads PF + 1 tiles ahead
        __syncthreads();
        if constexpr (PF == 1) {
            if (tile + 1 < ntiles) {
                store_tile(kc, vc);
                if (tile + 2 < ntiles) load_tile(tile + 2, kc, vc);
                __syncthreads();
            }
        } else {
            // unconditional: every step issues the same loads (past the chunk
            // they are empty), so the wait before the store covers only the
            // older register set
            store_tile(kc, vc);
            load_tile(tile + 3, kc, vc);
            __syncthreads();
        }
    };
    auto tl_loop_start = [&]() {
        if constexpr (TL) {
            tl_first = __builtin_amdgcn_s_memrealtime();
            tl_c0 = __builtin_amdgcn_s_memtime();
        }
    };
    if constexpr (PF == 1) {
        load_tile(0, kA, vA);
        store_tile(kA, vA);
        if (ntiles > 1) load_tile(1, kA, vA);
        __syncthreads();
        tl_loop_start();
        for (int tile = 0; tile < ntiles; ++tile) step(tile, kA, vA);
    } else {
        // set A holds the odd tiles' loads, set B the even ones'
        load_tile(0, kB, vB);
        load_tile(1, kA, vA);
        store_tile(kB, vB);
        load_tile(2, kB, vB);
        __syncthreads();
        tl_loop_start();
        for (int tile = 0; tile < ntiles; tile += 2) {
            step(tile, kA, vA);
            if (tile + 1 < ntiles) step(tile + 1, kB, vB);
        }
    }
    if constexpr (TL) {
        tl_loop1 = __builtin_amdgcn_s_memrealtime();
        tl_c1 = __builtin_amdgcn_s_memtime();
    }
    // the item's timeline record (thread 0 stores it once every wave is done)
    [[maybe_unused]] auto tl_record = [&]() {
        __syncthreads();
        const uint64_t tl_end = __builtin_amdgcn_s_memrealtime();
        const uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);    // HW_ID
        const uint32_t xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20);  // XCC_ID
        if (tid == 0) {
            uint64_t *rec = a.timeline + static_cast<int64_t>(blockIdx.x) * kTimelineWords;
            rec[0] = hw | (static_cast<uint64_t>(xcc & 0xff) << 32) | (static_cast<uint64_t>(is_suffix) << 40) |
                     (static_cast<uint64_t>(rows) << 48);
            rec[1] = tl_start;
            rec[2] = tl_first;
            rec[3] = tl_loop1;
            rec[4] = tl_end;
            rec[5] = static_cast<uint64_t>(ntok) | (static_cast<uint64_t>(ntiles) << 32);
            rec[6] = blockIdx.x;
            rec[7] = tl_c1 - tl_c0;
        }
    };

    // ---- the item's partials ------------------------------------------------
    l_run += __shfl_xor(l_run, 16, 64);
    l_run += __shfl_xor(l_run, 32, 64);
    if (Wt == 1) {
        // every row belongs to one wave: write its partial from the registers
        const int i = wc * 16 + l16;
        if (mine && i < rows) {
            const int64_t prow = static_cast<int64_t>(it.partial_row0) + i;
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt)
                *reinterpret_cast<f32x4 *>(a.pacc + prow * D + dt * 16 + g4 * 4) = acc[dt];
            if (g4 == 0) {
                a.pm[prow] = m_run;
                a.pl[prow] = l_run;
            }
        }
        if constexpr (TL) tl_record();
        return;
    }
    // Wt waves hold partials of the same rows over disjoint tokens: merge them
    // through LDS (the stage is free after the loop's last barrier); only the
    // item's rows are written (a suffix item has r of a column tile's 16)
    if (wc * 16 + l16 < rows) {
        const int slot = wave * 16 + l16;
        if (g4 == 0) {
            red_ml[slot * 2 + 0] = m_run;
            red_ml[slot * 2 + 1] = l_run;
        }
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
            *reinterpret_cast<f32x4 *>(red_acc + slot * C::RED_STRIDE + dt * 16 + g4 * 4) = acc[dt];
    }
    __syncthreads();
    for (int e = tid; e < rows * D; e += kThreads) {
        const int i = e / D, d = e % D;
        const int ct = i >> 4, q = i & 15;
        float Mx = -INFINITY;
        for (int w = 0; w < Wt; ++w) Mx = fmaxf(Mx, red_ml[((ct + w * Wc) * 16 + q) * 2]);
        float L = 0.f, A = 0.f;
        for (int w = 0; w < Wt; ++w) {
            const int slot = (ct + w * Wc) * 16 + q;
            const float f = fast_exp2(red_ml[slot * 2] - Mx);
            L += f * red_ml[slot * 2 + 1];
            A += f * red_acc[slot * C::RED_STRIDE + d];
        }
        const int64_t prow = static_cast<int64_t>(it.partial_row0) + i;
        a.pacc[prow * D + d] = A;
        if (d == 0) {
            a.pm[prow] = Mx;
            a.pl[prow] = L;
        }
    }
    if constexpr (TL) tl_record();
}

// Merges, per (sequence s, query head h) row, the partials of the prompt's
// prefix chunks and the candidate's suffix chunks.  RPW rows per wave, 64 /
// RPW lanes per row (row x of a wave in lanes x 64/RPW ..); the cross-lane
// reductions stay inside a row's lanes.  Two rows per wave put an 8B- or
// 32B-class step's 16384 rows in one round of resident waves; with few rows
// one row per wave keeps more waves, and loads, in flight.
// NB: value rows loaded per batch.  NB = 4 at D = 128 keeps the two-row
// kernel within 64 VGPRs, so 8 waves fit on a SIMD.
template <int D, int RPW, int NB>
__global__ __launch_bounds__(kThreads, NB == 4 ? 8 : 1) void decode_combine_kernel(DecodeArgs a) {
    release_staging(a.release);
    constexpr int LPR = 64 / RPW;                // lanes per row
    constexpr int PER_LANE = D / LPR;
    typedef float fvec __attribute__((ext_vector_type(PER_LANE)));
    const int lane = threadIdx.x & 63;
    const int slot = lane / LPR, hl = lane % LPR;
    const int64_t rows = static_cast<int64_t>(a.P) * a.G * a.Hq;
    const int64_t idx = (static_cast<int64_t>(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6)) * RPW + slot;
    const bool live = idx < rows;                // the last wave's second row may be past the end
    const int64_t ix = live ? idx : 0;
    const int64_t s = ix / a.Hq;
    const int h = static_cast<int>(ix % a.Hq);
    const int64_t p = s / a.G;
    const int g = static_cast<int>(s % a.G);
    const int kh = h / a.r, hr = h % a.r;
    const DevUnit pu = a.prefix_units[p];
    const DevUnit su = a.suffix_units[s];
    const int64_t Mp = static_cast<int64_t>(a.G) * a.r;
    const int pn = static_cast<int>(pu.nchunks);
    const int n = live ? pn + static_cast<int>(su.nchunks) : 0;
    // this kv head's partial rows of the prompt's prefix and the candidate's suffix
    const int64_t pbase = dec_prefix_partial_base(pu, kh, Mp, g, a.r, hr);
    const int64_t sbase = dec_suffix_partial_base(su, kh, a.r, hr);
    auto prow = [&](int j) -> int64_t { return dec_partial_row(pbase, sbase, Mp, pn, a.r, j); };
    auto row_max = [](float v) {
#pragma unroll
        for (int o = LPR / 2; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
        return v;
    };
    auto row_sum = [](float v) {
#pragma unroll
        for (int o = LPR / 2; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
        return v;
    };
    // the largest partial count of the wave's rows, the same in every lane
    const int nw = __builtin_amdgcn_readfirstlane(RPW == 2 ? max(n, __shfl_xor(n, 32, 64)) : n);
    float Mx = -INFINITY, L = 0.f;
    fvec o = {};
    if (nw <= LPR) {
        // lane j of a row holds partial j's (m, l): one load latency for all of
        // them; the value rows load NB at a time (the first NB alongside the
        // (m, l), as they do not depend on the weights), each weight taken by
        // readlane from the row's own lanes
        float mj = -INFINITY, lj = 0.f;
        if (hl < n) {
            const int64_t pr = prow(hl);
            mj = a.pm[pr];
            lj = a.pl[pr];
        }
        fvec v[NB];
        auto load_rows = [&](int j0) {
#pragma unroll
            for (int u = 0; u < NB; ++u)
                if (j0 + u < n) v[u] = *reinterpret_cast<const fvec *>(a.pacc + prow(j0 + u) * D + hl * PER_LANE);
        };
        load_rows(0);
        Mx = row_max(mj);
        const float fj = hl < n ? fast_exp2(mj - Mx) : 0.f;
        L = row_sum(fj * lj);
        for (int j0 = 0; j0 < nw; j0 += NB) {
            if (j0 > 0) load_rows(j0);
#pragma unroll
            for (int u = 0; u < NB; ++u) {
                if (j0 + u < nw) {               // uniform: the lanes read below are < 64
                    const float f0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(fj), j0 + u));
                    float f = f0;
                    if constexpr (RPW == 2) {
                        const float f1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(fj), 32 + j0 + u));
                        f = slot ? f1 : f0;
                    }
                    if (j0 + u < n) o += f * v[u];
                }
            }
        }
    } else {
        for (int j = hl; j < n; j += LPR) Mx = fmaxf(Mx, a.pm[prow(j)]);
        Mx = row_max(Mx);
        for (int j = 0; j < n; ++j) {
            const int64_t pr = prow(j);
            const float f = fast_exp2(a.pm[pr] - Mx);
            L += f * a.pl[pr];
            o += f * *reinterpret_cast<const fvec *>(a.pacc + pr * D + hl * PER_LANE);
        }
    }
    if (!live) return;
    uint16_t *out = a.out + idx * D + hl * PER_LANE;
    if (n == 0) {
#pragma unroll
        for (int e = 0; e < PER_LANE; ++e) out[e] = 0;
        if (a.lse && hl == 0) a.lse[idx] = -INFINITY;
        return;
    }
    const float inv = 1.f / L;
#pragma unroll
    for (int e = 0; e < PER_LANE; ++e) out[e] = f32_to_bf16_bits(o[e] * inv);
    if (a.lse && hl == 0) a.lse[idx] = (Mx + fast_log2(L)) * kLn2;
}

__global__ __launch_bounds__(kThreads) void plan_fetch_kernel(const u32x4 *__restrict__ src,
                                                              u32x4 *__restrict__ dst, int64_t n) {
    const int64_t step = static_cast<int64_t>(gridDim.x) * kThreads;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n; i += step)
        dst[i] = src[i];
}

template <int D>
hipError_t launch_decode_d(const DecodeArgs &a, hipStream_t stream, bool timeline) {
    if (a.n_items > 0) {
        if (a.deep_prefetch) {
            if (timeline)
                hipLaunchKernelGGL((decode_split_kernel<D, 2, true>), dim3(a.n_items), dim3(kThreads), 0, stream, a);
            else
                hipLaunchKernelGGL((decode_split_kernel<D, 2>), dim3(a.n_items), dim3(kThreads), 0, stream, a);
        } else {
            if (timeline)
                hipLaunchKernelGGL((decode_split_kernel<D, 1, true>), dim3(a.n_items), dim3(kThreads), 0, stream, a);
            else
                hipLaunchKernelGGL((decode_split_kernel<D, 1>), dim3(a.n_items), dim3(kThreads), 0, stream, a);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // one row per wave while the rows fit one round of resident waves (8 per
    // SIMD), two per wave (NB = 4 at D = 128, 8 waves per SIMD) beyond
    const int64_t rows = static_cast<int64_t>(a.P) * a.G * a.Hq;
    if (rows > 8 * 4 * kNumCUs) {
        const int64_t blocks = ((rows + 1) / 2 + 3) / 4;
        hipLaunchKernelGGL((decode_combine_kernel<D, 2, D == 128 ? 4 : 8>), dim3(static_cast<uint32_t>(blocks)),
                           dim3(kThreads), 0, stream, a);
    } else {
        const int64_t blocks = (rows + 3) / 4;
        hipLaunchKernelGGL((decode_combine_kernel<D, 1, 8>), dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0,
                           stream, a);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_plan_fetch(const void *host_src, void *dst, size_t bytes, hipStream_t stream) {
    if (bytes % 16 != 0) return hipErrorInvalidValue;
    const int64_t n = static_cast<int64_t>(bytes / 16);
    if (n == 0) return hipSuccess;
    const int64_t blocks = std::min<int64_t>((n + kThreads - 1) / kThreads, 256);
    hipLaunchKernelGGL(plan_fetch_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0, stream,
                       static_cast<const u32x4 *>(host_src), static_cast<u32x4 *>(dst), n);
    return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs &a, hipStream_t stream, bool timeline) {
    switch (a.D) {
        case 64: return launch_decode_d<64>(a, stream, timeline);
        case 128: return launch_decode_d<128>(a, stream, timeline);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace rlk
