// Causal extend (prefill) attention over a prompt-shared prefix for gfx950.
//
// One workgroup serves one block of up to 256 query rows of one candidate at
// one kv head.  Unit row u = token * r + head in the group, so the r query
// heads of a token sit side by side and share its causal limit.  The kernel
// is templated on NT, the 32-row MFMA column tiles per wave; the launched
// variant has NT = 1: 8 wave64s (two per SIMD, so one wave's softmax and LDS
// waits overlap the other's MFMAs), wave w owning rows 32w .. 32w+31.
//
// The visible context (the prompt's prefix, then the candidate's suffix up to
// the block's last token) streams through a 4-stage LDS ring in tiles of 64
// tokens.  Direct global->LDS loads fill it three tiles ahead.  Per tile a wave:
//  - computes S^T = K Q^T on MFMA 32x32x16 bf16, tokens on M and query rows on
//    N, so each lane holds 32 scores of one row and the row max and sum are
//    in-lane plus one shuffle across the lane halves;
//  - updates the online softmax in fp32 with exp2 and rounds the probabilities
//    to bf16;
//  - accumulates O^T += V^T P^T on MFMA 32x32x16.  P^T is the score tile's
//    output layout read in a token order that puts each lane's own scores on
//    its B-operand slots; the V^T operand follows that order through
//    transposing LDS reads.
// Tiles are stored unpadded with a per-row XOR swizzle of the 16-byte chunks,
// which keeps both fragment reads free of bank conflicts (64 banks) and lets
// every direct load write 1 KB contiguously.
#include "device_common.h"
#include "extend_index.h"
#include "kernels.h"
#include "lds_stage.h"

namespace rlk {
namespace {

constexpr int kBN = kExtTileTokens;   // KV tokens per tile
constexpr int kStages = 4;     // LDS ring depth

// NT: 32-row MFMA column tiles per wave; the workgroup's 256 rows take 8 / NT
// waves.
template <int D, int NT>
struct ECfg {
    static constexpr int WAVES = 8 / NT;
    static constexpr int THREADS = 64 * WAVES;
    static constexpr int CH = D / 8;              // 16-byte chunks per token row
    static constexpr int TILE = kBN * D;          // bf16 elements of one K or V tile
    static constexpr int KK = D / 16;             // k-steps of S^T = K Q^T
    static constexpr int DT = D / 32;             // 32-wide d tiles of O^T
    static constexpr int LPW = TILE / 512 / WAVES;  // 1 KB direct loads per wave per tensor per tile
    static_assert(LPW >= 1 && LPW * 512 * WAVES == TILE, "load split");
};

// Element offset of (token t, dimension d) inside a K or V tile (chunks
// swizzled by ext_swz).
template <int D>
__device__ __forceinline__ int kv_elem(int t, int d) {
    return t * D + ((((d >> 3) ^ ext_swz<D>(t))) << 3) + (d & 7);
}

// Rows keep the max they exponentiate against until a new score exceeds it by
// more than this many log2 units: probabilities stay below 2^8 (exact in
// fp32, in range for bf16), the accumulators are rescaled only when the max
// really moves, and out = acc / l and lse = m + log2 l are unchanged.
constexpr float kRescaleLog2 = 8.f;

template <int D, int NT>
__global__ __launch_bounds__(64 * (8 / NT), 1) void extend_attn_kernel(ExtendArgs a) {
    using C = ECfg<D, NT>;
    __shared__ __attribute__((aligned(16))) uint16_t ring[kStages * 2 * C::TILE];

    release_staging(a.release);
    const ExtItem it = a.items[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, h2 = lane >> 5, l16 = lane & 15, g16 = (lane >> 4) & 1;
    const int r = a.r;
    const ExtGeom gm = ext_geom(it, r);
    const int rows = gm.rows, i_lo = gm.i_lo;
    const int base_pos = gm.base_pos;             // suffix position of new token 0
    const int suf_ctx = gm.suf_ctx;               // suffix tokens the block reads
    const int np = gm.np, ntiles = gm.ntiles;

    const int64_t tok_stride = ext_tok_stride(a, D);
    const int64_t poff = ext_prefix_off(a, it, D);
    const int64_t soff = ext_suffix_off(a, it, D);
    const uint16_t *kpre = it.Lp > 0 ? a.k_prefix + poff : nullptr;
    const uint16_t *vpre = it.Lp > 0 ? a.v_prefix + poff : nullptr;
    const uint16_t *ksuf = a.k_suffix + soff;
    const uint16_t *vsuf = a.v_suffix + soff;

    // ---- this wave's query rows as MFMA B operands (Q^T, k = d) -------------
    bf16x8 qf[NT][C::KK];
    int lim[NT];                                  // last visible suffix position per row
#pragma unroll
    for (int tn = 0; tn < NT; ++tn) {
        const int row = wave * 32 * NT + tn * 32 + l32;
        const bool ok = row < rows;
        const int u = it.row_begin + (ok ? row : rows - 1);
        lim[tn] = base_pos + u / r;
        const int64_t qoff = ext_q_row(a, it, u) * D + h2 * 8;
#pragma unroll
        for (int kk = 0; kk < C::KK; ++kk)
            qf[tn][kk] = ok ? *reinterpret_cast<const bf16x8 *>(a.q + qoff + kk * 16) : bf16x8{};
    }

    // ---- tile t of the context into ring stage t % kStages -------------------
    // Lane i of load instruction j writes the 16-byte slot i of the 1 KB block
    // j, i.e. row (64j + i) / CH, slot (64j + i) % CH; it fetches the chunk that
    // the swizzle stores there.  In a ragged last tile, rows past its tokens
    // re-read its last token (never a row outside the range); their scores are
    // masked.
    // per-lane byte offsets of this wave's loads in a full tile (token row x
    // stride + swizzled chunk); a ragged last tile clamps the token row
    uint32_t ld_off[C::LPW];
    int ld_tok[C::LPW], ld_chk[C::LPW];
#pragma unroll
    for (int j = 0; j < C::LPW; ++j) {
        const int e = (wave * C::LPW + j) * 64 + lane;
        ld_tok[j] = ext_load_tok<D>(e);
        ld_chk[j] = ext_load_chunk<D>(e);
        ld_off[j] = ext_load_off_full(ld_tok[j], tok_stride, ld_chk[j]);
    }
    auto tile_tok0 = [&](int t) { return ext_tile_tok0(t, np); };
    auto tile_cnt = [&](int t) { return ext_tile_cnt(t, np, it.Lp, suf_ctx); };
    const uint32_t ring_l = lds_addr(ring);
    auto issue = [&](int t) {
        const uint32_t kl = ring_l + (t % kStages) * (2 * C::TILE * 2);
        const uint32_t vl = kl + C::TILE * 2;
        const bool pre = t < np;
        const int tok0 = tile_tok0(t), cnt = tile_cnt(t);
        const uint16_t *kg = (pre ? kpre : ksuf) + tok0 * tok_stride;
        const uint16_t *vg = (pre ? vpre : vsuf) + tok0 * tok_stride;
        if (cnt == kBN) {
#pragma unroll
            for (int j = 0; j < C::LPW; ++j) load_lds16_s(kg, ld_off[j], kl + (wave * C::LPW + j) * 1024);
#pragma unroll
            for (int j = 0; j < C::LPW; ++j) load_lds16_s(vg, ld_off[j], vl + (wave * C::LPW + j) * 1024);
        } else {
            uint32_t off[C::LPW];
#pragma unroll
            for (int j = 0; j < C::LPW; ++j)
                off[j] = ext_load_off(ld_tok[j], cnt, tok_stride, ld_chk[j]);
#pragma unroll
            for (int j = 0; j < C::LPW; ++j) load_lds16_s(kg, off[j], kl + (wave * C::LPW + j) * 1024);
#pragma unroll
            for (int j = 0; j < C::LPW; ++j) load_lds16_s(vg, off[j], vl + (wave * C::LPW + j) * 1024);
        }
    };
    auto stage_k = [&](int t) -> const uint16_t * { return ring + (t % kStages) * 2 * C::TILE; };

    // Per-lane LDS read offsets inside a tile.  The swizzle of row t depends
    // on t mod 16 only, so the 32-token half (K) and the 16-token k-step (V)
    // add compile-time offsets to these.
    int koff[C::KK];
#pragma unroll
    for (int kk = 0; kk < C::KK; ++kk) koff[kk] = kv_elem<D>(l32, kk * 16 + h2 * 8);
    const int tA = 4 * h2 + (l16 >> 2);
    const int dA = 16 * g16 + 4 * (l16 & 3);
    int voff[2][C::DT];
#pragma unroll
    for (int sel = 0; sel < 2; ++sel)
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt) voff[sel][dt] = C::TILE + kv_elem<D>(8 * sel + tA, 32 * dt + dA);

    // S^T of the 32-token half tm of the tile in stage kl: sc[tn][v] is token
    // 32 tm + 8 (v/4) + 4 h2 + v%4 of row tn*32 + l32
    auto scores = [&](const uint16_t *kl, int tm, f32x16 (&sc)[NT]) {
#pragma unroll
        for (int tn = 0; tn < NT; ++tn) sc[tn] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < C::KK; ++kk) {
            const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(kl + koff[kk] + 32 * tm * D);
#pragma unroll
            for (int tn = 0; tn < NT; ++tn)
                sc[tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[tn][kk], sc[tn], 0, 0, 0);
        }
    };
    // tokens past the tile's count, and suffix tokens after a row's own
    // position: a row sees the first vis tokens of the tile
    auto mask = [&](f32x16 (&sc)[NT], int tm, int t) {
        const int tok0 = tile_tok0(t), cnt = tile_cnt(t);
#pragma unroll
        for (int tn = 0; tn < NT; ++tn) {
            const int vis = (t < np ? cnt : min(cnt, lim[tn] - tok0 + 1)) - 32 * tm - 4 * h2;
#pragma unroll
            for (int v = 0; v < 16; ++v)
                sc[tn][v] = 8 * (v >> 2) + (v & 3) < vis ? sc[tn][v] : -INFINITY;
        }
    };
    auto masked_tile = [&](int t) {
        return tile_cnt(t) < kBN || (t >= np && tile_tok0(t) + kBN - 1 > base_pos + i_lo);
    };
    // O^T += V^T P^T over half tm.  Lane (l32, h2) needs V[16 ks + 4 h2 + 0..3]
    // [32 dt + l32] and V[16 ks + 8 + 4 h2 + 0..3][32 dt + l32]: one transposing
    // read each, source lane s of a 16-lane group pointing at token +s/4, d + 4 (s%4).
    f32x16 acc[C::DT][NT];
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int tn = 0; tn < NT; ++tn) acc[dt][tn] = f32x16{};
    auto values = [&](const uint16_t *kl, int tm, const bf16x8 (&pb)[NT][2]) {
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
            const int ks = 2 * tm + kh;
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt) {
                const bf16x4 lo = lds_read_tr16(kl + voff[0][dt] + 16 * ks * D);
                const bf16x4 hi = lds_read_tr16(kl + voff[1][dt] + 16 * ks * D);
                const bf16x8 va = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
                for (int tn = 0; tn < NT; ++tn)
                    acc[dt][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[tn][kh], acc[dt][tn], 0, 0, 0);
            }
        }
    };

    float m_ref[NT], l_run[NT];                   // reference max (log2 units); this lane's
    float mx[NT];                                 // share of the row sum; the half's row max
#pragma unroll
    for (int tn = 0; tn < NT; ++tn) {
        m_ref[tn] = -INFINITY;
        l_run[tn] = 0.f;
    }
    const float c2 = a.score_scale_log2;
    f32x16 s_cur[NT], s_next[NT];

    // One half-step (tile t, half h) on s_cur: mask, row max, and unless the
    // max moved past the reference (then it returns false having changed
    // nothing), the probabilities, the next half's scores and this half's
    // value products.  Nothing here touches the accumulators with VALU work,
    // so they stay in the MFMA accumulator registers.
    auto step = [&](int t, int h) -> bool {
        if (masked_tile(t)) mask(s_cur, h, t);
        bool mv = false;
#pragma unroll
        for (int tn = 0; tn < NT; ++tn) {
            float m = -INFINITY;
#pragma unroll
            for (int v = 0; v < 16; ++v) m = fmaxf(m, s_cur[tn][v]);
            mx[tn] = half_swap_max(m) * c2;
            mv |= mx[tn] > m_ref[tn] + kRescaleLog2;
        }
        if (__any(mv)) return false;
        if (h == 1 && t + 1 < ntiles) {
            // tile t+1 must have landed (only tile t+2's loads may be in flight);
            // the barrier also frees stage (t+3) % 4, last read for tile t-1
            if (t + 2 < ntiles) wait_vm<2 * C::LPW>();
            else wait_vm<0>();
            barrier();
            if (t + 3 < ntiles) issue(t + 3);
        }
        // probabilities as bf16 (the operand of the value MFMA); the row sum
        // in fp32, so lse keeps fp32 accuracy
        bf16x8 pb[NT][2];
#pragma unroll
        for (int tn = 0; tn < NT; ++tn) {
            float ps = 0.f;
#pragma unroll
            for (int kh = 0; kh < 2; ++kh)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float p = fast_exp2(fmaf(s_cur[tn][8 * kh + e], c2, -m_ref[tn]));
                    ps += p;
                    pb[tn][kh][e] = static_cast<__bf16>(p);
                }
            l_run[tn] += ps;
        }
        // the next half's scores: tile t's second half, or tile t+1's first
        // (past the last tile this reads a stale stage; the result is unused)
        scores(stage_k(h == 0 ? t : t + 1), h == 0 ? 1 : 0, s_next);
        values(stage_k(t), h, pb);
#pragma unroll
        for (int tn = 0; tn < NT; ++tn) s_cur[tn] = s_next[tn];
        return true;
    };

    issue(0);
    if (ntiles > 1) issue(1);
    if (ntiles > 2) issue(2);
    if (ntiles > 2) wait_vm<4 * C::LPW>();
    else if (ntiles > 1) wait_vm<2 * C::LPW>();
    else wait_vm<0>();
    barrier();
    scores(stage_k(0), 0, s_cur);

    int t = 0, h_start = 0;
    for (;;) {
        bool bail = false;
        for (; t < ntiles; ++t) {
            if (h_start == 0 && !step(t, 0)) { bail = true; break; }
            if (!step(t, 1)) { h_start = 1; bail = true; break; }
            h_start = 0;
        }
        if (!bail) break;
        // A row's max moved by more than the threshold (always on the first
        // half-step): move the reference to the new max and rescale what the
        // row has accumulated, then redo the step.
        float al[NT];
#pragma unroll
        for (int tn = 0; tn < NT; ++tn) {
            const bool up = mx[tn] > m_ref[tn] + kRescaleLog2;
            const float m_new = up ? mx[tn] : m_ref[tn];
            al[tn] = up ? fast_exp2(m_ref[tn] - m_new) : 1.f;
            m_ref[tn] = m_new;
            l_run[tn] *= al[tn];
        }
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
            for (int tn = 0; tn < NT; ++tn) acc[dt][tn] *= al[tn];
    }

    // ---- normalise and write: acc[dt][tn][v] is d = 32 dt + 8 (v/4) + 4 h2 + v%4
#pragma unroll
    for (int tn = 0; tn < NT; ++tn) {
        const float l = half_swap_sum(l_run[tn]);
        const int row = wave * 32 * NT + tn * 32 + l32;
        if (row < rows) {
            const int u = it.row_begin + row;
            const int64_t orow = ext_q_row(a, it, u);
            const float inv = 1.f / l;
            uint16_t *o = a.out + orow * D + 4 * h2;
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    bf16x4 w;
#pragma unroll
                    for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(acc[dt][tn][4 * q4 + e] * inv);
                    *reinterpret_cast<bf16x4 *>(o + 32 * dt + 8 * q4) = w;
                }
            if (h2 == 0 && a.lse) a.lse[orow] = (m_ref[tn] + fast_log2(l)) * kLn2;
        }
    }
}

// One 32-row column tile per wave, 8 waves: two waves per SIMD, so one
// wave's softmax and LDS waits overlap the other's MFMAs.
constexpr int kNT = 1;
static_assert(ECfg<128, kNT>::WAVES == kExtWaves && 32 * kNT == kExtRowsPerWave, "launch geometry of the replay");

template <int D>
hipError_t launch_extend_d(const ExtendArgs &a, hipStream_t stream) {
    if (a.n_items == 0) return hipSuccess;
    hipLaunchKernelGGL((extend_attn_kernel<D, kNT>), dim3(static_cast<uint32_t>(a.n_items)),
                       dim3(ECfg<D, kNT>::THREADS), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_extend(const ExtendArgs &a, hipStream_t stream) {
    switch (a.D) {
        case 64: return launch_extend_d<64>(a, stream);
        case 128: return launch_extend_d<128>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace rlk
