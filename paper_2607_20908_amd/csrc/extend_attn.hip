// Causal extend (prefill) attention over a prompt-shared prefix for gfx950.
//
// One workgroup (4 wave64s, one per SIMD) serves one block of up to 256 query
// rows of one candidate at one kv head.  Unit row u = token * r + head in the
// group, so the r query heads of a token sit side by side and share its causal
// limit.  Wave w owns rows 64w .. 64w+63 as two 32-row MFMA column tiles.
//
// The visible context (the prompt's prefix, then the candidate's suffix up to
// the block's last token) streams through a 3-stage LDS ring in tiles of 64
// tokens.  Direct global->LDS loads fill it two tiles ahead.  Per tile a wave:
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
#include "kernels.h"
#include "lds_stage.h"

namespace rlk {
namespace {

constexpr int kThreads = 256;
constexpr int kBN = 64;        // KV tokens per tile
constexpr int kStages = 3;     // LDS ring depth

template <int D>
struct ECfg {
    static constexpr int CH = D / 8;              // 16-byte chunks per token row
    static constexpr int TILE = kBN * D;          // bf16 elements of one K or V tile
    static constexpr int KK = D / 16;             // k-steps of S^T = K Q^T
    static constexpr int DT = D / 32;             // 32-wide d tiles of O^T
    static constexpr int LPW = TILE / 512 / 4;    // 1 KB direct loads per wave per tensor per tile
};

// Chunk swizzle of token row t.  D = 128: rows are 256 bytes (one window of
// the 64 banks); the 16 rows a K-fragment pass reads and the 4 rows x 4 chunks
// a V^T pass reads map to 16 distinct 16-byte slots.  D = 64: two 128-byte rows
// share a window; the same holds with the row parity selecting the half.
template <int D>
__device__ __forceinline__ int swz(int t) {
    if constexpr (D == 128) {
        return ((t & 3) << 2) | ((t >> 2) & 3);
    } else {
        const int v = (t >> 1) & 7;
        return ((v & 1) << 2) | (v >> 1);
    }
}

// Element offset of (token t, dimension d) inside a K or V tile.
template <int D>
__device__ __forceinline__ int kv_elem(int t, int d) {
    return t * D + ((((d >> 3) ^ swz<D>(t))) << 3) + (d & 7);
}

template <int D>
__global__ __launch_bounds__(kThreads, 1) void extend_attn_kernel(ExtendArgs a) {
    using C = ECfg<D>;
    __shared__ __attribute__((aligned(16))) uint16_t ring[kStages * 2 * C::TILE];

    const ExtItem it = a.items[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, h2 = lane >> 5, l16 = lane & 15, g16 = (lane >> 4) & 1;
    const int r = a.r;
    const int rows = min(kExtBlockRows, it.n * r - it.row_begin);
    const int i_lo = it.row_begin / r;
    const int i_hi = (it.row_begin + rows - 1) / r;
    const int base_pos = it.Ls - it.n;            // suffix position of new token 0
    const int suf_ctx = base_pos + i_hi + 1;      // suffix tokens the block reads
    const int np = (it.Lp + kBN - 1) / kBN;
    const int ntiles = np + (suf_ctx + kBN - 1) / kBN;

    // token-major [rows, Hkv, D]: a kv head's rows are Hkv*D apart;
    // head-major [Hkv, rows, D]: contiguous
    const bool head_major = a.kv_layout == RL_KV_HEAD_MAJOR;
    const int64_t tok_stride = head_major ? D : static_cast<int64_t>(a.Hkv) * D;
    const int64_t poff = head_major ? (it.kh * a.prefix_rows + it.prefix_row0) * D
                                    : (it.prefix_row0 * a.Hkv + it.kh) * D;
    const int64_t soff = head_major ? (it.kh * a.suffix_rows + it.suffix_row0) * D
                                    : (it.suffix_row0 * a.Hkv + it.kh) * D;
    const uint16_t *kpre = it.Lp > 0 ? a.k_prefix + poff : nullptr;
    const uint16_t *vpre = it.Lp > 0 ? a.v_prefix + poff : nullptr;
    const uint16_t *ksuf = a.k_suffix + soff;
    const uint16_t *vsuf = a.v_suffix + soff;

    // ---- this wave's query rows as MFMA B operands (Q^T, k = d) -------------
    bf16x8 qf[2][C::KK];
    int lim[2];                                   // last visible suffix position per row
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
        const int row = wave * 64 + tn * 32 + l32;
        const bool ok = row < rows;
        const int u = it.row_begin + (ok ? row : rows - 1);
        const int i = u / r, hr = u - i * r;
        lim[tn] = base_pos + i;
        const int64_t qoff = ((it.q_row0 + i) * a.Hq + it.kh * r + hr) * D + h2 * 8;
#pragma unroll
        for (int kk = 0; kk < C::KK; ++kk)
            qf[tn][kk] = ok ? *reinterpret_cast<const bf16x8 *>(a.q + qoff + kk * 16) : bf16x8{};
    }

    // ---- tile t of the context into ring stage t % kStages -------------------
    // Lane i of load instruction j writes the 16-byte slot i of the 1 KB block
    // j, i.e. row (64j + i) / CH, slot (64j + i) % CH; it fetches the chunk that
    // the swizzle stores there.  Rows past the tile's tokens re-read its last
    // token (never a row outside the range); their scores are masked.
    auto issue = [&](int t) {
        uint16_t *kl = ring + (t % kStages) * 2 * C::TILE;
        uint16_t *vl = kl + C::TILE;
        const bool pre = t < np;
        const int tok0 = (pre ? t : t - np) * kBN;
        const int cnt = min(kBN, (pre ? it.Lp : suf_ctx) - tok0);
        const uint16_t *kg = pre ? kpre : ksuf;
        const uint16_t *vg = pre ? vpre : vsuf;
#pragma unroll
        for (int j = 0; j < C::LPW; ++j) {
            const int inst = wave * C::LPW + j;
            const int e = inst * 64 + lane;
            const int tt = e / C::CH, slot = e % C::CH;
            const int64_t off = static_cast<int64_t>(tok0 + min(tt, cnt - 1)) * tok_stride +
                                ((slot ^ swz<D>(tt)) << 3);
            load_lds16(kg + off, kl + inst * 512);
        }
#pragma unroll
        for (int j = 0; j < C::LPW; ++j) {
            const int inst = wave * C::LPW + j;
            const int e = inst * 64 + lane;
            const int tt = e / C::CH, slot = e % C::CH;
            const int64_t off = static_cast<int64_t>(tok0 + min(tt, cnt - 1)) * tok_stride +
                                ((slot ^ swz<D>(tt)) << 3);
            load_lds16(vg + off, vl + inst * 512);
        }
    };

    float m_run[2] = {-INFINITY, -INFINITY};      // running max, log2 units
    float l_run[2] = {0.f, 0.f};                  // this lane's share of the row sum
    f32x16 acc[C::DT][2];
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) acc[dt][tn] = f32x16{};
    const float c2 = a.score_scale_log2;

    issue(0);
    if (ntiles > 1) issue(1);
    for (int t = 0; t < ntiles; ++t) {
        // tile t has landed once only tile t+1's loads may still be in flight;
        // the barrier also frees stage (t+2) % 3, last read for tile t-1
        if (t + 1 < ntiles) wait_vm<2 * C::LPW>();
        else wait_vm<0>();
        barrier();
        if (t + 2 < ntiles) issue(t + 2);
        const uint16_t *kl = ring + (t % kStages) * 2 * C::TILE;
        const uint16_t *vl = kl + C::TILE;
        const bool pre = t < np;
        const int tok0 = (pre ? t : t - np) * kBN;
        const int cnt = min(kBN, (pre ? it.Lp : suf_ctx) - tok0);

        // S^T: sc[tm][tn][v] is token 32 tm + 8 (v/4) + 4 h2 + v%4 of row tn*32 + l32
        f32x16 sc[2][2];
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
#pragma unroll
            for (int tn = 0; tn < 2; ++tn) sc[tm][tn] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < C::KK; ++kk) {
            const bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(kl + kv_elem<D>(l32, kk * 16 + h2 * 8));
            const bf16x8 a1 = *reinterpret_cast<const bf16x8 *>(kl + kv_elem<D>(32 + l32, kk * 16 + h2 * 8));
            sc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[0][kk], sc[0][0], 0, 0, 0);
            sc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[1][kk], sc[0][1], 0, 0, 0);
            sc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[0][kk], sc[1][0], 0, 0, 0);
            sc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[1][kk], sc[1][1], 0, 0, 0);
        }
        // tokens past the tile, and suffix tokens after a row's own position
        if (cnt < kBN || (!pre && tok0 + kBN - 1 > base_pos + i_lo)) {
#pragma unroll
            for (int tm = 0; tm < 2; ++tm)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int tok = 32 * tm + 8 * (v >> 2) + 4 * h2 + (v & 3);
#pragma unroll
                    for (int tn = 0; tn < 2; ++tn) {
                        const bool vis = tok < cnt && (pre || tok0 + tok <= lim[tn]);
                        if (!vis) sc[tm][tn][v] = -INFINITY;
                    }
                }
        }
        // online softmax; pb[tn][ks] slot e (of lane half h2) is token
        // 16 ks + 8 (e/4) + 4 h2 + e%4, i.e. score sc[ks/2][tn][8 (ks%2) + e]
        bf16x8 pb[2][4];
        float alpha[2];
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) {
            float mx = -INFINITY;
#pragma unroll
            for (int tm = 0; tm < 2; ++tm)
#pragma unroll
                for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sc[tm][tn][v]);
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const float m_new = fmaxf(m_run[tn], mx * c2);
            const float m_use = m_new == -INFINITY ? 0.f : m_new;
            alpha[tn] = fast_exp2(m_run[tn] - m_use);
            m_run[tn] = m_new;
            float ps = 0.f;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float p = fast_exp2(fmaf(sc[ks >> 1][tn][8 * (ks & 1) + e], c2, -m_use));
                    ps += p;
                    pb[tn][ks][e] = static_cast<__bf16>(p);
                }
            l_run[tn] = l_run[tn] * alpha[tn] + ps;
        }
        // the running max rarely moves after the first tiles: rescale only when
        // it moved for some row of the wave
        if (__any(alpha[0] != 1.f || alpha[1] != 1.f)) {
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt) {
                acc[dt][0] *= alpha[0];
                acc[dt][1] *= alpha[1];
            }
        }
        // O^T += V^T P^T.  Lane (l32, h2) needs V[16 ks + 4 h2 + 0..3][32 dt + l32]
        // and V[16 ks + 8 + 4 h2 + 0..3][32 dt + l32]: one transposing read each,
        // source lane s of a 16-lane group pointing at token +s/4, d + 4 (s%4).
        const int tA = 4 * h2 + (l16 >> 2);
        const int dA = 16 * g16 + 4 * (l16 & 3);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt) {
                const bf16x4 lo = lds_read_tr16(vl + kv_elem<D>(16 * ks + tA, 32 * dt + dA));
                const bf16x4 hi = lds_read_tr16(vl + kv_elem<D>(16 * ks + 8 + tA, 32 * dt + dA));
                const bf16x8 va = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                acc[dt][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[0][ks], acc[dt][0], 0, 0, 0);
                acc[dt][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[1][ks], acc[dt][1], 0, 0, 0);
            }
        }
    }

    // ---- normalise and write: acc[dt][tn][v] is d = 32 dt + 8 (v/4) + 4 h2 + v%4
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
        const float l = l_run[tn] + __shfl_xor(l_run[tn], 32, 64);
        const int row = wave * 64 + tn * 32 + l32;
        if (row < rows) {
            const int u = it.row_begin + row;
            const int i = u / r, hr = u - i * r;
            const int64_t orow = (it.q_row0 + i) * a.Hq + it.kh * r + hr;
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
            if (h2 == 0 && a.lse) a.lse[orow] = (m_run[tn] + fast_log2(l)) * kLn2;
        }
    }
}

template <int D>
hipError_t launch_extend_d(const ExtendArgs &a, hipStream_t stream) {
    if (a.n_items == 0) return hipSuccess;
    hipLaunchKernelGGL(extend_attn_kernel<D>, dim3(static_cast<uint32_t>(a.n_items)), dim3(kThreads), 0, stream,
                       a);
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
