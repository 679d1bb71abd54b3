// Index arithmetic of the extend (prefill) attention kernel, in one place:
// the kernel computes its global addresses through these functions, and the
// host replay in bounds.cpp calls the same functions to check that every
// global access of a call stays inside its allocation.  Nothing here touches
// memory.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"
#include "plan.h"

#define RLK_XHD __host__ __device__ __forceinline__

namespace rlk {

constexpr int kExtTileTokens = 64;      // KV tokens per tile of the context
// The launched kernel: 8 wave64s per block, wave w owning query rows
// 32 w .. 32 w + 31 of the block.
constexpr int kExtWaves = 8;
constexpr int kExtRowsPerWave = 32;

// Where a work block sits: its query rows and the tiles of context it reads.
// Unit row u = token * r + head in the group; the block's rows are
// [row_begin, row_begin + rows) of its candidate at its kv head.
struct ExtGeom {
    int rows;          // query rows of the block (<= kExtBlockRows)
    int i_lo, i_hi;    // first and last new token of the block
    int base_pos;      // suffix position of the candidate's new token 0
    int suf_ctx;       // suffix tokens the block reads (up to its last token)
    int np;            // prefix tiles
    int ntiles;        // prefix tiles, then suffix tiles
};
RLK_XHD ExtGeom ext_geom(const ExtItem &it, int r) {
    ExtGeom g;
    const int left = it.n * r - it.row_begin;
    g.rows = left < kExtBlockRows ? left : kExtBlockRows;
    g.i_lo = it.row_begin / r;
    g.i_hi = (it.row_begin + g.rows - 1) / r;
    g.base_pos = it.Ls - it.n;
    g.suf_ctx = g.base_pos + g.i_hi + 1;
    g.np = (it.Lp + kExtTileTokens - 1) / kExtTileTokens;
    g.ntiles = g.np + (g.suf_ctx + kExtTileTokens - 1) / kExtTileTokens;
    return g;
}

// K/V layouts: token-major [rows, Hkv, D] (a kv head's rows are Hkv*D
// elements apart) or head-major [Hkv, rows, D] (contiguous).  Element stride
// between consecutive tokens of one kv head, and the element offset of the
// item's first prefix / suffix token at its kv head.
RLK_XHD int64_t ext_tok_stride(const ExtendArgs &a, int D) {
    return a.kv_layout == RL_KV_HEAD_MAJOR ? D : static_cast<int64_t>(a.Hkv) * D;
}
RLK_XHD int64_t ext_prefix_off(const ExtendArgs &a, const ExtItem &it, int D) {
    return a.kv_layout == RL_KV_HEAD_MAJOR ? (it.kh * a.prefix_rows + it.prefix_row0) * D
                                           : (it.prefix_row0 * a.Hkv + it.kh) * D;
}
RLK_XHD int64_t ext_suffix_off(const ExtendArgs &a, const ExtItem &it, int D) {
    return a.kv_layout == RL_KV_HEAD_MAJOR ? (it.kh * a.suffix_rows + it.suffix_row0) * D
                                           : (it.suffix_row0 * a.Hkv + it.kh) * D;
}

// Query / output row (of the [q_rows, Hq] rows) of unit row u of the item.
RLK_XHD int64_t ext_q_row(const ExtendArgs &a, const ExtItem &it, int u) {
    const int i = u / a.r, hr = u - i * a.r;
    return (it.q_row0 + i) * a.Hq + it.kh * a.r + hr;
}

// Tile t: its first token (of the prefix for t < np, else of the suffix)
// and its token count (the last tile of each range may be ragged).
RLK_XHD int ext_tile_tok0(int t, int np) { return (t < np ? t : t - np) * kExtTileTokens; }
RLK_XHD int ext_tile_cnt(int t, int np, int Lp, int suf_ctx) {
    const int c = (t < np ? Lp : suf_ctx) - ext_tile_tok0(t, np);
    return c < kExtTileTokens ? c : kExtTileTokens;
}

// Chunk swizzle of token row t of a tile in LDS.  D = 128: rows are 256
// bytes (one window of the 64 banks); the 16 rows a K-fragment pass reads and
// the 4 rows x 4 chunks a V^T pass reads map to 16 distinct 16-byte slots.
// D = 64: two 128-byte rows share a window; the same holds with the row
// parity selecting the half.
template <int D>
RLK_XHD int ext_swz(int t) {
    if constexpr (D == 128) {
        return ((t & 3) << 2) | ((t >> 2) & 3);
    } else {
        const int v = (t >> 1) & 7;
        return ((v & 1) << 2) | (v >> 1);
    }
}

// Direct load e (= 64 * load instruction + lane) of a tile fills 16-byte LDS
// slot e % (D / 8) of token row e / (D / 8); it fetches the chunk the swizzle
// stores there.  Element offset of that chunk in the token's row.
template <int D>
RLK_XHD int ext_load_tok(int e) { return e / (D / 8); }
template <int D>
RLK_XHD int ext_load_chunk(int e) {
    const int tt = e / (D / 8), slot = e % (D / 8);
    return (slot ^ ext_swz<D>(tt)) << 3;
}
// Byte offset of that load from the tile's first token, in a full tile and
// in a ragged tile of cnt tokens (rows past its tokens re-read its last one).
RLK_XHD uint32_t ext_load_off_full(int tt, int64_t tok_stride, int chk) {
    return static_cast<uint32_t>((tt * tok_stride + chk) * 2);
}
RLK_XHD uint32_t ext_load_off(int tt, int cnt, int64_t tok_stride, int chk) {
    const int t = tt < cnt - 1 ? tt : cnt - 1;
    return static_cast<uint32_t>((t * tok_stride + chk) * 2);
}

}  // namespace rlk
