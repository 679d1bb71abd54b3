// Index arithmetic of the decode attention kernels (split and combine), in
// one place: the kernels compute their global addresses through these
// functions, and the host replay in bounds.cpp calls the same functions to
// check that every global access of a call stays inside its allocation.
// Nothing here touches memory.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"
#include "plan.h"

#define RLK_DHD __host__ __device__ __forceinline__

namespace rlk {

// The fields of a work item (DevItem::meta): its kv head, whether it is a
// suffix chunk, its first query row within its unit, and its token count;
// the unit's query rows (r for a suffix, G r for a prefix) and the item's
// (at most kMaxItemRows).
RLK_DHD int dec_kh(uint32_t meta) { return (meta >> 16) & 255; }
RLK_DHD bool dec_is_suffix(uint32_t meta) { return (meta >> 15) & 1; }
RLK_DHD int dec_row_begin(uint32_t meta) { return static_cast<int>(meta >> 24) * kMaxItemRows; }
RLK_DHD int dec_ntok(uint32_t meta) { return static_cast<int>(meta & 0x7fff); }
RLK_DHD int dec_unit_rows(const DecodeArgs &a, bool is_suffix) { return is_suffix ? a.r : a.G * a.r; }
RLK_DHD int dec_item_rows(int M, int row_begin) { return min(kMaxItemRows, M - row_begin); }
struct DecItem {
    int kh;
    bool is_suffix;
};

// K/V layouts: token-major [rows, Hkv, D] (rows of one kv head are Hkv*D
// elements apart) or head-major [Hkv, rows, D] (contiguous).  Element stride
// between consecutive tokens, and the element offset of the chunk's first
// token at the item's kv head in its (prefix or suffix) buffer.
RLK_DHD int64_t dec_tok_stride(const DecodeArgs &a, int D) {
    return a.kv_layout == RL_KV_HEAD_MAJOR ? D : static_cast<int64_t>(a.Hkv) * D;
}
RLK_DHD int64_t dec_kv_base(const DecodeArgs &a, const DevItem &it, const DecItem &d, int D) {
    const int64_t nrows = d.is_suffix ? a.suffix_rows : a.prefix_rows;
    const int64_t kv_row0 = it.kv_row0;
    return a.kv_layout == RL_KV_HEAD_MAJOR ? (d.kh * nrows + kv_row0) * D : (kv_row0 * a.Hkv + d.kh) * D;
}

// Element offset of the query row (of the [S, Hq, D] queries) of row ig of
// the item's unit.
RLK_DHD int64_t dec_q_off(const DecodeArgs &a, const DevItem &it, const DecItem &d, int ig, int D) {
    int s, h;
    if (d.is_suffix) {
        s = it.unit;
        h = d.kh * a.r + ig;
    } else {
        s = it.unit * a.G + ig / a.r;
        h = d.kh * a.r + ig % a.r;
    }
    return (static_cast<int64_t>(s) * a.Hq + h) * D;
}

// The buffer descriptor of the tile starting at token t0 of a chunk of ntok
// tokens: its first element (from the chunk's base) and its range in bytes,
// which ends with the chunk's last row, so rows past the chunk read as zeros;
// a tile past the chunk gets an empty range.
RLK_DHD int64_t dec_tile_first(int t0, int ntok, int64_t tok_stride) {
    return t0 < ntok ? static_cast<int64_t>(t0) * tok_stride : 0;
}
RLK_DHD int dec_tile_range(int t0, int ntok, int64_t tok_stride, int D) {
    return t0 < ntok ? static_cast<int>((static_cast<int64_t>(ntok - t0 - 1) * tok_stride + D) * 2) : 0;
}
// Byte offset, inside a tile's descriptor, of 16-byte load idx (chunk idx %
// ch of token idx / ch, ch = 16-byte chunks per token row).
RLK_DHD uint32_t dec_load_off(int idx, int ch, int64_t tok_stride) {
    return static_cast<uint32_t>((idx / ch) * tok_stride * 2 + (idx % ch) * 16);
}

// The partial rows that the combine merges for query row (sequence s, head
// h = kh r + hr, s = p G + g): the prompt's prefix chunks (unit pu), then the
// candidate's suffix chunks (unit su), at the head's kv head.  Partial j of
// the row is at dec_partial_row(pbase, sbase, Mp, pn, r, j), pn = pu.nchunks.
RLK_DHD int64_t dec_prefix_partial_base(const DevUnit &pu, int kh, int64_t Mp, int g, int r, int hr) {
    return pu.base + static_cast<int64_t>(kh) * pu.nchunks * Mp + g * r + hr;
}
RLK_DHD int64_t dec_suffix_partial_base(const DevUnit &su, int kh, int r, int hr) {
    return su.base + static_cast<int64_t>(kh) * su.nchunks * r + hr;
}
RLK_DHD int64_t dec_partial_row(int64_t pbase, int64_t sbase, int64_t Mp, int pn, int r, int j) {
    return j < pn ? pbase + j * Mp : sbase + static_cast<int64_t>(j - pn) * r;
}

}  // namespace rlk
