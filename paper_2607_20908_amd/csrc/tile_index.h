// Index arithmetic of the lm-head tile kernels and of the log-prob backward's
// kernels, in one place: the kernels compute every global address through
// these functions, and the host replay in bounds.cpp calls the same functions
// to check, launch by launch, that every global access stays inside its
// allocation.  Nothing here touches memory.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"
#include "plan.h"

#define RLK_HD __host__ __device__ __forceinline__

namespace rlk {

RLK_HD int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }
RLK_HD int mini(int a, int b) { return a < b ? a : b; }

// bf16 elements of one 256 x 64 stage of one operand (32 KB).
constexpr int kStageElems = kVocabTile * kHiddenStep;

// Wave64s per lm-head tile workgroup: wave w owns vocab half w & 1 (128
// entries) and token rows 64 (w >> 1) .. 64 (w >> 1) + 63 of the tile.
constexpr int kTileWaves = 8;

// Element offset of 16-byte chunk c (0..7) of row `row` in a [rows][64] bf16
// stage image.  Rows are 128 bytes, so two rows share one 256-byte window of
// the 64 LDS banks; XOR-ing the chunk with row bits 1..3 gives the 16 rows
// that one ds_read_b128 pass serves (same chunk, consecutive rows) 16 distinct
// 16-byte slots of that window.
RLK_HD int op_off(int row, int c) { return row * 64 + ((c ^ ((row >> 1) & 7)) << 3); }

// Logical tile index -> (n-tile, m-tile): groups of 4 m-tiles sweep the
// n-tiles together, so an n-tile's operand is fetched into an L2 once for 4
// m-tiles while the m-tiles' operand stays resident in L2 / the MALL.
RLK_HD void tile_of_logical(int64_t L, int64_t nnt, int64_t nmt, int64_t *nt, int64_t *mt) {
    constexpr int64_t GR = 4;
    const int64_t group = L / (GR * nnt);
    const int64_t in = L % (GR * nnt);
    const int64_t rows_in_group = min64(GR, nmt - group * GR);
    *mt = group * GR + in % rows_in_group;
    *nt = in / rows_in_group;
}

// Launch index -> logical index for a launch of `count` workgroups.  The
// hardware hands consecutive workgroups to the 8 XCDs in turn; renumbering
// gives each XCD a contiguous run of logical tiles, so the sharing above
// happens inside one XCD's L2.
RLK_HD int64_t xcd_logical(int64_t b, int64_t count) {
    const int64_t full = count / 8 * 8;
    return b < full ? (b % 8) * (count / 8) + b / 8 : b;
}

// Launch index -> (n-tile, m-tile) for a launch over logical tiles [base,
// base + count).
RLK_HD void tile_of(int64_t b, int64_t count, int64_t base, int64_t nnt, int64_t nmt, int64_t *nt, int64_t *mt) {
    tile_of_logical(base + xcd_logical(b, count), nnt, nmt, nt, mt);
}

// ---- tile kernel staging.  Lane i of 1 KB load block blk covers tile row
// 8 blk + i / 8 and LDS slot i % 8 of that row, which holds chunk
// (i % 8) ^ swizzle(row).  Rows past the vocabulary / the batch re-read the
// last valid row (`last`).  Stage `slot` loads hidden step kb + min(slot,
// nks - 1): past the last stage the loads refill a buffer nobody reads.
RLK_HD int stage_last(int64_t tile_rows, int64_t total, int64_t first) {
    return static_cast<int>(min64(tile_rows - 1, total - 1 - first));
}
RLK_HD int stage_row(int blk, int lane) { return blk * 8 + (lane >> 3); }
RLK_HD int stage_chunk(int row, int lane) { return (lane & 7) ^ ((row >> 1) & 7); }
RLK_HD int64_t stage_k0(int kb, int slot, int nks) {
    return static_cast<int64_t>(kb + mini(slot, nks - 1)) * kHiddenStep;
}
// Per-lane byte offset from the stage's wave-uniform base (tile's first row
// + k0); fits 32 bits because hidden <= kMaxHidden.
RLK_HD uint32_t stage_voff(int row, int last, int64_t H, int c) {
    return static_cast<uint32_t>((mini(row, last) * H + c * 8) * 2);
}

// ---- which tile a workgroup of the tile kernel computes.
// Epilogue modes of the tile kernel: the forward's (max, sum) partials; the
// backward's p = exp(inv_T z - lse) per (row, vocab entry) as bf16 into the
// blocked probability buffer; the sampling head's tempered fp32 logits (per-row
// temperature) plus the tile's row maxima; one hidden-dimension part of a
// tail tile (fp32 accumulators for the reduce kernel); the forward over the
// narrow tiles of a last round (TM < 4).
enum : int { kFwd = 0, kBwdProbs = 1, kLogits = 2, kPartialK = 3, kNarrow = 4 };

struct TileCoord {
    int64_t vt;        // partial slot of the tile (its vocab tile for whole tiles)
    int64_t rt;        // row tile
    int64_t v0;        // first vocab entry
    int kb, nks;       // hidden steps [kb, kb + nks)
};

// TM: 32-entry vocab blocks per wave (4: 256 x 256 tiles; 2, 3: the 128-
// and 192-wide narrow tiles).  Narrow tile j covers vocab [narrow_v0 + j 64 TM, + 64 TM)
// for row tile rt; the row tiles of one j are neighbours in launch order.
// Part s of tail tile j covers hidden steps [s n / S, (s + 1) n / S).
RLK_HD TileCoord tile_coord(int mode, int tm, int64_t b, const LogprobArgs &a) {
    TileCoord t;
    t.kb = 0;
    t.nks = a.H / kHiddenStep;
    if (tm != 4) {
        const int64_t L = xcd_logical(b, a.narrow_tiles * a.n_row_tiles);
        const int64_t j = L / a.n_row_tiles;
        t.rt = L % a.n_row_tiles;
        t.vt = a.narrow_slot0 + j;
        t.v0 = a.narrow_v0 + j * 64 * tm;
        return t;
    }
    if (mode == kPartialK) {
        const int64_t j = b / a.splits;
        const int sp = static_cast<int>(b % a.splits);
        tile_of_logical(a.tile_base + j, a.n_vocab_tiles, a.n_row_tiles, &t.vt, &t.rt);
        const int n = t.nks;
        t.kb = sp * n / a.splits;
        t.nks = (sp + 1) * n / a.splits - t.kb;
    } else {
        tile_of(b, a.tile_count, a.tile_base, a.n_vocab_tiles, a.n_row_tiles, &t.vt, &t.rt);
    }
    t.v0 = t.vt * kVocabTile;
    return t;
}

// Element offset, from the tail part buffer, of the 32 x 32 accumulator
// block of vocab half wm, 32-entry vocab block tm and 32-row block rb (token
// rows 32 rb .. 32 rb + 31) of part `part`: 4-float group q of lane `lane`
// in the MFMA's register layout, so each store writes 1 KB contiguously and
// one block's 16 KB are contiguous.
RLK_HD int64_t part_elem(int64_t part, int wm, int rb, int tm, int q, int lane) {
    return part * (kVocabTile * kRowTile) + ((((rb * 2 + wm) * 4 + tm) * 4 + q) * 64 + lane) * 4;
}

// ---- blocked probabilities of the backward: for row tile rt and vocab
// step ks (64 entries) a 256 x 64 block laid out as the stage image op_off.
RLK_HD int64_t probs_block(int64_t rt, int64_t n_vsteps, int64_t ks) { return (rt * n_vsteps + ks) * kStageElems; }
// The tile kernel's epilogue: accumulator (tm, 4-entry group q) of lane half
// h2 at tile row `row`, relative to the block of the wave's vocab half (vocab
// step vt * 4 + wm * 2): one 8-byte store of 4 consecutive vocab entries.
RLK_HD int probs_store_off(int tm, int q, int row, int h2) {
    return (tm >> 1) * kStageElems + op_off(row, (tm & 1) * 4 + q) + 4 * h2;
}

// ---- backward GEMM (S = P W over a vocabulary range).
// W band image: row v (0..63) holds 256 hidden entries as 32 chunks of 8;
// chunk c sits in slot c ^ (4 * (v % 4)).  One transposing read pass (32
// lanes) touches 4 consecutive rows x 4 consecutive chunks (c0 = 0 mod 4);
// the XOR spreads them over the 16 slots of a 256-byte bank window.
RLK_HD int band_off(int v, int c) { return v * 256 + ((c ^ (4 * (v & 3))) << 3); }

// Launch index -> (split, h tile, row tile).  XCD renumbering as in tile_of;
// splits are outermost, so the workgroups of one XCD share a vocabulary
// range, and inside a split 4 row tiles sweep the h tiles together.
RLK_HD void gemm_tile_of(int64_t b, int n_h_tiles, int n_row_tiles, int splits, int *split, int *ht, int *rt) {
    const int64_t per_split = static_cast<int64_t>(n_h_tiles) * n_row_tiles;
    const int64_t L = xcd_logical(b, per_split * splits);
    *split = static_cast<int>(L / per_split);
    int64_t nt, mt;
    tile_of_logical(L % per_split, n_h_tiles, n_row_tiles, &nt, &mt);
    *ht = static_cast<int>(nt);
    *rt = static_cast<int>(mt);
}

// Probability operand: block blk (0..31) of stage `slot` is the 1 KB at this
// element offset from the chunk's blocked buffer, lane i's 16 bytes at byte
// offset 16 i from it (the saddr form: a wave-uniform base plus a fixed
// per-lane offset).
RLK_HD int64_t bwd_a_base(int rt, int n_vsteps, int ks0, int slot, int nks, int blk) {
    return probs_block(rt, n_vsteps, ks0 + mini(slot, nks - 1)) + blk * 512;
}
RLK_HD uint32_t bwd_a_voff(int lane) { return static_cast<uint32_t>(lane) * 16; }

// W operand: block blk holds band rows 2 blk and 2 blk + 1; lane i fills slot
// i % 32 of row 2 blk + i / 32 with chunk slot ^ (4 (row % 4)).  Rows past
// the vocabulary re-read the last row (their probabilities are 0); columns
// past the hidden size re-read the last chunk (never stored).  In the saddr
// form the wave-uniform base is the block's first row, clamped to V - 1, and
// lanes i >= 32 add one row only while that row exists (`pair`, the same for
// the whole wave), which clamps every lane's row to V - 1 exactly as
// min(first row + i / 32, V - 1) would.
RLK_HD int bwd_b_row(int blk, int lane) { return 2 * blk + (lane >> 5); }
RLK_HD int bwd_b_chunk(int row, int lane) { return (lane & 31) ^ (4 * (row & 3)); }
RLK_HD int64_t bwd_b_first(int ks0, int slot, int nks, int blk) {
    return static_cast<int64_t>(ks0 + mini(slot, nks - 1)) * 64 + 2 * blk;
}
RLK_HD int64_t bwd_b_base_row(int64_t first, int V) { return min64(first, static_cast<int64_t>(V - 1)); }
RLK_HD bool bwd_b_pair(int64_t first, int V) { return first + 1 <= static_cast<int64_t>(V - 1); }
RLK_HD uint32_t bwd_b_voff(int lane, bool pair, int c, int clast, int64_t H) {
    return static_cast<uint32_t>(((pair ? (lane >> 5) : 0) * H + 8 * mini(c, clast)) * 2);
}
RLK_HD int bwd_clast(int H, int h0) { return mini(256, H - h0) / 8 - 1; }

// Output of (split, row tile rt, h tile at h0) in the [splits, rows_pad, H]
// partial sums (or dh itself when unsplit): the tile's base element, and the
// offset of (tile row, tile column h) from it.
RLK_HD int64_t bwd_out_base(int split, int64_t rows_pad, int rt, int64_t H, int h0) {
    return (split * rows_pad + static_cast<int64_t>(rt) * 256) * H + h0;
}
RLK_HD int64_t bwd_out_off(int row, int64_t H, int h) { return static_cast<int64_t>(row) * H + h; }
// The finish kernel's view of split sp's partial sums at (row r, column h).
RLK_HD int64_t bwd_part_elem(int sp, int64_t rows_pad, int64_t r, int64_t H, int h) { return (sp * rows_pad + r) * H + h; }

// ---- launch shapes (host), shared by the launchers and the replay.
// Weight-ring depth of the tile kernels: with few row tiles the hidden rows
// stay in L2 and a third weight stage gives the streaming weights two stages
// to arrive (the whole 160 KB of LDS); with many row tiles two stages measure
// better.
inline int tile_weight_stages(int64_t n_row_tiles) { return n_row_tiles <= 8 ? 3 : 2; }
// Hidden-row stages of the tile kernel with TM 32-entry vocab blocks per
// wave: 2, or 3 for the 128-wide narrow tiles, whose short stages would not
// cover the hidden rows' latency with one stage to arrive (and whose LDS has
// room: 3 x 16 KB of weights + 3 x 32 KB of hidden rows).
constexpr int tile_hidden_stages(int tm) { return tm == 2 ? 3 : 2; }
inline int64_t bwd_gemm_blocks(const LogprobBwdArgs &a) {
    return static_cast<int64_t>(a.n_row_tiles) * a.n_h_tiles * a.splits;
}
constexpr int kBwdFinishThreads = 256;
// Wave64s per backward GEMM workgroup: wave w owns tile rows 128 (w & 1) ..
// +127 and hidden entries 64 (w >> 1) .. +63 of its 256 x 256 output tile.
constexpr int kBwdGemmWaves = 8;
inline int64_t bwd_finish_blocks(const LogprobBwdArgs &a) {
    return (a.rows * (a.H / 4) + kBwdFinishThreads - 1) / kBwdFinishThreads;
}
// The combine kernel a forward of R rows uses: one workgroup per row up to
// 4096 rows, one wave per row below 32768, one thread per row beyond.
enum : int { kCombineBlock = 0, kCombineWave = 1, kCombineRow = 2 };
inline int logprob_combine_kind(int64_t R) { return R <= 4096 ? kCombineBlock : R < 32768 ? kCombineWave : kCombineRow; }

}  // namespace rlk
