// Host-side argument validation and planning for rl_decode_attn,
// rl_extend_attn and rl_token_logprob.  Plain C++17: no HIP calls, so every check here can be
// exercised on a machine without a GPU.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "rl_kernels.h"

namespace rlk {

// Largest number of query rows one decode work item serves (16 per MFMA column
// tile, one column tile per wave, 4 waves).
constexpr int kMaxItemRows = 64;
// Largest Hq / Hkv the decode path accepts.
constexpr int kMaxHeadsPerKv = 128;
// KV tokens staged per LDS tile in the split kernel.
constexpr int kTileTokens = 64;
// Vocabulary entries per lm-head work tile.
constexpr int kVocabTile = 256;
// Token rows per lm-head work tile.
constexpr int kRowTile = 256;
// Hidden-dimension step of the lm-head kernel.
constexpr int kHiddenStep = 64;
// Compute units of an MI355X; the automatic split size is planned for them.
constexpr int kNumCUs = 256;
// XCDs: the hardware deals consecutive workgroups of a launch to them in turn.
constexpr int kNumXcds = 8;
constexpr float kLog2eHost = 1.4426950408889634f;

// One split-K work item as the split kernel reads it (16 bytes; the work list
// is uploaded over PCIe on every call, so it is kept small).
struct DevItem {
    uint32_t kv_row0;       // KV row of the chunk's first token in its buffer
    uint32_t partial_row0;  // partial row of the item's first query row
    int32_t unit;           // prompt p (prefix) or candidate s (suffix)
    uint32_t meta;          // tokens (bits 0-14, >= 1) | suffix (bit 15) | kv head (bits 16-23)
                            // | first query row / kMaxItemRows (bits 24-31)
};
static_assert(sizeof(DevItem) == 16, "DevItem layout");

// Where the partial results of one unit (prompt or candidate) live: at kv
// head kh, chunk c's row i is partial row base + (kh * nchunks + c) *
// rows_per_chunk + i.
struct DevUnit {
    uint32_t base;
    uint32_t nchunks;
};
static_assert(sizeof(DevUnit) == 8, "DevUnit layout");

// Limits of that encoding: tokens per item, kv heads, query rows per prefix
// unit (G * Hq / Hkv, 256 blocks of kMaxItemRows), and KV or partial rows.
constexpr int64_t kMaxItemTokens = 16384;
constexpr int64_t kMaxDecodeKvHeads = 256;
constexpr int64_t kMaxUnitRows = 16384;
constexpr int64_t kMaxDecodeRows = 0xffffffffLL;

// How much of the plan to build: the workspace size needs only the counts;
// a launch needs the device work list; the debug export also wants the
// rl_plan_item view of it.
enum class PlanDetail { kSizes, kDevice, kDebug };

struct DecodePlan {
    // problem
    int32_t P = 0, G = 0, Hq = 0, Hkv = 0, D = 0, r = 0;
    float scale = 0.f;
    int32_t kv_layout = RL_KV_TOKEN_MAJOR;
    int64_t prefix_rows = 0, suffix_rows = 0;
    int32_t split_prefix = 0, split_suffix = 0;  // chunk sizes used
    // work list in launch order (items: kDebug only; dev_items: kDevice and up)
    int64_t n_items = 0;
    std::vector<rl_plan_item> items;
    std::vector<DevItem> dev_items;
    std::vector<DevUnit> prefix_units;   // [P]
    std::vector<DevUnit> suffix_units;   // [S]
    int64_t partial_rows = 0;
    // nonzero when items of more than 48 query rows (four sub-tiles per wave)
    // hold most of the KV tokens: the split kernel then keeps two tiles in
    // flight per workgroup
    int32_t deep_prefetch = 0;
    // workspace layout (byte offsets; every section 256-byte aligned)
    size_t off_items = 0, off_prefix_units = 0, off_suffix_units = 0;
    size_t off_m = 0, off_l = 0, off_acc = 0;
    size_t meta_bytes = 0;   // items + unit tables (uploaded from the host)
    size_t total_bytes = 0;
    // scratch reused across calls when the same plan object is planned again
    std::vector<DevItem> tmp_items;
    std::vector<uint64_t> tmp_keys, tmp_keys2;
};

// Validates shape and lengths (not device pointers) and builds the plan to the
// requested detail.  The plan object's vectors keep their capacity between
// calls, so a caller that reuses one object plans without allocating.
// On failure returns the status and sets *err.
rl_status plan_decode(const rl_decode_shape *shape, const rl_decode_lens *lens,
                      DecodePlan *plan, std::string *err, PlanDetail detail = PlanDetail::kDevice);

// Validates the device pointers of a decode call against a built plan.
rl_status check_decode_ptrs(const DecodePlan &plan, const rl_decode_lens *lens,
                            const rl_decode_ptrs *ptrs, std::string *err);

// A last round of lm-head tiles that would leave at least half the CUs idle
// is split over the hidden dimension into up to this many parts.
constexpr int kMaxTailSplits = 4;

// One pass of `tiles` 256 x 256 lm-head tiles over `nks` hidden steps: the
// whole rounds over the CUs run as they are (logical tiles [0, dp_tiles)).
// A last round that would leave at least half of the CUs idle runs as
// `splits` hidden-dimension parts per tile instead, as many as fit one round
// (up to kMaxTailSplits, at least 4 hidden steps per part), so that it takes
// a fraction of a tile's time; tail_tiles = 0 when the last round runs whole.
struct TailSplit {
    int64_t dp_tiles = 0, tail_tiles = 0;
    int32_t splits = 1;
};
TailSplit plan_tail_split(int64_t tiles, int64_t nks);
// The tile kernels address a weight or hidden row of a tile as a 32-bit byte
// offset from the tile's first row (255 rows of 2 * hidden bytes).
constexpr int64_t kMaxHidden = 1 << 22;
// Narrow last-round tiles are 64 narrow_tm vocab entries wide, narrow_tm 2
// or 3 (the narrower that fits one round); they need every row tile of a
// vocab tile next to each other in launch order, which holds for at most
// kNarrowMaxRowTiles row tiles.
constexpr int kNarrowMinTM = 2, kNarrowMaxTM = 3;
constexpr int64_t kNarrowMaxRowTiles = 4;

struct LogprobPlan {
    int64_t R = 0;
    int32_t H = 0, V = 0;
    int64_t n_vocab_tiles = 0, n_row_tiles = 0;
    // tiles [0, n_dp_tiles) run whole; the n_tail_tiles after them run as
    // tail_splits hidden-dimension parts whose fp32 accumulators (one
    // 256 x 256 tile each, at off_part) a reduce kernel sums
    int64_t n_dp_tiles = 0, n_tail_tiles = 0;
    int32_t tail_splits = 1;
    // or: a last round more than half full runs as narrow_tiles tiles of
    // 64 narrow_tm vocab entries over [narrow_v0, V) (per row tile), their
    // partials in slots narrow_slot0.. after the whole tiles' slots
    int64_t narrow_v0 = 0, narrow_tiles = 0, narrow_slot0 = 0;
    int32_t narrow_tm = 0;
    int64_t n_partials = 0;          // (max, sum) partial slots per row
    size_t off_m = 0, off_l = 0, off_zt = 0, off_part = 0, total_bytes = 0;
};

rl_status plan_logprob(int64_t rows, int32_t hidden, int32_t vocab, LogprobPlan *plan,
                       std::string *err);

// The tiles of one lm-head pass over `rows` rows: logical tiles [0,
// dp_tiles) whole, then (when narrow_tiles > 0) the vocabulary from
// narrow_v0 on as one round of tiles 64 narrow_tm entries wide per row tile,
// with partial slots narrow_slot0.. ; n_partials slots per row in all.
// Narrow tiles are taken when the tiles leave a partial last round, there
// are at most kNarrowMaxRowTiles row tiles and the narrow tiles fit in one
// round; of the widths that fit, the narrowest (the most CUs busy).
struct TileRounds {
    int64_t dp_tiles = 0, narrow_v0 = 0, narrow_tiles = 0, narrow_slot0 = 0, n_partials = 0;
    int32_t narrow_tm = 0;
};
TileRounds plan_tile_rounds(int64_t rows, int32_t vocab);

rl_status check_logprob_args(const LogprobPlan &plan, const void *hidden_states,
                             const void *w_lm, const int32_t *target, float inv_temperature,
                             const float *logprob, const float *lse, std::string *err);

// Backward of the token log-prob: rows are processed in chunks whose bf16
// probabilities (chunk rows x padded vocabulary) live in the workspace,
// followed by the split partial sums when the GEMM is split over the
// vocabulary.
constexpr int64_t kBwdChunkRows = 16384;

struct LogprobBwdPlan {
    int64_t R = 0;
    int32_t H = 0, V = 0;
    int64_t chunk_rows = 0;          // rows per chunk (the last may have fewer)
    int64_t n_chunks = 0;
    int64_t n_vocab_tiles = 0;       // 256-entry vocab tiles
    int32_t n_vsteps = 0;            // 64-entry vocab steps = 4 * n_vocab_tiles
    int32_t chunk_row_tiles = 0;     // 256-row tiles of a full chunk
    int32_t n_h_tiles = 0;           // 256-entry hidden tiles
    int32_t splits = 1, steps_per_split = 0;
    // [off_part, total_bytes) holds, one after the other within a chunk, the
    // hidden-dimension parts of the probability pass's tail tiles (summed
    // before the GEMM starts) and the GEMM's split partial sums
    size_t off_probs = 0, off_part = 0, total_bytes = 0;
};

// The probability pass of the backward chunk of `n` rows: its tail split.
TailSplit bwd_probs_tail(const LogprobBwdPlan &plan, int64_t n);

rl_status plan_logprob_bwd(int64_t rows, int32_t hidden, int32_t vocab, LogprobBwdPlan *plan,
                           std::string *err);

// Nucleus sampling: the tempered fp32 logits of a chunk of rows and their
// per-tile maxima live in the workspace.
constexpr int64_t kSampleChunkRows = 8192;
constexpr int32_t kSampleMaxVocab = 1 << 21;

struct SamplePlan {
    int64_t R = 0;
    int32_t H = 0, V = 0;
    int64_t chunk_rows = 0;
    int64_t n_vocab_tiles = 0;
    int64_t pm_slots = 0;            // row-maximum slots per row (whole and narrow tiles)
    int64_t ld = 0;                  // row stride of the logits: the vocab tiles plus one tile of padding
    size_t off_logits = 0, off_pm = 0, total_bytes = 0;
};

rl_status plan_sample(int64_t rows, int32_t hidden, int32_t vocab, SamplePlan *plan, std::string *err);

// Extend attention: one block of at most kExtBlockRows query rows (new token x
// query head of one candidate at one kv head) per workgroup.
constexpr int kExtBlockRows = 256;

struct ExtItem {
    int64_t prefix_row0;   // first prefix row of the prompt (0 when Lp = 0)
    int64_t suffix_row0;   // first suffix row of the candidate
    int64_t q_row0;        // query / output row of the candidate's first new token
    int32_t Lp, Ls, n;     // prefix length, suffix length (new tokens included), new tokens
    int32_t kh;            // kv head
    int32_t row_begin;     // first unit row of the block (unit row = token * r + head in group)
    int32_t pad;
};
static_assert(sizeof(ExtItem) == 48, "ExtItem layout");

struct ExtendPlan {
    int32_t P = 0, G = 0, Hq = 0, Hkv = 0, D = 0, r = 0;
    float scale = 0.f;
    int32_t kv_layout = RL_KV_TOKEN_MAJOR;
    int64_t prefix_rows = 0, suffix_rows = 0, q_rows = 0;
    int64_t n_items = 0;
    bool any_prefix = false;           // some block reads prefix rows
    double ctx_tokens = 0;             // sum over query rows of visible tokens (flop count / 4D)
    std::vector<ExtItem> items;        // launch order (built when requested)
    size_t total_bytes = 0;            // workspace: the work list
    // scratch kept between calls
    std::vector<std::pair<int64_t, int64_t>> tmp_ranges;
    std::vector<std::pair<int64_t, int64_t>> tmp_units;
    std::vector<ExtItem> tmp_items;
};

// Validates an extend call (shape, lengths, query ranges; not device pointers)
// and, with build = true, lays out the work list: the blocks of one (prompt,
// kv head) are consecutive, units with more work first, and inside a unit the
// blocks with the longest visible context first.
rl_status plan_extend(const rl_decode_shape *shape, const rl_extend_lens *lens, ExtendPlan *plan,
                      std::string *err, bool build);

rl_status check_extend_ptrs(const ExtendPlan &plan, const rl_decode_ptrs *ptrs, std::string *err);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace rlk
