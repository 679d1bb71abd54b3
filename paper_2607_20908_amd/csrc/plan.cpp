// Host-side validation and split-K planning (no HIP calls).
//
// Decode attention is split into work items, each covering one chunk of KV
// tokens of one unit at one kv head:
//   prefix unit (p, kh): the prompt's shared KV, serving all G*r query rows of
//                        the group (r = Hq/Hkv), so the chunk is read once for
//                        the whole group of candidates;
//   suffix unit (s, kh): candidate s's own KV, serving its r query rows.
// Each item leaves an online-softmax partial (max, sum, weighted value sum)
// per query row; the combine kernel merges the partials of a sequence.
#include "plan.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>

namespace rlk {

namespace {

rl_status fail(std::string *err, rl_status st, const std::string &msg) {
    if (err) *err = msg;
    return st;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t round_up16(int64_t x) { return (x + 15) / 16 * 16; }

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

rl_status plan_decode(const rl_decode_shape *shape, const rl_decode_lens *lens,
                      DecodePlan *plan, std::string *err) {
    if (!shape) return fail(err, RL_ERR_NULL_POINTER, "shape is NULL");
    if (!lens) return fail(err, RL_ERR_NULL_POINTER, "lens is NULL");
    const rl_decode_shape &sh = *shape;
    if (sh.num_prompts < 0) return fail(err, RL_ERR_INVALID_SHAPE, "num_prompts < 0");
    if (sh.group_size < 1) return fail(err, RL_ERR_INVALID_SHAPE, "group_size < 1");
    if (sh.num_q_heads < 1 || sh.num_kv_heads < 1)
        return fail(err, RL_ERR_INVALID_SHAPE, "head counts must be >= 1");
    if (sh.num_q_heads % sh.num_kv_heads)
        return fail(err, RL_ERR_INVALID_SHAPE, "num_q_heads must be a multiple of num_kv_heads");
    if (!(std::isfinite(sh.softmax_scale) && sh.softmax_scale > 0.f))
        return fail(err, RL_ERR_INVALID_SHAPE, "softmax_scale must be finite and > 0");
    if (sh.split_tokens < 0 || (sh.split_tokens > 0 && (sh.split_tokens < 16 || sh.split_tokens % 16)))
        return fail(err, RL_ERR_INVALID_SHAPE, "split_tokens must be 0 or a positive multiple of 16");
    if (sh.head_dim <= 0) return fail(err, RL_ERR_INVALID_SHAPE, "head_dim must be > 0");
    if (sh.head_dim != 64 && sh.head_dim != 128)
        return fail(err, RL_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
    if (lens->prefix_rows < 0 || lens->suffix_rows < 0)
        return fail(err, RL_ERR_INVALID_SHAPE, "row counts must be >= 0");

    DecodePlan &pl = *plan;
    pl = DecodePlan{};
    pl.P = sh.num_prompts;
    pl.G = sh.group_size;
    pl.Hq = sh.num_q_heads;
    pl.Hkv = sh.num_kv_heads;
    pl.D = sh.head_dim;
    pl.r = sh.num_q_heads / sh.num_kv_heads;
    pl.scale = sh.softmax_scale;
    const int64_t P = pl.P, G = pl.G, S = P * G, Hkv = pl.Hkv, r = pl.r;
    if (S > INT32_MAX / 2 || S * pl.Hq > INT32_MAX)
        return fail(err, RL_ERR_UNSUPPORTED, "too many sequences x heads");
    if (S == 0) return RL_OK;   // valid no-op

    if (!lens->prefix_start || !lens->prefix_len || !lens->suffix_start || !lens->suffix_len)
        return fail(err, RL_ERR_NULL_POINTER, "length arrays must not be NULL when P*G > 0");
    int64_t sum_lp = 0, sum_ls = 0;
    for (int64_t p = 0; p < P; ++p) {
        const int64_t st = lens->prefix_start[p], n = lens->prefix_len[p];
        if (n < 0) return fail(err, RL_ERR_INVALID_SHAPE, "prefix_len[" + std::to_string(p) + "] < 0");
        if (n > 0 && (st < 0 || st > lens->prefix_rows - n))
            return fail(err, RL_ERR_INVALID_SHAPE,
                        "prefix range of prompt " + std::to_string(p) + " exceeds prefix_rows");
        sum_lp += n;
    }
    for (int64_t s = 0; s < S; ++s) {
        const int64_t st = lens->suffix_start[s], n = lens->suffix_len[s];
        if (n < 0) return fail(err, RL_ERR_INVALID_SHAPE, "suffix_len[" + std::to_string(s) + "] < 0");
        if (n > 0 && (st < 0 || st > lens->suffix_rows - n))
            return fail(err, RL_ERR_INVALID_SHAPE,
                        "suffix range of candidate " + std::to_string(s) + " exceeds suffix_rows");
        sum_ls += n;
    }

    // --- split sizes --------------------------------------------------------
    const int64_t Mp = G * r;                       // query rows per prefix unit
    const int64_t ncg = ceil_div(Mp, kMaxItemRows); // column groups per prefix chunk
    if (r > kMaxItemRows) return fail(err, RL_ERR_UNSUPPORTED, "Hq/Hkv must be <= 128");
    int64_t cs, cp;
    if (sh.split_tokens > 0) {
        cs = cp = sh.split_tokens;
    } else {
        // Aim for ~8 items per compute unit so the hardware dispatcher balances
        // skewed lengths; prefix chunks are at least 32 tokens per query row so
        // their partials cost a few percent of the KV bytes they summarise.
        const int64_t work = Hkv * (sum_lp * ncg + sum_ls);
        const int64_t target = 8 * kNumCUs;
        cs = std::min<int64_t>(4096, std::max<int64_t>(128, round_up16(ceil_div(work, target))));
        cp = std::max<int64_t>(cs, round_up16(32 * std::min<int64_t>(Mp, kMaxItemRows)));
        cp = std::min<int64_t>(cp, 16384);
    }
    pl.split_prefix = static_cast<int32_t>(cp);
    pl.split_suffix = static_cast<int32_t>(cs);

    // --- items in creation order, partial rows in unit order ---------------
    std::vector<rl_plan_item> items;
    std::vector<int64_t> item_prow;
    pl.prefix_units.assign(P * Hkv, DevUnit{0, 0, 0});
    pl.suffix_units.assign(S * Hkv, DevUnit{0, 0, 0});
    int64_t prow = 0;
    auto add_unit = [&](int32_t kind, int32_t unit, int32_t kh, int64_t L, int64_t C,
                        int64_t M, DevUnit *du) {
        du->base = prow;
        if (L == 0) { du->nchunks = 0; return; }
        const int64_t n = ceil_div(L, C);
        const int64_t b = round_up16(ceil_div(L, n));
        du->nchunks = static_cast<int32_t>(n);
        for (int64_t c = 0; c < n; ++c) {
            const int64_t beg = c * b, cnt = std::min(b, L - beg);
            for (int64_t rb = 0; rb < M; rb += kMaxItemRows) {
                rl_plan_item it{};
                it.kind = kind;
                it.unit = unit;
                it.kv_head = kh;
                it.chunk = static_cast<int32_t>(c);
                it.tok_begin = beg;
                it.tok_count = static_cast<int32_t>(cnt);
                it.row_begin = static_cast<int32_t>(rb);
                it.row_count = static_cast<int32_t>(std::min<int64_t>(kMaxItemRows, M - rb));
                items.push_back(it);
                item_prow.push_back(prow + c * M + rb);
            }
        }
        prow += n * M;
    };
    for (int64_t p = 0; p < P; ++p)
        for (int64_t kh = 0; kh < Hkv; ++kh)
            add_unit(0, (int32_t)p, (int32_t)kh, lens->prefix_len[p], cp, Mp,
                     &pl.prefix_units[p * Hkv + kh]);
    for (int64_t s = 0; s < S; ++s)
        for (int64_t kh = 0; kh < Hkv; ++kh)
            add_unit(1, (int32_t)s, (int32_t)kh, lens->suffix_len[s], cs, r,
                     &pl.suffix_units[s * Hkv + kh]);
    pl.partial_rows = prow;

    // --- launch order: longest work first (stable) -------------------------
    const int64_t kv_bytes_per_tok = 4LL * pl.D;              // K + V, bf16
    const int64_t partial_bytes_per_row = 2LL * (8 + 4LL * pl.D);  // written, then read
    std::vector<int64_t> cost(items.size());
    for (size_t i = 0; i < items.size(); ++i)
        cost[i] = items[i].tok_count * kv_bytes_per_tok + items[i].row_count * partial_bytes_per_row;
    std::vector<size_t> order(items.size());
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](size_t a, size_t b) { return cost[a] > cost[b]; });
    pl.items.reserve(items.size());
    pl.dev_items.reserve(items.size());
    for (size_t i : order) {
        const rl_plan_item &it = items[i];
        pl.items.push_back(it);
        DevItem d{};
        const int64_t start = it.kind == 0 ? lens->prefix_start[it.unit] : lens->suffix_start[it.unit];
        d.kv_row0 = start + it.tok_begin;
        d.partial_row0 = item_prow[i];
        d.ntok = it.tok_count;
        d.kind_kh = it.kv_head | (it.kind << 16);
        d.unit = it.unit;
        d.row_begin = it.row_begin;
        pl.dev_items.push_back(d);
    }
    if (pl.dev_items.size() > static_cast<size_t>(INT32_MAX))
        return fail(err, RL_ERR_UNSUPPORTED, "too many work items");

    // --- workspace layout --------------------------------------------------
    size_t off = 0;
    pl.off_items = off;
    off = align_up(off + pl.dev_items.size() * sizeof(DevItem), 256);
    pl.off_prefix_units = off;
    off = align_up(off + pl.prefix_units.size() * sizeof(DevUnit), 256);
    pl.off_suffix_units = off;
    off = align_up(off + pl.suffix_units.size() * sizeof(DevUnit), 256);
    pl.meta_bytes = off;
    pl.off_m = off;
    off = align_up(off + static_cast<size_t>(prow) * 4, 256);
    pl.off_l = off;
    off = align_up(off + static_cast<size_t>(prow) * 4, 256);
    pl.off_acc = off;
    off = align_up(off + static_cast<size_t>(prow) * pl.D * 4, 256);
    pl.total_bytes = off;
    return RL_OK;
}

rl_status check_decode_ptrs(const DecodePlan &pl, const rl_decode_lens *lens,
                            const rl_decode_ptrs *ptrs, std::string *err) {
    if (!ptrs) return fail(err, RL_ERR_NULL_POINTER, "ptrs is NULL");
    const int64_t S = (int64_t)pl.P * pl.G;
    if (S == 0) return RL_OK;
    if (!ptrs->q) return fail(err, RL_ERR_NULL_POINTER, "q is NULL");
    if (!ptrs->out) return fail(err, RL_ERR_NULL_POINTER, "out is NULL");
    bool any_prefix = false, any_suffix = false;
    for (int64_t p = 0; p < pl.P; ++p) any_prefix |= lens->prefix_len[p] > 0;
    for (int64_t s = 0; s < S; ++s) any_suffix |= lens->suffix_len[s] > 0;
    if (any_prefix && (!ptrs->k_prefix || !ptrs->v_prefix))
        return fail(err, RL_ERR_NULL_POINTER, "k_prefix/v_prefix is NULL");
    if (any_suffix && (!ptrs->k_suffix || !ptrs->v_suffix))
        return fail(err, RL_ERR_NULL_POINTER, "k_suffix/v_suffix is NULL");
    const void *a16[] = {ptrs->q, ptrs->k_prefix, ptrs->v_prefix, ptrs->k_suffix, ptrs->v_suffix, ptrs->out};
    const char *names[] = {"q", "k_prefix", "v_prefix", "k_suffix", "v_suffix", "out"};
    for (int i = 0; i < 6; ++i)
        if (a16[i] && !aligned(a16[i], 16))
            return fail(err, RL_ERR_MISALIGNED, std::string(names[i]) + " is not 16-byte aligned");
    if (ptrs->lse && !aligned(ptrs->lse, 4))
        return fail(err, RL_ERR_MISALIGNED, "lse is not 4-byte aligned");
    return RL_OK;
}

rl_status plan_logprob(int64_t rows, int32_t hidden, int32_t vocab, LogprobPlan *plan,
                       std::string *err) {
    if (rows < 0) return fail(err, RL_ERR_INVALID_SHAPE, "rows < 0");
    if (hidden <= 0) return fail(err, RL_ERR_INVALID_SHAPE, "hidden must be > 0");
    if (vocab <= 0) return fail(err, RL_ERR_INVALID_SHAPE, "vocab must be > 0");
    if (hidden % kHiddenStep)
        return fail(err, RL_ERR_UNSUPPORTED, "hidden must be a multiple of 64");
    LogprobPlan &pl = *plan;
    pl = LogprobPlan{};
    pl.R = rows;
    pl.H = hidden;
    pl.V = vocab;
    pl.n_vocab_tiles = ceil_div(vocab, kVocabTile);
    pl.n_row_tiles = ceil_div(rows, kRowTile);
    if (pl.n_vocab_tiles * pl.n_row_tiles > INT32_MAX)
        return fail(err, RL_ERR_UNSUPPORTED, "too many rows x vocab tiles");
    if (rows == 0) return RL_OK;
    size_t off = 0;
    pl.off_m = off;
    off = align_up(off + static_cast<size_t>(pl.n_vocab_tiles) * rows * 4, 256);
    pl.off_l = off;
    off = align_up(off + static_cast<size_t>(pl.n_vocab_tiles) * rows * 4, 256);
    pl.off_zt = off;
    off = align_up(off + static_cast<size_t>(rows) * 4, 256);
    pl.total_bytes = off;
    return RL_OK;
}

rl_status check_logprob_args(const LogprobPlan &pl, const void *hidden_states,
                             const void *w_lm, const int32_t *target, float inv_temperature,
                             const float *logprob, const float *lse, std::string *err) {
    if (!(std::isfinite(inv_temperature) && inv_temperature > 0.f))
        return fail(err, RL_ERR_INVALID_SHAPE, "inv_temperature must be finite and > 0");
    if (pl.R == 0) return RL_OK;
    if (!hidden_states) return fail(err, RL_ERR_NULL_POINTER, "hidden_states is NULL");
    if (!w_lm) return fail(err, RL_ERR_NULL_POINTER, "w_lm is NULL");
    if (!target) return fail(err, RL_ERR_NULL_POINTER, "target is NULL");
    if (!logprob) return fail(err, RL_ERR_NULL_POINTER, "logprob is NULL");
    if (!aligned(hidden_states, 16)) return fail(err, RL_ERR_MISALIGNED, "hidden_states is not 16-byte aligned");
    if (!aligned(w_lm, 16)) return fail(err, RL_ERR_MISALIGNED, "w_lm is not 16-byte aligned");
    if (!aligned(target, 4)) return fail(err, RL_ERR_MISALIGNED, "target is not 4-byte aligned");
    if (!aligned(logprob, 4)) return fail(err, RL_ERR_MISALIGNED, "logprob is not 4-byte aligned");
    if (lse && !aligned(lse, 4)) return fail(err, RL_ERR_MISALIGNED, "lse is not 4-byte aligned");
    return RL_OK;
}

}  // namespace rlk
