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

// Clears a plan but keeps the capacity of its vectors.
void reset(DecodePlan *pl) {
    std::vector<rl_plan_item> items = std::move(pl->items);
    std::vector<DevItem> dev = std::move(pl->dev_items), tmp = std::move(pl->tmp_items);
    std::vector<DevUnit> pu = std::move(pl->prefix_units), su = std::move(pl->suffix_units);
    std::vector<uint64_t> k1 = std::move(pl->tmp_keys), k2 = std::move(pl->tmp_keys2);
    *pl = DecodePlan{};
    items.clear(); dev.clear(); tmp.clear(); pu.clear(); su.clear(); k1.clear(); k2.clear();
    pl->items = std::move(items);
    pl->dev_items = std::move(dev);
    pl->tmp_items = std::move(tmp);
    pl->prefix_units = std::move(pu);
    pl->suffix_units = std::move(su);
    pl->tmp_keys = std::move(k1);
    pl->tmp_keys2 = std::move(k2);
}

// The checks of a decode shape that every attention entry point shares.
rl_status check_shape(const rl_decode_shape &sh, std::string *err) {
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
    if (sh.kv_layout != RL_KV_TOKEN_MAJOR && sh.kv_layout != RL_KV_HEAD_MAJOR)
        return fail(err, RL_ERR_INVALID_SHAPE, "kv_layout must be RL_KV_TOKEN_MAJOR or RL_KV_HEAD_MAJOR");
    if (sh.head_dim <= 0) return fail(err, RL_ERR_INVALID_SHAPE, "head_dim must be > 0");
    if (sh.head_dim != 64 && sh.head_dim != 128)
        return fail(err, RL_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
    return RL_OK;
}

// Prefix ranges of P prompts and suffix ranges of S candidates inside the
// allocated rows.
rl_status check_ranges(int64_t P, int64_t S, const int64_t *prefix_start, const int32_t *prefix_len,
                       int64_t prefix_rows, const int64_t *suffix_start, const int32_t *suffix_len,
                       int64_t suffix_rows, int64_t *sum_lp, int64_t *sum_ls, std::string *err) {
    *sum_lp = *sum_ls = 0;
    for (int64_t p = 0; p < P; ++p) {
        const int64_t st = prefix_start[p], n = prefix_len[p];
        if (n < 0) return fail(err, RL_ERR_INVALID_SHAPE, "prefix_len[" + std::to_string(p) + "] < 0");
        if (n > 0 && (st < 0 || st > prefix_rows - n))
            return fail(err, RL_ERR_INVALID_SHAPE,
                        "prefix range of prompt " + std::to_string(p) + " exceeds prefix_rows");
        *sum_lp += n;
    }
    for (int64_t s = 0; s < S; ++s) {
        const int64_t st = suffix_start[s], n = suffix_len[s];
        if (n < 0) return fail(err, RL_ERR_INVALID_SHAPE, "suffix_len[" + std::to_string(s) + "] < 0");
        if (n > 0 && (st < 0 || st > suffix_rows - n))
            return fail(err, RL_ERR_INVALID_SHAPE,
                        "suffix range of candidate " + std::to_string(s) + " exceeds suffix_rows");
        *sum_ls += n;
    }
    return RL_OK;
}

}  // namespace

rl_status plan_decode(const rl_decode_shape *shape, const rl_decode_lens *lens,
                      DecodePlan *plan, std::string *err, PlanDetail detail) {
    if (!shape) return fail(err, RL_ERR_NULL_POINTER, "shape is NULL");
    if (!lens) return fail(err, RL_ERR_NULL_POINTER, "lens is NULL");
    const rl_decode_shape &sh = *shape;
    rl_status st0 = check_shape(sh, err);
    if (st0 != RL_OK) return st0;
    if (lens->prefix_rows < 0 || lens->suffix_rows < 0)
        return fail(err, RL_ERR_INVALID_SHAPE, "row counts must be >= 0");

    DecodePlan &pl = *plan;
    reset(&pl);
    pl.P = sh.num_prompts;
    pl.G = sh.group_size;
    pl.Hq = sh.num_q_heads;
    pl.Hkv = sh.num_kv_heads;
    pl.D = sh.head_dim;
    pl.r = sh.num_q_heads / sh.num_kv_heads;
    pl.scale = sh.softmax_scale;
    pl.kv_layout = sh.kv_layout;
    pl.prefix_rows = lens->prefix_rows;
    pl.suffix_rows = lens->suffix_rows;
    const int64_t P = pl.P, G = pl.G, S = P * G, Hkv = pl.Hkv, r = pl.r;
    if (S > INT32_MAX / 2 || S * pl.Hq > INT32_MAX)
        return fail(err, RL_ERR_UNSUPPORTED, "too many sequences x heads");
    if (S == 0) return RL_OK;   // valid no-op

    if (!lens->prefix_start || !lens->prefix_len || !lens->suffix_start || !lens->suffix_len)
        return fail(err, RL_ERR_NULL_POINTER, "length arrays must not be NULL when P*G > 0");
    int64_t sum_lp = 0, sum_ls = 0;
    st0 = check_ranges(P, S, lens->prefix_start, lens->prefix_len, lens->prefix_rows, lens->suffix_start,
                       lens->suffix_len, lens->suffix_rows, &sum_lp, &sum_ls, err);
    if (st0 != RL_OK) return st0;

    // --- split sizes --------------------------------------------------------
    const int64_t Mp = G * r;                       // query rows per prefix unit
    const int64_t ncg = ceil_div(Mp, kMaxItemRows); // column groups per prefix chunk
    if (r > kMaxHeadsPerKv) return fail(err, RL_ERR_UNSUPPORTED, "Hq/Hkv must be <= 128");
    if (Hkv > kMaxDecodeKvHeads) return fail(err, RL_ERR_UNSUPPORTED, "num_kv_heads must be <= 256");
    if (Mp > kMaxUnitRows) return fail(err, RL_ERR_UNSUPPORTED, "group_size * Hq/Hkv must be <= 16384");
    if (lens->prefix_rows > kMaxDecodeRows || lens->suffix_rows > kMaxDecodeRows)
        return fail(err, RL_ERR_UNSUPPORTED, "prefix_rows and suffix_rows must be < 2^32");
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
    // a forced split above the item limit covers fewer tokens per item,
    // which the split bound allows
    cp = std::min<int64_t>(cp, kMaxItemTokens);
    cs = std::min<int64_t>(cs, kMaxItemTokens);
    pl.split_prefix = static_cast<int32_t>(cp);
    pl.split_suffix = static_cast<int32_t>(cs);

    // --- unit tables; partial rows in unit order ------------------------------
    // A unit of L tokens splits into n = ceil(L / C) chunks of b = ceil(L / n)
    // tokens rounded up to 16 (the last one shorter), each chunk into
    // ceil(M / kMaxItemRows) items of at most kMaxItemRows query rows.
    // The kv heads of a unit follow each other, so one table entry per unit
    // serves them all.
    pl.prefix_units.assign(P, DevUnit{0, 0});
    pl.suffix_units.assign(S, DevUnit{0, 0});
    int64_t prow = 0, n_items = 0, item_tokens = 0, wide_tokens = 0;
    auto size_unit = [&](int64_t L, int64_t C, int64_t M, DevUnit *du) {
        const int64_t n = L == 0 ? 0 : ceil_div(L, C);
        item_tokens += L * ceil_div(M, kMaxItemRows);
        wide_tokens += L * (M / kMaxItemRows + (M % kMaxItemRows > 48 ? 1 : 0));
        du->base = static_cast<uint32_t>(std::min(prow, kMaxDecodeRows));   // checked below
        du->nchunks = static_cast<uint32_t>(n);
        prow += Hkv * n * M;
        n_items += Hkv * n * ceil_div(M, kMaxItemRows);
    };
    for (int64_t p = 0; p < P; ++p) size_unit(lens->prefix_len[p], cp, Mp, &pl.prefix_units[p]);
    for (int64_t s = 0; s < S; ++s) size_unit(lens->suffix_len[s], cs, r, &pl.suffix_units[s]);
    pl.partial_rows = prow;
    pl.n_items = n_items;
    pl.deep_prefetch = 2 * wide_tokens > item_tokens ? 1 : 0;
    if (n_items > static_cast<int64_t>(INT32_MAX))
        return fail(err, RL_ERR_UNSUPPORTED, "too many work items");
    if (prow > kMaxDecodeRows) return fail(err, RL_ERR_UNSUPPORTED, "too many partial rows (2^32 or more)");

    if (detail != PlanDetail::kSizes) {
        // --- items in creation order with their cost -----------------------------
        const uint64_t kv_bytes_per_tok = 4ull * pl.D;                // K + V, bf16
        const uint64_t partial_bytes_per_row = 2ull * (8 + 4ull * pl.D);  // written, then read
        std::vector<DevItem> &tmp = pl.tmp_items;
        std::vector<uint64_t> &key = pl.tmp_keys;
        tmp.resize(static_cast<size_t>(n_items));
        key.resize(static_cast<size_t>(n_items));
        size_t w = 0;
        uint64_t max_cost = 0;
        auto add_items = [&](int32_t kind, int32_t unit, int32_t kh, int64_t start, int64_t L,
                             int64_t M, const DevUnit &du) {
            const int64_t n = du.nchunks;
            if (n == 0) return;
            const int64_t b = round_up16(ceil_div(L, n));
            const int64_t base = du.base + kh * n * M;
            for (int64_t c = 0; c < n; ++c) {
                const int64_t beg = c * b, cnt = std::min(b, L - beg);
                for (int64_t rb = 0; rb < M; rb += kMaxItemRows) {
                    const int64_t rows = std::min<int64_t>(kMaxItemRows, M - rb);
                    DevItem &d = tmp[w];
                    d.kv_row0 = static_cast<uint32_t>(start + beg);
                    d.partial_row0 = static_cast<uint32_t>(base + c * M + rb);
                    d.unit = unit;
                    d.meta = static_cast<uint32_t>(cnt) | (static_cast<uint32_t>(kind) << 15) |
                             (static_cast<uint32_t>(kh) << 16) | (static_cast<uint32_t>(rb / kMaxItemRows) << 24);
                    const uint64_t cost = static_cast<uint64_t>(cnt) * kv_bytes_per_tok +
                                          static_cast<uint64_t>(rows) * partial_bytes_per_row;
                    key[w] = cost;
                    max_cost = std::max(max_cost, cost);
                    ++w;
                }
            }
        };
        for (int64_t p = 0; p < P; ++p)
            for (int64_t kh = 0; kh < Hkv; ++kh)
                add_items(0, (int32_t)p, (int32_t)kh, lens->prefix_start[p], lens->prefix_len[p], Mp,
                          pl.prefix_units[p]);
        for (int64_t s = 0; s < S; ++s)
            for (int64_t kh = 0; kh < Hkv; ++kh)
                add_items(1, (int32_t)s, (int32_t)kh, lens->suffix_start[s], lens->suffix_len[s], r,
                          pl.suffix_units[s]);

        // --- launch order: longest work first, ties in creation order ------------
        // Stable LSD radix sort of (max_cost - cost) in 8-bit digits; the item
        // index rides in the low 32 bits of each key.
        std::vector<uint64_t> &k2 = pl.tmp_keys2;
        k2.resize(key.size());
        int digits = 0;
        for (uint64_t m = max_cost; m; m >>= 8) ++digits;
        if (digits > 4) {
            // costs above 2^32 (a split of billions of tokens): fall back to a
            // comparison sort on the full cost
            std::vector<uint64_t> cost(key);
            for (size_t i = 0; i < key.size(); ++i) key[i] = i;
            std::stable_sort(key.begin(), key.end(),
                             [&](uint64_t x, uint64_t y) { return cost[x] > cost[y]; });
        } else {
            for (size_t i = 0; i < key.size(); ++i) key[i] = ((max_cost - key[i]) << 32) | i;
            for (int d = 0; d < digits; ++d) {
                size_t count[257] = {0};
                const int sh8 = 32 + 8 * d;
                for (uint64_t v : key) ++count[((v >> sh8) & 255) + 1];
                for (int i = 0; i < 256; ++i) count[i + 1] += count[i];
                for (uint64_t v : key) k2[count[(v >> sh8) & 255]++] = v;
                key.swap(k2);
            }
        }
        // --- one XCD per chunk ---------------------------------------------------
        // A chunk of more than kMaxItemRows query rows (a wide prefix group)
        // is served by g items of equal cost, neighbours after the sort, and
        // neighbours land on different XCDs: each would fetch the chunk into
        // its own L2.  Where kNumXcds such chunks of one cost follow each
        // other, their items are transposed (item j of chunk k to window
        // position j kNumXcds + k), so a chunk's items start on one XCD at
        // about the same time and the later ones read it from that L2.  The
        // window holds items of one cost, so the order stays longest first.
        auto item_of = [&](size_t i) { return static_cast<uint32_t>(key[i] & 0xffffffffu); };
        auto item_cost = [&](uint32_t x) {
            const DevItem &d = tmp[x];
            const int64_t M = (d.meta >> 15) & 1 ? r : Mp;
            const int64_t rows = std::min<int64_t>(kMaxItemRows, M - static_cast<int64_t>(d.meta >> 24) * kMaxItemRows);
            return static_cast<uint64_t>(d.meta & 0x7fff) * kv_bytes_per_tok +
                   static_cast<uint64_t>(rows) * partial_bytes_per_row;
        };
        auto same_chunk = [&](uint32_t x, uint32_t y) {
            return tmp[x].kv_row0 == tmp[y].kv_row0 && tmp[x].unit == tmp[y].unit &&
                   (tmp[x].meta & 0x00ffffffu) == (tmp[y].meta & 0x00ffffffu);
        };
        const size_t n_sorted = key.size();
        auto group_len = [&](size_t p) {
            size_t g = 1;
            while (p + g < n_sorted && same_chunk(item_of(p), item_of(p + g))) ++g;
            return g;
        };
        std::vector<uint64_t> &win = pl.tmp_keys2;
        for (size_t p = 0; p < n_sorted;) {
            const size_t g = group_len(p);
            bool ok = g >= 2 && p + kNumXcds * g <= n_sorted;
            const uint64_t c0 = item_cost(item_of(p));
            for (size_t i = p; ok && i < p + kNumXcds * g; ++i) ok = item_cost(item_of(i)) == c0;
            for (int k = 0; ok && k < kNumXcds; ++k) ok = group_len(p + k * g) == g;
            if (!ok) {
                p += g;
                continue;
            }
            win.assign(key.begin() + p, key.begin() + p + kNumXcds * g);
            for (int k = 0; k < kNumXcds; ++k)
                for (size_t j = 0; j < g; ++j) key[p + j * kNumXcds + k] = win[k * g + j];
            p += kNumXcds * g;
        }
        pl.dev_items.resize(key.size());
        for (size_t i = 0; i < key.size(); ++i) pl.dev_items[i] = tmp[item_of(i)];
        if (detail == PlanDetail::kDebug) {
            pl.items.resize(pl.dev_items.size());
            for (size_t i = 0; i < pl.dev_items.size(); ++i) {
                const DevItem &d = pl.dev_items[i];
                rl_plan_item &it = pl.items[i];
                it = rl_plan_item{};
                it.kind = (d.meta >> 15) & 1;
                it.unit = d.unit;
                it.kv_head = (d.meta >> 16) & 255;
                const DevUnit &du = it.kind == 0 ? pl.prefix_units[d.unit] : pl.suffix_units[d.unit];
                const int64_t M = it.kind == 0 ? Mp : r;
                const int64_t start = it.kind == 0 ? lens->prefix_start[d.unit] : lens->suffix_start[d.unit];
                const int64_t base = du.base + static_cast<int64_t>(it.kv_head) * du.nchunks * M;
                it.chunk = static_cast<int32_t>((static_cast<int64_t>(d.partial_row0) - base) / M);
                it.tok_begin = static_cast<int64_t>(d.kv_row0) - start;
                it.tok_count = static_cast<int32_t>(d.meta & 0x7fff);
                it.row_begin = static_cast<int32_t>((d.meta >> 24) * kMaxItemRows);
                it.row_count = static_cast<int32_t>(std::min<int64_t>(kMaxItemRows, M - it.row_begin));
                it.split_variant = pl.deep_prefetch;
            }
        }
    }

    // --- workspace layout --------------------------------------------------
    size_t off = 0;
    pl.off_items = off;
    off = align_up(off + static_cast<size_t>(n_items) * sizeof(DevItem), 256);
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

rl_status plan_extend(const rl_decode_shape *shape, const rl_extend_lens *lens, ExtendPlan *plan,
                      std::string *err, bool build) {
    if (!shape) return fail(err, RL_ERR_NULL_POINTER, "shape is NULL");
    if (!lens) return fail(err, RL_ERR_NULL_POINTER, "lens is NULL");
    const rl_decode_shape &sh = *shape;
    rl_status st = check_shape(sh, err);
    if (st != RL_OK) return st;
    if (lens->prefix_rows < 0 || lens->suffix_rows < 0 || lens->q_rows < 0)
        return fail(err, RL_ERR_INVALID_SHAPE, "row counts must be >= 0");
    ExtendPlan &pl = *plan;
    pl.P = sh.num_prompts;
    pl.G = sh.group_size;
    pl.Hq = sh.num_q_heads;
    pl.Hkv = sh.num_kv_heads;
    pl.D = sh.head_dim;
    pl.r = sh.num_q_heads / sh.num_kv_heads;
    pl.scale = sh.softmax_scale;
    pl.kv_layout = sh.kv_layout;
    pl.prefix_rows = lens->prefix_rows;
    pl.suffix_rows = lens->suffix_rows;
    pl.q_rows = lens->q_rows;
    pl.n_items = 0;
    pl.any_prefix = false;
    pl.ctx_tokens = 0;
    pl.total_bytes = 0;
    pl.items.clear();
    const int64_t P = pl.P, G = pl.G, S = P * G, r = pl.r;
    if (S > INT32_MAX / 2 || S * pl.Hq > INT32_MAX)
        return fail(err, RL_ERR_UNSUPPORTED, "too many sequences x heads");
    if (S == 0) return RL_OK;
    if (!lens->prefix_start || !lens->prefix_len || !lens->suffix_start || !lens->suffix_len ||
        !lens->new_len || !lens->q_start)
        return fail(err, RL_ERR_NULL_POINTER, "length arrays must not be NULL when P*G > 0");
    int64_t sum_lp = 0, sum_ls = 0;
    st = check_ranges(P, S, lens->prefix_start, lens->prefix_len, lens->prefix_rows, lens->suffix_start,
                      lens->suffix_len, lens->suffix_rows, &sum_lp, &sum_ls, err);
    if (st != RL_OK) return st;
    // new tokens and their query rows; two candidates must not write one row
    pl.tmp_ranges.clear();
    for (int64_t s = 0; s < S; ++s) {
        const int64_t n = lens->new_len[s], q0 = lens->q_start[s];
        if (n < 0 || n > lens->suffix_len[s])
            return fail(err, RL_ERR_INVALID_SHAPE,
                        "new_len[" + std::to_string(s) + "] must be in [0, suffix_len]");
        if (n == 0) continue;
        if (n * r > INT32_MAX) return fail(err, RL_ERR_UNSUPPORTED, "new_len x Hq/Hkv too large");
        if (q0 < 0 || q0 > lens->q_rows - n)
            return fail(err, RL_ERR_INVALID_SHAPE,
                        "query rows of candidate " + std::to_string(s) + " exceed q_rows");
        pl.tmp_ranges.emplace_back(q0, q0 + n);
    }
    std::sort(pl.tmp_ranges.begin(), pl.tmp_ranges.end());
    for (size_t i = 1; i < pl.tmp_ranges.size(); ++i)
        if (pl.tmp_ranges[i].first < pl.tmp_ranges[i - 1].second)
            return fail(err, RL_ERR_INVALID_SHAPE, "two candidates share query rows");

    // blocks: per (prompt, kv head) unit, per candidate, kExtBlockRows unit rows each
    const int64_t Hkv = pl.Hkv;
    int64_t n_items = 0;
    double ctx = 0;
    for (int64_t s = 0; s < S; ++s) {
        const int64_t n = lens->new_len[s];
        if (n == 0) continue;
        n_items += ceil_div(n * r, kExtBlockRows) * Hkv;
        pl.any_prefix |= lens->prefix_len[s / G] > 0;
        const int64_t base = lens->prefix_len[s / G] + lens->suffix_len[s] - n;
        ctx += static_cast<double>(Hkv * r) * (static_cast<double>(n) * base + 0.5 * n * (n + 1));
    }
    pl.n_items = n_items;
    pl.ctx_tokens = ctx;
    pl.total_bytes = align_up(static_cast<size_t>(n_items) * sizeof(ExtItem), 256);
    if (n_items > INT32_MAX) return fail(err, RL_ERR_UNSUPPORTED, "too many work blocks");
    if (!build || n_items == 0) return RL_OK;

    // units by work, largest first; blocks inside a unit by visible context, longest first
    pl.tmp_units.clear();
    for (int64_t p = 0; p < P; ++p) {
        int64_t work = 0;
        for (int64_t g = 0; g < G; ++g) {
            const int64_t s = p * G + g, n = lens->new_len[s];
            work += n * (lens->prefix_len[p] + lens->suffix_len[s]);
        }
        if (work > 0)
            for (int64_t kh = 0; kh < Hkv; ++kh) pl.tmp_units.emplace_back(-work, p * Hkv + kh);
    }
    std::stable_sort(pl.tmp_units.begin(), pl.tmp_units.end());
    pl.items.reserve(static_cast<size_t>(n_items));
    for (const auto &u : pl.tmp_units) {
        const int64_t p = u.second / Hkv, kh = u.second % Hkv;
        pl.tmp_items.clear();
        for (int64_t g = 0; g < G; ++g) {
            const int64_t s = p * G + g, n = lens->new_len[s];
            for (int64_t rb = 0; rb < n * r; rb += kExtBlockRows) {
                ExtItem it{};
                it.prefix_row0 = lens->prefix_len[p] > 0 ? lens->prefix_start[p] : 0;
                it.suffix_row0 = lens->suffix_start[s];
                it.q_row0 = lens->q_start[s];
                it.Lp = lens->prefix_len[p];
                it.Ls = lens->suffix_len[s];
                it.n = static_cast<int32_t>(n);
                it.kh = static_cast<int32_t>(kh);
                it.row_begin = static_cast<int32_t>(rb);
                // visible context of the block's last token, kept in pad for the sort
                const int64_t i_hi = std::min<int64_t>(rb + kExtBlockRows, n * r) - 1;
                it.pad = static_cast<int32_t>(std::min<int64_t>(INT32_MAX, it.Lp + it.Ls - n + i_hi / r + 1));
                pl.tmp_items.push_back(it);
            }
        }
        std::stable_sort(pl.tmp_items.begin(), pl.tmp_items.end(),
                         [](const ExtItem &a, const ExtItem &b) { return a.pad > b.pad; });
        for (ExtItem &it : pl.tmp_items) {
            it.pad = 0;
            pl.items.push_back(it);
        }
    }
    return RL_OK;
}

rl_status check_extend_ptrs(const ExtendPlan &pl, const rl_decode_ptrs *ptrs, std::string *err) {
    if (!ptrs) return fail(err, RL_ERR_NULL_POINTER, "ptrs is NULL");
    if (pl.n_items == 0) return RL_OK;
    if (!ptrs->q) return fail(err, RL_ERR_NULL_POINTER, "q is NULL");
    if (!ptrs->out) return fail(err, RL_ERR_NULL_POINTER, "out is NULL");
    // every candidate with new tokens has a non-empty suffix; the prefix may be empty
    if (!ptrs->k_suffix || !ptrs->v_suffix) return fail(err, RL_ERR_NULL_POINTER, "k_suffix/v_suffix is NULL");
    if (pl.any_prefix && (!ptrs->k_prefix || !ptrs->v_prefix))
        return fail(err, RL_ERR_NULL_POINTER, "k_prefix/v_prefix is NULL");
    const void *a16[] = {ptrs->q, ptrs->k_prefix, ptrs->v_prefix, ptrs->k_suffix, ptrs->v_suffix, ptrs->out};
    const char *names[] = {"q", "k_prefix", "v_prefix", "k_suffix", "v_suffix", "out"};
    for (int i = 0; i < 6; ++i)
        if (a16[i] && !aligned(a16[i], 16))
            return fail(err, RL_ERR_MISALIGNED, std::string(names[i]) + " is not 16-byte aligned");
    if (ptrs->lse && !aligned(ptrs->lse, 4)) return fail(err, RL_ERR_MISALIGNED, "lse is not 4-byte aligned");
    return RL_OK;
}

TailSplit plan_tail_split(int64_t tiles, int64_t nks) {
    TailSplit ts;
    ts.dp_tiles = tiles;
    const int64_t dp = tiles / kNumCUs * kNumCUs, tail = tiles - dp;
    if (dp > 0 && tail > 0 && 2 * tail <= kNumCUs) {
        const int64_t s = std::min<int64_t>(std::min<int64_t>(kMaxTailSplits, kNumCUs / tail), nks / 4);
        if (s >= 2) {
            ts.dp_tiles = dp;
            ts.tail_tiles = tail;
            ts.splits = static_cast<int32_t>(s);
        }
    }
    return ts;
}

TailSplit bwd_probs_tail(const LogprobBwdPlan &plan, int64_t n) {
    return plan_tail_split(plan.n_vocab_tiles * ceil_div(n, kRowTile), plan.H / kHiddenStep);
}

TileRounds plan_tile_rounds(int64_t rows, int32_t vocab) {
    // With at most 4 row tiles (the tiles of one vocab tile are neighbours in
    // launch order), the whole vocab tiles of the full rounds run as they are
    // and the rest of the vocabulary runs as one round of tiles 128 or 192
    // entries wide, the narrower that fits on the CUs (a tile of either takes
    // less time than a whole one, and every tile of the round runs at once).
    TileRounds tr;
    const int64_t nvt = ceil_div(vocab, kVocabTile), nrt = ceil_div(rows, kRowTile);
    const int64_t tiles = nvt * nrt;
    const int64_t dp = tiles / kNumCUs * kNumCUs, tail = tiles - dp;
    tr.dp_tiles = tiles;
    tr.n_partials = nvt;
    if (dp > 0 && tail > 0 && nrt <= kNarrowMaxRowTiles) {
        const int64_t vt0 = dp / nrt;
        for (int tm = kNarrowMinTM; tm <= kNarrowMaxTM; ++tm) {
            const int64_t n = ceil_div(vocab - vt0 * kVocabTile, 64 * tm);
            if (n * nrt > kNumCUs) continue;
            tr.dp_tiles = vt0 * nrt;
            tr.narrow_v0 = vt0 * kVocabTile;
            tr.narrow_tiles = n;
            tr.narrow_slot0 = vt0;
            tr.narrow_tm = tm;
            tr.n_partials = vt0 + n;
            break;
        }
    }
    return tr;
}

rl_status plan_logprob(int64_t rows, int32_t hidden, int32_t vocab, LogprobPlan *plan,
                       std::string *err) {
    if (rows < 0) return fail(err, RL_ERR_INVALID_SHAPE, "rows < 0");
    if (hidden <= 0) return fail(err, RL_ERR_INVALID_SHAPE, "hidden must be > 0");
    if (vocab <= 0) return fail(err, RL_ERR_INVALID_SHAPE, "vocab must be > 0");
    if (hidden % kHiddenStep)
        return fail(err, RL_ERR_UNSUPPORTED, "hidden must be a multiple of 64");
    if (hidden > kMaxHidden)
        return fail(err, RL_ERR_UNSUPPORTED, "hidden must be <= 4194304");
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
    const TailSplit ts = plan_tail_split(pl.n_vocab_tiles * pl.n_row_tiles, hidden / kHiddenStep);
    pl.n_dp_tiles = ts.dp_tiles;
    pl.n_tail_tiles = ts.tail_tiles;
    pl.tail_splits = ts.splits;
    pl.n_partials = pl.n_vocab_tiles;
    // A last round more than half full: narrow tiles, when they fit.
    if (pl.n_tail_tiles == 0) {
        const TileRounds tr = plan_tile_rounds(rows, vocab);
        pl.n_dp_tiles = tr.dp_tiles;
        pl.narrow_v0 = tr.narrow_v0;
        pl.narrow_tiles = tr.narrow_tiles;
        pl.narrow_slot0 = tr.narrow_slot0;
        pl.narrow_tm = tr.narrow_tm;
        pl.n_partials = tr.n_partials;
    }
    size_t off = 0;
    pl.off_m = off;
    off = align_up(off + static_cast<size_t>(pl.n_partials) * rows * 4, 256);
    pl.off_l = off;
    off = align_up(off + static_cast<size_t>(pl.n_partials) * rows * 4, 256);
    pl.off_zt = off;
    off = align_up(off + static_cast<size_t>(rows) * 4, 256);
    pl.off_part = off;
    off += static_cast<size_t>(pl.n_tail_tiles) * pl.tail_splits * kVocabTile * kRowTile * 4;
    pl.total_bytes = off;
    return RL_OK;
}

rl_status plan_logprob_bwd(int64_t rows, int32_t hidden, int32_t vocab, LogprobBwdPlan *plan,
                           std::string *err) {
    LogprobPlan fwd;
    const rl_status st = plan_logprob(rows, hidden, vocab, &fwd, err);
    if (st != RL_OK) return st;
    LogprobBwdPlan &pl = *plan;
    pl = LogprobBwdPlan{};
    pl.R = rows;
    pl.H = hidden;
    pl.V = vocab;
    pl.n_vocab_tiles = ceil_div(vocab, kVocabTile);
    pl.n_vsteps = static_cast<int32_t>(pl.n_vocab_tiles * (kVocabTile / kHiddenStep));
    pl.n_h_tiles = static_cast<int32_t>(ceil_div(hidden, 256));
    if (rows == 0) return RL_OK;
    pl.chunk_rows = std::min<int64_t>(rows, kBwdChunkRows);
    pl.n_chunks = ceil_div(rows, pl.chunk_rows);
    pl.chunk_row_tiles = static_cast<int32_t>(ceil_div(pl.chunk_rows, kRowTile));
    // Split the vocabulary when a chunk has fewer output tiles than the GPU
    // has compute units, keeping at least 16 vocab steps per split.
    const int64_t tiles = static_cast<int64_t>(pl.chunk_row_tiles) * pl.n_h_tiles;
    int64_t splits = tiles >= 256 ? 1 : 256 / tiles;
    splits = std::max<int64_t>(1, std::min<int64_t>(splits, pl.n_vsteps / 16));
    pl.steps_per_split = static_cast<int32_t>(ceil_div(pl.n_vsteps, splits));
    pl.splits = static_cast<int32_t>(ceil_div(pl.n_vsteps, pl.steps_per_split));
    if (tiles * pl.splits > INT32_MAX || pl.n_vocab_tiles * pl.chunk_row_tiles > INT32_MAX)
        return fail(err, RL_ERR_UNSUPPORTED, "too many tiles");
    const size_t rows_pad = static_cast<size_t>(pl.chunk_row_tiles) * kRowTile;
    size_t off = 0;
    pl.off_probs = off;
    off = align_up(off + rows_pad * static_cast<size_t>(pl.n_vsteps) * kHiddenStep * 2, 256);
    // the GEMM's split sums and the probability tail's parts share one
    // section: the reduce kernel has summed the parts before the GEMM writes
    pl.off_part = off;
    size_t part_bytes = pl.splits > 1 ? static_cast<size_t>(pl.splits) * rows_pad * hidden * 4 : 0;
    for (const int64_t n : {pl.chunk_rows, rows % pl.chunk_rows}) {
        if (n == 0) continue;
        const TailSplit ts = bwd_probs_tail(pl, n);
        part_bytes = std::max(part_bytes, static_cast<size_t>(ts.tail_tiles) * ts.splits * kVocabTile * kRowTile * 4);
    }
    if (part_bytes > 0) off = align_up(off + part_bytes, 256);
    pl.total_bytes = off;
    return RL_OK;
}

rl_status plan_sample(int64_t rows, int32_t hidden, int32_t vocab, SamplePlan *plan, std::string *err) {
    LogprobPlan fwd;
    const rl_status st = plan_logprob(rows, hidden, vocab, &fwd, err);
    if (st != RL_OK) return st;
    if (vocab > kSampleMaxVocab) return fail(err, RL_ERR_UNSUPPORTED, "vocab must be <= 2097152");
    SamplePlan &pl = *plan;
    pl = SamplePlan{};
    pl.R = rows;
    pl.H = hidden;
    pl.V = vocab;
    pl.n_vocab_tiles = ceil_div(vocab, kVocabTile);
    // one tile of padding past the vocab tiles: a narrow last round's tiles
    // (128 or 192 wide from a whole tile's edge) end at most 191 entries past V
    pl.ld = (pl.n_vocab_tiles + 1) * kVocabTile;
    if (rows == 0) return RL_OK;
    pl.chunk_rows = std::min<int64_t>(rows, kSampleChunkRows);
    const int64_t rows_pad = ceil_div(pl.chunk_rows, kRowTile) * kRowTile;
    size_t off = 0;
    pl.off_logits = off;
    off = align_up(off + static_cast<size_t>(rows_pad) * pl.ld * 4, 256);
    // row-maximum slots: the whole tiles' and, per chunk, those of its narrow
    // last round (at most twice as many tiles cover the rest of the vocabulary)
    pl.pm_slots = std::max(pl.n_vocab_tiles, plan_tile_rounds(pl.chunk_rows, vocab).n_partials);
    if (rows % pl.chunk_rows)
        pl.pm_slots = std::max(pl.pm_slots, plan_tile_rounds(rows % pl.chunk_rows, vocab).n_partials);
    pl.off_pm = off;
    off = align_up(off + static_cast<size_t>(pl.pm_slots) * pl.chunk_rows * 4, 256);
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
