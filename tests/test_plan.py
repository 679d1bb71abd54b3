"""Properties of the split-K work list (host-only, exact integer checks).

The plan must cover every KV token of every (unit, kv head) exactly once for
every query row the unit serves, respect the chunk bound, be deterministic,
and be ordered longest-first so skewed lengths balance across compute units.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import paper_2607_20908_amd as rk
import workloads as W


def plan_for(P, G, Hq, Hkv, D, lp, ls, split=0):
    lp = np.asarray(lp, np.int32)
    ls = np.asarray(ls, np.int32)
    ps, ss = W.packed_starts(lp), W.packed_starts(ls)
    items = rk.decode_plan(P, G, Hq, Hkv, D, ps, lp, ss, ls, int(lp.sum()), int(ls.sum()),
                           split_tokens=split)
    return items, lp, ls


def check_cover(items, P, G, Hq, Hkv, lp, ls, split=None):
    r = Hq // Hkv
    S = P * G
    assert (items["tok_count"] >= 1).all()
    assert (items["row_count"] >= 1).all() and (items["row_count"] <= 64).all()
    if split:
        assert (items["tok_count"] <= split).all()
    # exact coverage: every (kind, unit, kh, token, row) exactly once
    cover = {}
    for it in items:
        key = (int(it["kind"]), int(it["unit"]), int(it["kv_head"]))
        arr = cover.setdefault(key, [])
        arr.append((int(it["tok_begin"]), int(it["tok_count"]), int(it["row_begin"]),
                    int(it["row_count"])))
    for p in range(P):
        for kh in range(Hkv):
            grid = np.zeros((lp[p], G * r), np.int32)
            for (a, n, rb, rc) in cover.get((0, p, kh), []):
                grid[a:a + n, rb:rb + rc] += 1
            assert (grid == 1).all(), f"prefix ({p},{kh}) not covered exactly once"
    for s in range(S):
        for kh in range(Hkv):
            grid = np.zeros((ls[s], r), np.int32)
            for (a, n, rb, rc) in cover.get((1, s, kh), []):
                grid[a:a + n, rb:rb + rc] += 1
            assert (grid == 1).all(), f"suffix ({s},{kh}) not covered exactly once"
    # no items for units that do not exist
    for (kind, unit, kh) in cover:
        assert 0 <= kh < Hkv
        assert 0 <= unit < (P if kind == 0 else S)


def cost(items, D=128):
    return items["tok_count"].astype(np.int64) * 4 * D + items["row_count"] * 2 * (8 + 4 * D)


def test_workload_plans_cover_and_balance():
    for name in ("tiny", "8b", "32b", "longctx"):
        cfg = W.DECODE_CONFIGS[name]
        ls = W.suffix_lengths(cfg, 0)
        lp = np.full(cfg.num_prompts, cfg.prefix_len, np.int32)
        items, lp, ls = plan_for(cfg.num_prompts, cfg.group_size, cfg.num_q_heads,
                                 cfg.num_kv_heads, cfg.head_dim, lp, ls)
        check_cover(items, cfg.num_prompts, cfg.group_size, cfg.num_q_heads, cfg.num_kv_heads, lp, ls)
        c = cost(items, cfg.head_dim)
        assert (np.diff(c) <= 0).all(), "launch order must be longest first"
        if name != "tiny":
            # enough items to spread over 256 compute units, none dominating
            assert len(items) >= 512, (name, len(items))
            assert c.max() <= 0.6 * c.sum() / 256, (name, c.max(), c.sum() / 256)
    # a prefix chunk serves its group's query rows in items of at most 64 rows:
    # G*r = 16*8 = 128 rows -> two items per chunk, rows [0, 64) and [64, 128)
    cfg = W.DECODE_CONFIGS["32b"]
    items, _, _ = plan_for(cfg.num_prompts, cfg.group_size, cfg.num_q_heads, cfg.num_kv_heads,
                           cfg.head_dim, np.full(16, 2048), W.suffix_lengths(cfg, 0))
    pre = items[items["kind"] == 0]
    assert (pre["row_count"] == 64).all() and sorted(set(pre["row_begin"])) == [0, 64]


def test_row_blocks_of_a_chunk_share_an_xcd():
    # workgroups go to the 8 XCDs in turn: the items of one wide prefix chunk
    # are 8 launch positions apart, so they run on one XCD and share its L2
    cfg = W.DECODE_CONFIGS["32b"]
    items, _, _ = plan_for(cfg.num_prompts, cfg.group_size, cfg.num_q_heads, cfg.num_kv_heads,
                           cfg.head_dim, np.full(16, 2048), W.suffix_lengths(cfg, 0))
    pos = {}
    for i, it in enumerate(items):
        if it["kind"] == 0:
            pos.setdefault((int(it["unit"]), int(it["kv_head"]), int(it["tok_begin"])), []).append(
                (int(it["row_begin"]), i))
    assert len(pos) == 16 * 8
    for blocks in pos.values():
        (rb0, i0), (rb1, i1) = sorted(blocks)
        assert (rb0, rb1) == (0, 64) and i1 - i0 == 8, blocks
    # three blocks per chunk (G*r = 192): 8 chunks of one cost at a time
    items, _, _ = plan_for(4, 24, 64, 8, 128, np.full(4, 1024), np.full(96, 700))
    pre = np.flatnonzero(items["kind"] == 0)
    by_chunk = {}
    for i in pre:
        it = items[i]
        by_chunk.setdefault((int(it["unit"]), int(it["kv_head"]), int(it["tok_begin"])), []).append(int(i))
    full = [sorted(v) for v in by_chunk.values() if len(v) == 3]
    assert full and all(np.all(np.diff(v) == 8) for v in full)


@pytest.mark.parametrize("lengths", ["equal", "one_giant", "geometric", "zeros"])
def test_skewed_lengths(lengths):
    P, G, Hq, Hkv = 4, 8, 64, 8
    rng = np.random.Generator(np.random.PCG64(3))
    if lengths == "equal":
        ls = np.full(P * G, 700)
    elif lengths == "one_giant":
        ls = np.full(P * G, 10); ls[5] = 60000
    elif lengths == "geometric":
        ls = np.minimum(rng.geometric(1 / 1024, P * G), 4096)
    else:
        ls = np.zeros(P * G, np.int32)
    lp = np.array([24576, 0, 100, 3000])
    items, lp, ls = plan_for(P, G, Hq, Hkv, 128, lp, ls)
    check_cover(items, P, G, Hq, Hkv, lp, ls)
    again, _, _ = plan_for(P, G, Hq, Hkv, 128, lp, ls)
    assert np.array_equal(items, again), "plan must be deterministic"


def test_forced_split():
    items, lp, ls = plan_for(2, 3, 8, 2, 64, [100, 37], [16, 1, 0, 45, 80, 17], split=16)
    check_cover(items, 2, 3, 8, 2, lp, ls, split=16)
    assert items["tok_count"].max() == 16


def test_wide_groups_split_rows():
    # G*r = 32*8 = 256 query rows per kv head -> four row blocks per prefix chunk
    items, lp, ls = plan_for(1, 32, 16, 2, 128, [300], np.full(32, 5))
    check_cover(items, 1, 32, 16, 2, lp, ls)
    pre = items[items["kind"] == 0]
    assert sorted(set(pre["row_begin"])) == [0, 64, 128, 192]


@settings(max_examples=60, deadline=None)
@given(P=st.integers(1, 3), G=st.integers(1, 5), Hkv=st.integers(1, 3), r=st.integers(1, 6),
       split=st.sampled_from([0, 16, 48, 64, 112]), data=st.data())
def test_cover_fuzz(P, G, Hkv, r, split, data):
    S = P * G
    lp = data.draw(st.lists(st.integers(0, 300), min_size=P, max_size=P))
    ls = data.draw(st.lists(st.integers(0, 300), min_size=S, max_size=S))
    items, lp, ls = plan_for(P, G, Hkv * r, Hkv, 64, lp, ls, split=split)
    check_cover(items, P, G, Hkv * r, Hkv, lp, ls, split=split or None)


def test_split_variant_follows_item_widths():
    # prompts shared by G * r = 64 query rows dominating the KV: two tiles in flight
    P, G, Hq, Hkv = 3, 8, 16, 2
    lp = np.array([700, 0, 193], np.int32)
    ls = np.array([5, 0, 17, 64, 1, 65, 0, 30] + [3, 9, 0, 2, 40, 1, 0, 12] + [63, 0, 1, 2, 3, 4, 5, 6], np.int32)
    ps = np.array([0, 700, 700], np.int64)
    ss = np.concatenate([[0], np.cumsum(ls)[:-1]]).astype(np.int64)
    it = rk.decode_plan(P, G, Hq, Hkv, 128, ps, lp, ss, ls, 1000, int(ls.sum()))
    assert set(it["split_variant"]) == {1}
    # the 8B-class step: 4-row suffix items hold most of the KV
    cfg = W.DECODE_CONFIGS["8b"]
    sl = W.suffix_lengths(cfg, seed=0).astype(np.int32)
    ss = np.concatenate([[0], np.cumsum(sl)[:-1]]).astype(np.int64)
    it = rk.decode_plan(64, 8, 32, 8, 128, np.arange(64, dtype=np.int64) * 1024, np.full(64, 1024, np.int32),
                        ss, sl, 65536, int(sl.sum()))
    assert set(it["split_variant"]) == {0}
