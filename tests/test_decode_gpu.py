"""Decode attention: the HIP path against the fp64 oracle on the same bits.

Bar: attention output max-abs <= 1e-2, lse max-abs <= 1e-3, and bit-exact
indexing (one-hot probes reproduce the chosen value row exactly; uniform
attention recovers each context length exactly).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_20908_amd as rk
import workloads as W
from gpu_util import (ATTN_LSE_TOL, ATTN_OUT_TOL, decode_host_case, dev, max_abs, say, to_dev)

pytestmark = pytest.mark.gpu


def run_gpu(c, scale, split=0, workspace=None, layout="token"):
    """GPU call on host-side token-major bits; layout "head" transposes the KV first."""
    def kv(bits):
        return to_dev(np.ascontiguousarray(np.transpose(bits, (1, 0, 2))) if layout == "head" else bits)
    t = {k: kv(c[k]) for k in ("k_prefix", "v_prefix", "k_suffix", "v_suffix")}
    t["q"] = to_dev(c["q"])
    out, lse = rk.decode_attn(t["q"], t["k_prefix"], t["v_prefix"], t["k_suffix"], t["v_suffix"],
                              c["prefix_start"], c["prefix_len"], c["suffix_start"], c["suffix_len"],
                              c["group_size"], scale=scale, split_tokens=split, return_lse=True,
                              workspace=workspace, kv_layout=layout)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), lse.cpu().numpy(), W.bf16_bits(out)


def run_oracle(c, scale):
    return oracle.decode_attn(c["q"], c["k_prefix"], c["v_prefix"], c["k_suffix"], c["v_suffix"],
                              c["prefix_start"], c["prefix_len"], c["suffix_start"], c["suffix_len"],
                              c["group_size"], scale)


def check(c, scale, split=0, what="", layout="token"):
    say(f"decode parity {what} split={split} layout={layout}")
    o, l, _ = run_gpu(c, scale, split, layout=layout)
    ro, rl = run_oracle(c, scale)
    eo, el = max_abs(o, ro), max_abs(l, rl)
    assert eo <= ATTN_OUT_TOL, f"{what}: out max-abs {eo}"
    assert el <= ATTN_LSE_TOL, f"{what}: lse max-abs {el}"
    return eo, el


def test_tiny_config():
    cfg = W.DECODE_CONFIGS["tiny"]
    x = W.make_decode_inputs(cfg, "cpu")
    c = dict(q=W.bf16_bits(x.q), k_prefix=W.bf16_bits(x.k_prefix), v_prefix=W.bf16_bits(x.v_prefix),
             k_suffix=W.bf16_bits(x.k_suffix), v_suffix=W.bf16_bits(x.v_suffix),
             prefix_start=x.prefix_start, prefix_len=x.prefix_len, suffix_start=x.suffix_start,
             suffix_len=x.suffix_len, group_size=cfg.group_size)
    check(c, x.scale, what="tiny config")


@pytest.mark.parametrize("layout", ["token", "head"])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("split", [0, 16, 48, 64, 112])
def test_ragged_multi_tile(D, split, layout):
    # several 64-token tiles per unit, ragged tails, empty prefixes and suffixes
    P, G, Hq, Hkv = 3, 4, 16, 4
    lp = [300, 0, 129]
    ls = [200, 1, 0, 63, 64, 65, 0, 17, 250, 3, 128, 31]
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=D + split, gap=3)
    check(c, 1.0 / math.sqrt(D), split, f"ragged D={D}", layout)


@pytest.mark.parametrize("layout", ["token", "head"])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("split", [0, 16, 64, 112, 176])
def test_wide_items_two_tiles_in_flight(D, split, layout):
    """Prefix items of 64 query rows (G * r = 64) hold most of the KV tokens
    (893 of about 1300), so the split kernel keeps two tiles in flight per
    workgroup; chunks of one to three tiles with ragged ends exercise the
    empty loads issued past a chunk's last tile."""
    P, G, Hq, Hkv = 3, 8, 16, 2
    lp = [700, 0, 193]
    ls = ([5, 0, 17, 64, 1, 65, 0, 30] + [3, 9, 0, 2, 40, 1, 0, 12] + [63, 0, 1, 2, 3, 4, 5, 6])
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=D * 7 + split, gap=2)
    assert set(plan_of(c, Hq, Hkv, D, split)["split_variant"]) == {1}, "two tiles in flight expected"
    check(c, 1.0 / math.sqrt(D), split, f"wide items D={D}", layout)


def plan_of(c, Hq, Hkv, D, split=0):
    P = len(c["prefix_len"])
    return rk.decode_plan(P, c["group_size"], Hq, Hkv, D, c["prefix_start"], c["prefix_len"], c["suffix_start"],
                          c["suffix_len"], c["k_prefix"].shape[0], c["k_suffix"].shape[0], split_tokens=split)


@pytest.mark.parametrize("layout", ["token", "head"])
@pytest.mark.parametrize("D", [64, 128])
def test_one_query_head_per_kv_head(D, layout):
    """Hq = Hkv (r = 1): plain multi-head attention, each candidate's suffix
    item serving one query row per kv head; the prefix items serve G rows."""
    P, G, Hq, Hkv = 3, 5, 8, 8
    lp = [257, 0, 64]
    ls = [1, 0, 130, 64, 17] + [0, 5, 300, 2, 63] + [65, 1, 0, 128, 40]
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=11 * D, gap=3)
    check(c, 1.0 / math.sqrt(D), 0, f"r=1 D={D}", layout)
    check(c, 1.0 / math.sqrt(D), 32, f"r=1 D={D}", layout)


@pytest.mark.parametrize("G,Hq,Hkv", [(16, 64, 8),   # 128 query rows per kv head: two 64-row items per chunk
                                       (20, 16, 2),   # 160 rows: three row blocks per prefix chunk
                                       (5, 12, 4),    # 15 rows: one partial column tile
                                       (3, 24, 2),    # r = 12 per candidate
                                       (2, 160, 2),   # r = 80: two row blocks per suffix chunk too
                                       (1, 128, 1)])  # r = 128, the largest: G = 1
def test_group_shapes(G, Hq, Hkv):
    P = 2
    rng = np.random.Generator(np.random.PCG64(G * 100 + Hq))
    lp = [257, 90]
    ls = rng.integers(0, 160, P * G)
    c = decode_host_case(P, G, Hq, Hkv, 128, lp, ls, seed=G + Hq, gap=1)
    check(c, 1.0 / math.sqrt(128), 0, f"G={G} Hq={Hq} Hkv={Hkv}")
    check(c, 1.0 / math.sqrt(128), 32, f"G={G} Hq={Hq} Hkv={Hkv}", "head")


@pytest.mark.parametrize("D", [64, 128])
def test_many_rows_many_partials(D):
    """More rows than one round of one-row waves (16384 > 8192), so the
    combine runs two rows per wave, with 16-token chunks, so rows merge 10 to
    about 40 partials: the value batches (4 rows at D = 128) and the path for
    more than 32 partials of that launch both run."""
    P, G, Hq, Hkv = 16, 8, 128, 8
    rng = np.random.Generator(np.random.PCG64(4242 + D))
    lp = rng.integers(150, 220, P)
    ls = rng.integers(1, 420, P * G)
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=77 + D, gap=2)
    check(c, 1.0 / math.sqrt(D), 16, f"16384 rows, 16-token chunks, D={D}", "head")


def test_peaky_scores():
    c = decode_host_case(2, 4, 8, 2, 128, [200, 77], [40, 0, 90, 5, 66, 1, 0, 130], seed=9,
                         qmul=4.0, gap=2)
    check(c, 1.0 / math.sqrt(128), 0, "peaky")


def test_nan_poisoned_padding_and_workspace():
    c = decode_host_case(2, 3, 8, 2, 128, [150, 64], [10, 0, 70, 33, 1, 129], seed=4, gap=5,
                         poison=True)
    scale = 1.0 / math.sqrt(128)
    need = rk.decode_attn_workspace_size(2, 3, 8, 2, 128, c["prefix_start"], c["prefix_len"],
                                         c["suffix_start"], c["suffix_len"],
                                         c["k_prefix"].shape[0], c["k_suffix"].shape[0], scale)
    ws = torch.full((need // 4,), float("nan"), dtype=torch.float32, device=dev()).view(torch.uint8)
    ro, rl = run_oracle(c, scale)
    for layout in ("token", "head"):
        say(f"decode poisoned padding + workspace, layout {layout}")
        ws.view(torch.float32).fill_(float("nan"))
        o, l, _ = run_gpu(c, scale, 0, workspace=ws, layout=layout)
        assert np.isfinite(o).all() and np.isfinite(l).all()
        assert max_abs(o, ro) <= ATTN_OUT_TOL and max_abs(l, rl) <= ATTN_LSE_TOL


def test_nan_poisoned_two_tiles_in_flight():
    """The two-tiles-in-flight variant (items of G * r = 64 query rows hold
    most of the KV) against NaN gap rows and a NaN workspace: the empty loads
    past a chunk's last tile and the final merge must touch neither."""
    P, G, Hq, Hkv, D = 2, 8, 16, 2, 128
    lp, ls = [450, 129], [3, 0, 64, 1, 17, 2, 0, 65, 5, 1, 0, 33, 2, 64, 1, 0]
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=21, gap=4, poison=True)
    scale = 1.0 / math.sqrt(D)
    assert set(plan_of(c, Hq, Hkv, D)["split_variant"]) == {1}
    need = rk.decode_attn_workspace_size(P, G, Hq, Hkv, D, c["prefix_start"], c["prefix_len"], c["suffix_start"],
                                         c["suffix_len"], c["k_prefix"].shape[0], c["k_suffix"].shape[0], scale)
    ws = torch.full((need // 4 + 1,), float("nan"), dtype=torch.float32, device=dev()).view(torch.uint8)
    ro, rl = run_oracle(c, scale)
    for layout in ("token", "head"):
        say(f"decode poisoned padding + workspace, two tiles in flight, layout {layout}")
        ws.view(torch.float32).fill_(float("nan"))
        o, l, _ = run_gpu(c, scale, 0, workspace=ws, layout=layout)
        assert np.isfinite(o).all() and np.isfinite(l).all()
        assert max_abs(o, ro) <= ATTN_OUT_TOL and max_abs(l, rl) <= ATTN_LSE_TOL


def test_many_calls_in_flight():
    """100 calls enqueued without a synchronisation, four problems in turn:
    more calls than the 64 pinned staging buffers, so buffers are reused (or
    waited for) while earlier calls are still queued.  Every output must match
    the oracle; a work list overwritten before its fetch ran would not."""
    D = 128
    cases = [decode_host_case(2, 4, 8, 2, D, [100 + 37 * i, 64], [(i * 13 + 7 * j) % 90 for j in range(8)],
                              seed=40 + i, gap=1) for i in range(4)]
    scale = 1.0 / math.sqrt(D)
    refs = [run_oracle(c, scale) for c in cases]
    dev_in = []
    for c in cases:
        t = {k: to_dev(c[k]) for k in ("q", "k_prefix", "v_prefix", "k_suffix", "v_suffix")}
        dev_in.append(t)
    say("decode: 100 calls in flight")
    outs = []
    for n in range(100):
        c, t = cases[n % 4], dev_in[n % 4]
        outs.append(rk.decode_attn(t["q"], t["k_prefix"], t["v_prefix"], t["k_suffix"], t["v_suffix"],
                                   c["prefix_start"], c["prefix_len"], c["suffix_start"], c["suffix_len"],
                                   c["group_size"], scale=scale, return_lse=True))
    torch.cuda.synchronize()
    for n, (o, l) in enumerate(outs):
        ro, rl = refs[n % 4]
        assert max_abs(o.float().cpu().numpy(), ro) <= ATTN_OUT_TOL, f"call {n}"
        assert max_abs(l.cpu().numpy(), rl) <= ATTN_LSE_TOL, f"call {n}"


def test_bitwise_deterministic():
    c = decode_host_case(2, 8, 32, 8, 128, [700, 333], np.arange(16) * 37 % 500, seed=5, gap=0)
    scale = 1.0 / math.sqrt(128)
    say("decode determinism")
    _, l1, b1 = run_gpu(c, scale)
    _, l2, b2 = run_gpu(c, scale)
    assert np.array_equal(b1, b2) and np.array_equal(l1.view(np.uint32), l2.view(np.uint32))


def test_one_hot_probe_bit_exact():
    """One dominant key per (sequence, kv head): the output is that value row, bit for bit."""
    P, G, Hq, Hkv, D = 3, 4, 16, 4, 128
    r = Hq // Hkv
    rng = np.random.Generator(np.random.PCG64(21))
    lp = np.array([300, 1, 140], np.int32)
    ls = rng.integers(1, 200, P * G).astype(np.int32)
    ls[[2, 7]] = 0
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=21, gap=2)
    S = P * G
    q = np.zeros((S, Hq, D), np.float32); q[:, :, 0] = 1.0
    kp = np.zeros((c["k_prefix"].shape[0], Hkv, D), np.float32)
    ks = np.zeros((c["k_suffix"].shape[0], Hkv, D), np.float32)
    vp = np.zeros_like(kp); vs = np.zeros_like(ks)
    for arr, tag in ((vp, 1.0), (vs, 2.0)):
        rows = np.arange(arr.shape[0])
        for kh in range(Hkv):
            arr[:, kh, 0] = tag
            arr[:, kh, 1] = kh
            arr[:, kh, 2] = rows % 256
            arr[:, kh, 3] = rows // 256
            arr[:, kh, 4 + kh] = 1.0 + (rows % 7)
    expect = np.zeros((S, Hq, D), np.float32)
    for p in range(P):
        for kh in range(Hkv):
            j = int(c["prefix_start"][p] + rng.integers(0, lp[p]))
            kp[j, kh, 0] = 256.0
            for g in range(G):
                s = p * G + g
                if ls[s] and rng.random() < 0.5:
                    jj = int(c["suffix_start"][s] + rng.integers(0, ls[s]))
                    ks[jj, kh, 0] = 512.0
                    src = vs[jj, kh]
                else:
                    src = vp[j, kh]
                expect[s, kh * r:(kh + 1) * r] = src
    bits = lambda a: W.bf16_bits(torch.from_numpy(a).to(torch.bfloat16))
    c.update(q=bits(q), k_prefix=bits(kp), v_prefix=bits(vp), k_suffix=bits(ks), v_suffix=bits(vs))
    say("decode one-hot probe")
    for split, layout in ((0, "token"), (16, "token"), (64, "token"), (0, "head"), (16, "head")):
        _, _, out_bits = run_gpu(c, 1.0, split, layout=layout)
        assert np.array_equal(out_bits, bits(expect)), f"one-hot probe mismatch (split {split}, {layout})"


def test_length_probe_exact():
    """Zero keys give uniform weights: round(exp(lse)) is each context length exactly."""
    P, G, Hq, Hkv, D = 4, 4, 8, 2, 64
    rng = np.random.Generator(np.random.PCG64(22))
    lp = np.array([0, 1000, 64, 5], np.int32)
    ls = rng.integers(0, 300, P * G).astype(np.int32)
    ls[0] = 0
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=22, gap=1)
    c["k_prefix"] = np.zeros_like(c["k_prefix"])
    c["k_suffix"] = np.zeros_like(c["k_suffix"])
    say("decode length probe")
    o, l, _ = run_gpu(c, 1.0 / 8, 48, layout="head")
    T = np.array([lp[s // G] + ls[s] for s in range(P * G)])
    for s in range(P * G):
        if T[s] == 0:
            assert (l[s] == -np.inf).all() and (o[s] == 0).all()
        else:
            assert (np.rint(np.exp(l[s].astype(np.float64))) == T[s]).all(), (s, T[s], l[s])
    ro, _ = run_oracle(c, 1.0 / 8)
    assert max_abs(o, ro) <= ATTN_OUT_TOL


def test_prefix_sharing_equals_concatenation():
    P, G, Hq, Hkv, D = 2, 4, 16, 4, 128
    lp = np.array([180, 70], np.int32)
    ls = np.array([5, 0, 60, 130, 1, 2, 64, 40], np.int32)
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=23)
    scale = 1.0 / math.sqrt(D)
    kr, vr, st, ln = [], [], [], []
    pos = 0
    for s in range(P * G):
        p = s // G
        a, n = c["prefix_start"][p], lp[p]
        b, m = c["suffix_start"][s], ls[s]
        kr.append(np.concatenate([c["k_prefix"][a:a + n], c["k_suffix"][b:b + m]]))
        vr.append(np.concatenate([c["v_prefix"][a:a + n], c["v_suffix"][b:b + m]]))
        st.append(pos); ln.append(n + m); pos += n + m
    c2 = dict(c, k_prefix=c["k_prefix"][:1], v_prefix=c["v_prefix"][:1],
              prefix_start=np.zeros(P, np.int64), prefix_len=np.zeros(P, np.int32),
              k_suffix=np.concatenate(kr), v_suffix=np.concatenate(vr),
              suffix_start=np.array(st, np.int64), suffix_len=np.array(ln, np.int32))
    say("decode prefix sharing")
    o1, l1, _ = run_gpu(c, scale)
    o2, l2, _ = run_gpu(c2, scale)
    ro, rl = run_oracle(c, scale)
    for o, l in ((o1, l1), (o2, l2)):
        assert max_abs(o, ro) <= ATTN_OUT_TOL and max_abs(l, rl) <= ATTN_LSE_TOL
    assert max_abs(o1, o2) <= 2 * ATTN_OUT_TOL


def test_empty_batch_noop():
    q = torch.empty((0, 8, 128), dtype=torch.bfloat16, device=dev())
    kv = torch.empty((0, 2, 128), dtype=torch.bfloat16, device=dev())
    out = rk.decode_attn(q, kv, kv, kv, kv, [], [], [], [], group_size=4)
    assert out.shape == (0, 8, 128)


@pytest.mark.slow
@pytest.mark.parametrize("name,layout", [("8b", "head"), ("32b", "head"), ("longctx", "head"),
                                         ("8b", "token")])
def test_full_size_workloads(name, layout):
    """The full-size decode workloads in the configuration the bench times (head-major KV),
    and the 8B-class step in the token-major layout."""
    cfg = W.DECODE_CONFIGS[name]
    say(f"decode full-size {name} {layout}: generating")
    x = W.make_decode_inputs(cfg, dev(), kv_layout=layout)
    say(f"decode full-size {name} {layout}: gpu")
    out, lse = rk.decode_attn(x.q, x.k_prefix, x.v_prefix, x.k_suffix, x.v_suffix,
                              x.prefix_start, x.prefix_len, x.suffix_start, x.suffix_len,
                              cfg.group_size, scale=x.scale, return_lse=True, kv_layout=layout)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    l = lse.cpu().numpy()
    say(f"decode full-size {name} {layout}: oracle")
    tm = x.token_major
    ro, rl = oracle.decode_attn(W.bf16_bits(x.q), W.bf16_bits(tm(x.k_prefix)), W.bf16_bits(tm(x.v_prefix)),
                                W.bf16_bits(tm(x.k_suffix)), W.bf16_bits(tm(x.v_suffix)),
                                x.prefix_start, x.prefix_len, x.suffix_start, x.suffix_len,
                                cfg.group_size, x.scale)
    eo, el = max_abs(o, ro), max_abs(l, rl)
    say(f"decode full-size {name}: out max-abs {eo:.3g}, lse max-abs {el:.3g}")
    assert eo <= ATTN_OUT_TOL and el <= ATTN_LSE_TOL


def _timeline_case(c, D, Hq, Hkv, layout, split=0):
    """rl_debug_decode_timeline against rl_decode_attn on the same inputs: the
    same output and lse bit for bit, and one record per work item of the plan,
    in plan order, with its kind, rows and tokens and ordered timestamps."""
    def kv(bits):
        return to_dev(np.ascontiguousarray(np.transpose(bits, (1, 0, 2))) if layout == "head" else bits)
    t = {k: kv(c[k]) for k in ("k_prefix", "v_prefix", "k_suffix", "v_suffix")}
    q = to_dev(c["q"])
    args = (q, t["k_prefix"], t["v_prefix"], t["k_suffix"], t["v_suffix"], c["prefix_start"], c["prefix_len"],
            c["suffix_start"], c["suffix_len"], c["group_size"])
    scale = 1.0 / math.sqrt(D)
    o0, l0 = rk.decode_attn(*args, scale=scale, split_tokens=split, return_lse=True, kv_layout=layout)
    o1, l1, rec = rk.decode_attn_timeline(*args, scale=scale, split_tokens=split, kv_layout=layout)
    torch.cuda.synchronize()
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16)) and torch.equal(l0, l1)
    items = plan_of(c, Hq, Hkv, D, split)
    r = rec.cpu().numpy()
    assert len(r) == len(items)
    assert (r[:, 6] == np.arange(len(items))).all()
    assert (((r[:, 0] >> 40) & 0xFF) == items["kind"]).all()
    assert (((r[:, 0] >> 48) & 0xFFFF) == items["row_count"]).all()
    assert ((r[:, 5] & 0xFFFFFFFF) == items["tok_count"]).all()
    assert ((r[:, 5] >> 32) == (items["tok_count"] + 63) // 64).all()
    st, first, loop1, en = (r[:, i] for i in range(1, 5))
    assert (st > 0).all() and (st <= first).all() and (first <= loop1).all() and (loop1 <= en).all()
    assert (((r[:, 0] >> 32) & 0xFF) < 8).all()


@pytest.mark.parametrize("layout", ["token", "head"])
def test_timeline_same_outputs_and_records(layout):
    # both split variants: narrow items (one tile in flight) and wide ones (two)
    c = decode_host_case(3, 8, 16, 4, 128, [700, 0, 193], list(np.arange(24) * 37 % 300), seed=71, gap=2)
    _timeline_case(c, 128, 16, 4, layout)
    c = decode_host_case(3, 8, 16, 2, 64, [700, 0, 193],
                         [5, 0, 17, 64, 1, 65, 0, 30, 3, 9, 0, 2, 40, 1, 0, 12, 63, 0, 1, 2, 3, 4, 5, 6], seed=72, gap=2)
    assert set(plan_of(c, 16, 2, 64)["split_variant"]) == {1}
    _timeline_case(c, 64, 16, 2, layout)
