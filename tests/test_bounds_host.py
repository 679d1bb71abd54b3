"""Host replay of the lm-head log-prob kernels' global accesses (no GPU).

rl_debug_logprob_bounds replays every launch of rl_token_logprob (op 0),
rl_token_logprob_backward (op 1) and rl_sample_top_p (op 2), workgroup by
workgroup and lane by lane, with
the arguments the entry points build and the kernels' own index functions, and
checks each load and store against the allocation or workspace section it must
fall in.  The shapes are the ones the bench and the parity tests run (the
8B-class and 32B-class decode-step rows, one full 16384-row backward chunk,
the 262144-row policy pass) plus ragged small shapes replayed at every stage.

A call's accesses depend only on (rows, hidden, vocab) and its own pointers:
neither entry point keeps state between calls, so a sequence of calls (one
forward, then many backward calls at one shape, then at another) is covered by
replaying each shape once.

The shrink checks make one allocation 16 bytes smaller than the entry point
requires: every allocation the kernels use up to its last byte must then
report a violation, which shows that the checker sees overruns and that each
allocation is exactly as large as the kernels need.
"""
import ctypes

import pytest

import paper_2607_20908_amd as rk

_f = rk.lib().rl_debug_logprob_bounds

V = 151936
# (rows, hidden, vocab, every_stage)
SHAPES = [
    (512, 4096, V, 0),        # 8B-class decode step: whole tiles + narrow last round; backward split 8 ways
    (256, 5120, V, 0),        # 32B-class decode step: 594 tiles, the last 82 split 3 ways
    (16384, 5120, V, 0),      # one full backward chunk, unsplit
    (262144, 5120, V, 0),     # policy pass: 16 backward chunks, one-thread-per-row combine
    (300, 128, 1000, 1),      # ragged rows and vocab
    (40000, 64, 700, 1),      # ragged last backward chunk; row combine; split hidden
    (1, 64, 1, 1),            # one row, one vocab entry
    (4097, 192, 77777, 0),    # wave combine; ragged vocab tile
    (8000, 4096, 2500, 0),    # tail parts: 320 tiles, the last 64 split 4 ways over the hidden dimension
    (300, 512, 40000, 1),     # tail parts: 314 tiles, the last 58 split 2 ways; ragged rows and vocab
    (256, 256, 76800, 1),     # too few hidden steps to split: the last 44 tiles as 88 narrow tiles 128 wide
]


def replay(op, rows, hidden, vocab, every=0, shrink=-1):
    return rk.logprob_bounds(op, rows, hidden, vocab, every_stage=bool(every), shrink_region=shrink)


@pytest.mark.parametrize("op", [0, 1], ids=["forward", "backward"])
@pytest.mark.parametrize("rows,hidden,vocab,every", SHAPES)
def test_every_access_inside_its_allocation(op, rows, hidden, vocab, every):
    rep = replay(op, rows, hidden, vocab, every)
    assert rep.accesses > 0 and rep.launches >= 2
    assert rep.violations == 0, rep.first_violation.decode()


def test_backward_launch_count_per_chunk():
    # three launches (probabilities, GEMM, finish) per 16384-row chunk, and
    # two more (tail tiles' hidden parts, their reduce) when the probability
    # pass's last round is split: a full 5120-wide chunk has 594 x 64 tiles,
    # a last round of 128
    assert replay(1, 262144, 5120, V).launches == 5 * 16
    assert replay(1, 40000, 64, 700).launches == 3 * 3
    # 32B-class rows: 594 tiles, the last 82 in 3 parts; 8B-class rows: 1188
    # tiles, a last round of 164 runs whole
    assert replay(1, 256, 5120, V).launches == 5
    assert replay(1, 512, 4096, V).launches == 3
    # the GPU parity tests' split-tail shapes
    assert replay(1, 200, 1024, 75739).launches == 5
    assert replay(1, 300, 512, 40000).launches == 5


def test_forward_launches_follow_the_plan():
    # 8B-class: whole tiles, narrow last round, combine;
    # 8000 x 4096 x 2500 has a hidden-split tail (tile parts + reduce)
    assert replay(0, 512, 4096, V).launches == 3
    assert replay(0, 8000, 4096, 2500).launches == 4


# region indices (in the order the replay allocates them) that the kernels
# use up to their last byte; the parent workspace allocation itself is only
# checked through its sections
FWD_TIGHT = {"hidden": 0, "w_lm": 1, "target": 2, "logprob": 3, "lse": 4, "partial max": 6, "partial sum": 7,
             "target logits": 8}
BWD_TIGHT = {"hidden": 0, "w_lm": 1, "target": 2, "lse": 3, "grad_logprob": 4, "grad_hidden": 5, "probabilities": 7}


@pytest.mark.parametrize("rows,hidden,vocab", [(512, 4096, V), (300, 128, 1000), (8000, 4096, 2500)])
def test_shrunk_allocation_is_caught_forward(rows, hidden, vocab):
    n = replay(0, rows, hidden, vocab).regions
    for name, i in FWD_TIGHT.items():
        rep = replay(0, rows, hidden, vocab, shrink=i)
        assert rep.violations > 0, f"shrinking {name} went unnoticed"
    assert replay(0, rows, hidden, vocab, shrink=5).violations == 0   # the workspace's own extent
    # tail parts exist only with a hidden-split last round
    tail = replay(0, rows, hidden, vocab, shrink=9).violations
    assert (tail > 0) == (rows == 8000)
    assert n == 10


# part: what the section after the probabilities holds (the GEMM's split
# sums, the probability pass's tail parts, both, or nothing)
@pytest.mark.parametrize("rows,hidden,vocab,part", [(512, 4096, V, "splits"), (16384, 5120, V, "tail"),
                                                    (256, 5120, V, "both"), (300, 128, 1000, None),
                                                    (300, 128, 20000, "splits")])
def test_shrunk_allocation_is_caught_backward(rows, hidden, vocab, part):
    rep0 = replay(1, rows, hidden, vocab)
    for name, i in BWD_TIGHT.items():
        rep = replay(1, rows, hidden, vocab, shrink=i)
        assert rep.violations > 0, f"shrinking {name} went unnoticed"
    assert replay(1, rows, hidden, vocab, shrink=6).violations == 0   # the workspace's own extent
    assert rep0.regions == (9 if part else 8)
    if part:
        # the section is as large as the larger user.  Tail parts fill it (256
        # KB each).  The split sums are padded to whole 256-row tiles: used to
        # the last byte only when the rows fill their last tile.
        tight = part != "splits" or rows % 256 == 0
        assert (replay(1, rows, hidden, vocab, shrink=8).violations > 0) == tight


def test_invalid_arguments():
    rep = rk.BoundsReport()
    assert _f(3, 8, 64, 100, 0, -1, ctypes.byref(rep)) == 2          # unknown op
    assert _f(0, 8, 96, 100, 0, -1, ctypes.byref(rep)) == 3          # hidden not a multiple of 64
    assert _f(1, 8, 64, 100, 0, -1, None) == 1
    assert replay(0, 0, 64, 100).launches == 0


# ---------------------------------------------------------------- sampling head
# (rows, hidden, vocab, every_stage)
SAMPLE_SHAPES = [
    (512, 4096, V, 0),        # 8B-class decode step: whole tiles + a narrow last round of 109 x 2 tiles
    (256, 5120, V, 0),        # 32B-class decode step: the last 82 tiles as 163 narrow tiles 128 wide
    (300, 512, 51001, 1),     # 2 row tiles, narrow tiles ending past the vocabulary
    (300, 128, 1000, 1),      # one round, ragged rows and vocab
    (8192 + 300, 64, 300, 1), # two row chunks of logits
    (3, 64, 1 << 21, 0),      # the largest vocabulary
    (1, 64, 1, 1),            # one row, one vocab entry
]


@pytest.mark.parametrize("rows,hidden,vocab,every", SAMPLE_SHAPES)
def test_sampling_accesses_inside_their_allocations(rows, hidden, vocab, every):
    rep = replay(2, rows, hidden, vocab, every)
    assert rep.accesses > 0 and rep.launches >= 2
    assert rep.violations == 0, rep.first_violation.decode()


def test_sampling_launches_follow_the_plan():
    # per chunk of logits: whole tiles, (a narrow last round,) the selection
    assert replay(2, 512, 4096, V).launches == 3
    assert replay(2, 256, 5120, V).launches == 3
    assert replay(2, 300, 128, 1000).launches == 2
    assert replay(2, 8192 + 300, 64, 300).launches == 4


SAMPLE_TIGHT = {"hidden": 0, "w_lm": 1, "inv_temperature": 2, "uniform": 3, "token": 4, "logprob": 5,
                "row maxima": 8}


@pytest.mark.parametrize("rows,hidden,vocab", [(512, 4096, V), (256, 5120, V), (300, 128, 1000), (8192 + 300, 64, 300)])
def test_shrunk_allocation_is_caught_sampling(rows, hidden, vocab):
    assert replay(2, rows, hidden, vocab).regions == 9
    for name, i in SAMPLE_TIGHT.items():
        assert replay(2, rows, hidden, vocab, shrink=i).violations > 0, f"shrinking {name} went unnoticed"
    assert replay(2, rows, hidden, vocab, shrink=6).violations == 0   # the workspace's own extent


# ---------------------------------------------------------------- extend
# rl_debug_extend_bounds replays rl_extend_attn: every work block of the plan,
# every lane, with the arguments the entry point builds and the kernel's own
# index functions (csrc/extend_index.h).
import numpy as np  # noqa: E402

import workloads as W  # noqa: E402


def _packed(lengths):
    s = np.zeros(len(lengths), np.int64)
    s[1:] = np.cumsum(np.asarray(lengths, np.int64))[:-1]
    return s


def _extend(P, G, Hq, Hkv, D, lp, ls, n, layout="head", every=False, shrink=-1, gap=0):
    # sequences packed with `gap` unused rows after each one
    lp, ls, n = (np.asarray(x, np.int32) for x in (lp, ls, n))
    ps = _packed(lp + gap)
    ss = _packed(ls + gap)
    qs = _packed(n + gap)
    return rk.extend_bounds(P, G, Hq, Hkv, D, ps, lp, ss, ls, n, qs, int((lp + gap).sum()), int((ls + gap).sum()),
                            int((n + gap).sum()), kv_layout=layout, every_stage=every, shrink_region=shrink)


def _workload(name):
    cfg = W.DECODE_CONFIGS[name]
    ls = W.suffix_lengths(cfg, 0)
    return (cfg.num_prompts, cfg.group_size, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim,
            np.full(cfg.num_prompts, cfg.prefix_len, np.int32), ls, ls.copy())


def _ragged(seed, P, G, Hq, Hkv, D):
    rng = np.random.Generator(np.random.PCG64(seed))
    lp = rng.integers(0, 300, P)
    lp[0] = 0                                     # a prompt without a prefix
    ls = rng.integers(1, 400, P * G)
    n = np.minimum(ls, rng.integers(0, 300, P * G))
    if len(n) > 2:
        n[1] = 0                                  # a candidate with no new tokens
    n[-1] = ls[-1]                                # the last suffix read to its end
    return P, G, Hq, Hkv, D, lp, ls, n


EXTEND_CASES = [
    ("longctx", "head", False), ("longctx", "token", False), ("8b", "head", False), ("32b", "head", False),
]


@pytest.mark.parametrize("name,layout,every", EXTEND_CASES)
def test_extend_accesses_inside_their_allocations(name, layout, every):
    rep = _extend(*_workload(name), layout=layout, every=every)
    assert rep.accesses > 0 and rep.launches == 1 and rep.regions == 9
    assert rep.violations == 0, rep.first_violation.decode()


@pytest.mark.parametrize("case", [(1, 3, 2, 12, 4, 128), (2, 4, 3, 8, 8, 64), (3, 2, 5, 16, 2, 128),
                                  (4, 1, 1, 128, 1, 128)],
                         ids=["r3", "r1-D64", "r8", "G1-r128"])
@pytest.mark.parametrize("layout", ["head", "token"])
@pytest.mark.parametrize("gap", [0, 5])
def test_extend_ragged_every_tile(case, layout, gap):
    rep = _extend(*_ragged(*case), layout=layout, every=True, gap=gap)
    assert rep.accesses > 0
    assert rep.violations == 0, rep.first_violation.decode()


EXTEND_TIGHT = {"q": 0, "k_prefix": 1, "v_prefix": 2, "k_suffix": 3, "v_suffix": 4, "out": 5, "lse": 6,
                "work list": 8}


@pytest.mark.parametrize("layout", ["head", "token"])
def test_extend_shrunk_allocation_is_caught(layout):
    args = _ragged(3, 2, 5, 16, 2, 128)
    for name, i in EXTEND_TIGHT.items():
        rep = _extend(*args, layout=layout, every=True, shrink=i)
        assert rep.violations > 0, f"shrinking {name} went unnoticed"
    assert _extend(*args, layout=layout, every=True, shrink=7).violations == 0   # the workspace's own extent


def test_extend_bounds_arguments():
    # no new tokens: no work, nothing replayed
    rep = _extend(1, 2, 8, 8, 64, [10], [5, 6], [0, 0])
    assert rep.launches == 0 and rep.accesses == 0
    with pytest.raises(rk.RLError):
        _extend(1, 2, 8, 8, 64, [10], [5, 6], [6, 0])     # more new tokens than the suffix holds
    assert rk.lib().rl_debug_extend_bounds(None, None, 0, -1, None) == 1


# ---------------------------------------------------------------- decode
# rl_debug_decode_bounds replays rl_decode_attn: the work list's upload, every
# item of the split kernel (each tile's buffer descriptor, the item's query
# and partial rows) and every row of the combine, through the kernels' own
# index functions (csrc/decode_index.h).
def _decode(P, G, Hq, Hkv, D, lp, ls, layout="head", split=0, gap=0, shrink=-1):
    lp, ls = np.asarray(lp, np.int32), np.asarray(ls, np.int32)
    return rk.decode_bounds(P, G, Hq, Hkv, D, _packed(lp + gap), lp, _packed(ls + gap), ls, int((lp + gap).sum()),
                            int((ls + gap).sum()), split_tokens=split, kv_layout=layout, shrink_region=shrink)


def _decode_workload(name):
    cfg = W.DECODE_CONFIGS[name]
    return (cfg.num_prompts, cfg.group_size, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim,
            np.full(cfg.num_prompts, cfg.prefix_len, np.int32), W.suffix_lengths(cfg, 0))


def _decode_ragged(seed, P, G, Hq, Hkv, D):
    rng = np.random.Generator(np.random.PCG64(seed))
    lp = rng.integers(1, 700, P)
    lp[0] = 0 if P > 1 else lp[0]                 # a prompt without a prefix
    return P, G, Hq, Hkv, D, lp, rng.integers(1, 900, P * G)


@pytest.mark.parametrize("name", ["tiny", "8b", "32b", "longctx"])
@pytest.mark.parametrize("layout", ["head", "token"])
def test_decode_accesses_inside_their_allocations(name, layout):
    rep = _decode(*_decode_workload(name), layout=layout)
    assert rep.accesses > 0 and rep.launches == 3 and rep.regions == 15
    assert rep.violations == 0, rep.first_violation.decode()


@pytest.mark.parametrize("case", [(1, 3, 2, 12, 4, 128), (2, 4, 3, 8, 8, 64), (3, 2, 40, 64, 8, 128),
                                  (4, 1, 1, 128, 1, 128)],
                         ids=["r3", "r1-D64", "G40-r8-wide", "G1-r128"])
@pytest.mark.parametrize("layout", ["head", "token"])
@pytest.mark.parametrize("split,gap", [(0, 0), (48, 3)])
def test_decode_ragged(case, layout, split, gap):
    rep = _decode(*_decode_ragged(*case), layout=layout, split=split, gap=gap)
    assert rep.accesses > 0
    assert rep.violations == 0, rep.first_violation.decode()


DECODE_TIGHT = {"q": 0, "k_prefix": 1, "v_prefix": 2, "k_suffix": 3, "v_suffix": 4, "out": 5, "lse": 6,
                "work list and unit tables": 8, "work list": 9, "prefix units": 10, "suffix units": 11,
                "partial max": 12, "partial sum": 13, "partial values": 14}


@pytest.mark.parametrize("layout", ["head", "token"])
def test_decode_shrunk_allocation_is_caught(layout):
    args = _decode_ragged(3, 2, 40, 64, 8, 128)
    args = args[:5] + (np.maximum(args[5], 1),) + args[6:]      # every prompt with a prefix
    for name, i in DECODE_TIGHT.items():
        rep = _decode(*args, layout=layout, split=48, shrink=i)
        assert rep.violations > 0, f"shrinking {name} went unnoticed"
    assert _decode(*args, layout=layout, split=48, shrink=7).violations == 0   # the workspace's own extent


def test_decode_bounds_arguments():
    rep = _decode(0, 4, 8, 8, 64, [], [])
    assert rep.launches == 0 and rep.accesses == 0
    with pytest.raises(rk.RLError):
        _decode(1, 2, 8, 3, 64, [4], [5, 6])        # Hq not a multiple of Hkv
    assert rk.lib().rl_debug_decode_bounds(None, None, -1, None) == 1
