"""The C ABI on the host: the library loads, exports what the header declares,
and rejects bad arguments with the documented status before touching the GPU.

No compute call reaches a kernel here: every call either fails validation or
is a valid no-op, so these run without a GPU.  Device pointers are fake,
suitably aligned integers that the library never dereferences on these paths.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2607_20908_amd as rk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rl_kernels.h")

OK, NULLP, SHAPE, UNSUP, MISAL, WSPACE = 0, 1, 2, 3, 4, 5
FAKE = 0x7f0000000000          # 256-byte aligned, never dereferenced


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rl_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_function():
    names = header_functions()
    assert set(names) == set(rk.EXPORTS), names
    lib = ctypes.CDLL(rk.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} not exported"


def test_one_hip_runtime_mapped():
    assert len(rk.hip_runtimes_mapped()) == 1, rk.hip_runtimes_mapped()


def test_status_strings_and_version():
    lib = rk.lib()
    assert lib.rl_abi_version() == 13
    for code, name in rk.STATUS_NAMES.items():
        assert lib.rl_status_string(code).decode() == name
    assert lib.rl_status_string(99).decode() == "RL_ERR_UNKNOWN"


# ---------------------------------------------------------------- decode
def decode_call(P=2, G=3, Hq=4, Hkv=2, D=128, scale=0.125, split=0, lp=None, ls=None,
                prefix_rows=None, suffix_rows=None, ptrs=None, ws=None, ws_bytes=1 << 30,
                null_shape=False, null_lens=False, null_ptrs=False, starts=None, layout=0):
    lib = rk.lib()
    S = P * G
    lp = np.full(P, 5, np.int32) if lp is None else np.asarray(lp, np.int32)
    ls = np.full(S, 3, np.int32) if ls is None else np.asarray(ls, np.int32)
    ps = (np.arange(P, dtype=np.int64) * 5) if starts is None else np.asarray(starts[0], np.int64)
    ss = (np.arange(S, dtype=np.int64) * 3) if starts is None else np.asarray(starts[1], np.int64)
    shape = rk.DecodeShape(P, G, Hq, Hkv, D, scale, split, layout)
    lens = rk.DecodeLens(ps.ctypes.data, lp.ctypes.data, ss.ctypes.data, ls.ctypes.data,
                         5 * P if prefix_rows is None else prefix_rows,
                         3 * S if suffix_rows is None else suffix_rows)
    p = dict(q=FAKE, k_prefix=FAKE + 256, v_prefix=FAKE + 512, k_suffix=FAKE + 768,
             v_suffix=FAKE + 1024, out=FAKE + 1280, lse=FAKE + 1536)
    p.update(ptrs or {})
    dp = rk.DecodePtrs(p["q"], p["k_prefix"], p["v_prefix"], p["k_suffix"], p["v_suffix"],
                       p["out"], p["lse"])
    st = lib.rl_decode_attn(None if null_shape else ctypes.byref(shape),
                            None if null_lens else ctypes.byref(lens),
                            None if null_ptrs else ctypes.byref(dp), ws, ws_bytes, None)
    return st, lib.rl_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(null_shape=True), NULLP),
    (dict(null_lens=True), NULLP),
    (dict(null_ptrs=True), NULLP),
    (dict(ptrs=dict(q=None)), NULLP),
    (dict(ptrs=dict(out=None)), NULLP),
    (dict(ptrs=dict(k_prefix=None)), NULLP),
    (dict(ptrs=dict(v_suffix=None)), NULLP),
    (dict(G=0), SHAPE),
    (dict(P=-1, lp=[], ls=[], starts=([], [])), SHAPE),
    (dict(Hq=6, Hkv=4), SHAPE),
    (dict(Hkv=0), SHAPE),
    (dict(scale=0.0), SHAPE),
    (dict(scale=float("nan")), SHAPE),
    (dict(scale=float("inf")), SHAPE),
    (dict(split=8), SHAPE),
    (dict(split=40), SHAPE),
    (dict(split=-16), SHAPE),
    (dict(lp=[5, -1]), SHAPE),
    (dict(ls=[3, 3, -2, 3, 3, 3]), SHAPE),
    (dict(prefix_rows=9), SHAPE),             # prompt 1 needs rows [5, 10)
    (dict(suffix_rows=17), SHAPE),            # candidate 5 needs rows [15, 18)
    (dict(prefix_rows=-1), SHAPE),
    (dict(starts=([0, -5], [0, 3, 6, 9, 12, 15])), SHAPE),
    (dict(layout=2), SHAPE),
    (dict(layout=-1), SHAPE),
    (dict(D=96), UNSUP),
    (dict(D=256), UNSUP),
    (dict(D=0), SHAPE),
    (dict(Hq=258, Hkv=2), UNSUP),             # Hq/Hkv = 129 > 128
    (dict(Hq=514, Hkv=257), UNSUP),           # more than 256 kv heads (the work item holds 8 bits)
    (dict(G=129, Hq=256, Hkv=2, ls=np.full(258, 3)), UNSUP),   # G * Hq/Hkv = 16512 > 16384 rows
    (dict(prefix_rows=1 << 32), UNSUP),       # KV rows are 32-bit in the work list
    (dict(suffix_rows=1 << 32), UNSUP),
    (dict(ptrs=dict(q=FAKE + 8)), MISAL),
    (dict(ptrs=dict(v_prefix=FAKE + 2)), MISAL),
    (dict(ptrs=dict(out=FAKE + 4)), MISAL),
    (dict(ptrs=dict(lse=FAKE + 2)), MISAL),
    (dict(ws=None), WSPACE),
    (dict(ws=FAKE, ws_bytes=64), WSPACE),
])
def test_decode_validation(kw, expect):
    kw.setdefault("ws", FAKE)
    st, msg = decode_call(**kw)
    assert st == expect, (st, msg)
    assert msg, "a failing call must leave an error message"


def test_decode_split_above_item_limit():
    """A forced split above 16384 tokens acts as 16384 (items may cover fewer
    tokens than the bound): a 40000-token prefix becomes 3 chunks."""
    lp = np.array([40000], np.int32)
    ls = np.array([20, 0], np.int32)
    it = rk.decode_plan(1, 2, 4, 2, 128, np.array([0], np.int64), lp, np.array([0, 20], np.int64), ls,
                        40000, 20, split_tokens=32768)
    pre = it[it["kind"] == 0]
    assert pre["tok_count"].max() <= 16384
    for kh in range(2):
        mine = np.sort(pre[pre["kv_head"] == kh], order="tok_begin")
        assert len(mine) == 3 and mine["tok_count"].sum() == 40000
        assert np.array_equal(mine["tok_begin"][1:], np.cumsum(mine["tok_count"])[:-1])


def test_decode_empty_batch_is_noop():
    st, msg = decode_call(P=0, ws=None)
    assert st == OK and msg == ""
    # nullable pointers: no prefix anywhere -> prefix pointers may be NULL, but the
    # call then proceeds to the workspace check (no device work before it)
    st, _ = decode_call(lp=[0, 0], ptrs=dict(k_prefix=None, v_prefix=None), ws=None)
    assert st == WSPACE


def test_decode_workspace_size_queries():
    args = (2, 3, 4, 2, 128, np.array([0, 5]), np.array([5, 5]), np.arange(6) * 3,
            np.full(6, 3), 10, 18)
    n = rk.decode_attn_workspace_size(*args)
    assert n > 0 and n % 256 == 0
    assert rk.decode_attn_workspace_size(*args) == n               # deterministic
    with pytest.raises(rk.RLError) as e:
        rk.decode_attn_workspace_size(2, 3, 4, 2, 96, *args[5:])
    assert e.value.status == UNSUP
    assert rk.decode_attn_workspace_size(0, 3, 4, 2, 128, [], [], [], [], 0, 0) == 0


# --------------------------------------------------------------- logprob
def logprob_call(R=8, H=256, V=1000, hs=FAKE, w=FAKE + 256, t=FAKE + 512, invT=1.0,
                 lp=FAKE + 768, lse=FAKE + 1024, ws=FAKE, ws_bytes=1 << 30):
    lib = rk.lib()
    st = lib.rl_token_logprob(R, H, V, hs, w, t, invT, lp, lse, ws, ws_bytes, None)
    return st, lib.rl_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(hs=None), NULLP),
    (dict(w=None), NULLP),
    (dict(t=None), NULLP),
    (dict(lp=None), NULLP),
    (dict(R=-1), SHAPE),
    (dict(H=0), SHAPE),
    (dict(V=0), SHAPE),
    (dict(V=-5), SHAPE),
    (dict(invT=0.0), SHAPE),
    (dict(invT=-1.0), SHAPE),
    (dict(invT=float("nan")), SHAPE),
    (dict(H=100), UNSUP),
    (dict(H=(1 << 22) + 64), UNSUP),      # 32-bit byte offsets within a tile's rows
    (dict(H=32), UNSUP),
    (dict(hs=FAKE + 8), MISAL),
    (dict(w=FAKE + 4), MISAL),
    (dict(t=FAKE + 2), MISAL),
    (dict(lp=FAKE + 1), MISAL),
    (dict(lse=FAKE + 2), MISAL),
    (dict(ws=None), WSPACE),
    (dict(ws_bytes=16), WSPACE),
    (dict(ws=FAKE + 4), MISAL),
])
def test_logprob_validation(kw, expect):
    st, msg = logprob_call(**kw)
    assert st == expect, (st, msg)
    assert msg


def test_logprob_empty_is_noop():
    st, msg = logprob_call(R=0, hs=None, w=None, t=None, lp=None, lse=None, ws=None, ws_bytes=0)
    assert st == OK and msg == ""


def tail_part_bytes(R, H, V, cus=256, max_splits=4):
    """fp32 accumulators of the hidden-dimension parts of a short last round
    of 256 x 256 tiles (at most half the CUs busy): tail x splits x 256 KB."""
    tiles = -(-V // 256) * -(-R // 256)
    dp, tail = tiles // cus * cus, tiles % cus
    if dp == 0 or tail == 0 or 2 * tail > cus:
        return 0
    s = min(max_splits, cus // tail, H // 64 // 4)
    if s < 2:
        return 0
    return tail * s * 256 * 256 * 4


def narrow_tiles(R, H, V, cus=256, split=True):
    """(whole vocab tiles before the narrow region, narrow tiles per row
    tile) when a partial last round of 256 x 256 tiles runs as one round of
    128-wide tiles, or else 192-wide ones (at most 4 row tiles, the narrower
    that fits), else None.  split: the forward, which splits a tail of at
    most half a round over the hidden dimension instead when it can."""
    nrt = -(-R // 256)
    tiles = -(-V // 256) * nrt
    dp, tail = tiles // cus * cus, tiles % cus
    if dp == 0 or tail == 0 or (split and tail_part_bytes(R, H, V)) or nrt > 4:
        return None
    vt0 = dp // nrt
    for width in (128, 192):
        n = -(-(V - vt0 * 256) // width)
        if n * nrt <= cus:
            return (vt0, n)
    return None


def test_logprob_workspace_size():
    # per (partial slot, row): max and sum, one slot per vocab tile (the
    # narrow tiles of a last round have their own); per row: the target
    # logit; the tail's partial accumulators when the last round is split
    for R, H, V in ((1000, 5120, 151936), (256, 5120, 151936), (512, 4096, 151936), (40, 64, 1000),
                    (256, 256, 76800), (262144, 5120, 151936), (300, 512, 51001), (600, 512, 35700),
                    (1000, 512, 25500)):
        n = rk.token_logprob_workspace_size(R, H, V)
        nt = narrow_tiles(R, H, V)
        slots = -(-V // 256) if nt is None else nt[0] + nt[1]
        base = (2 * slots * R + R) * 4 + tail_part_bytes(R, H, V)
        assert base <= n < base + 3 * 256, (R, H, V)
    # the 8B-class step (1188 tiles: 4 rounds + 164) runs its last round as
    # 109 x 2 tiles 192 wide over vocab [131072, 151936); the 32B-class one
    # (594 tiles: 2 rounds + 82) splits its tail instead; the policy pass
    # has no partial round; 5 row tiles are too many for narrow tiles
    assert narrow_tiles(512, 4096, 151936) == (512, 109)
    assert narrow_tiles(256, 5120, 151936) is None
    assert narrow_tiles(262144, 5120, 151936) is None
    assert narrow_tiles(300, 512, 51001) == (128, 95)
    assert narrow_tiles(600, 512, 35700) == (85, 73)      # 255 whole tiles: 85 per row tile
    assert narrow_tiles(1000, 512, 25500) == (64, 48)
    assert narrow_tiles(1200, 512, 20000) is None         # 5 row tiles
    assert narrow_tiles(200, 512, 55000) is None          # 215 tiles: no full round
    # a tail too short in hidden steps to split: 44 tiles as 88 tiles 128 wide
    assert narrow_tiles(256, 256, 76800) == (256, 88)
    # the sampling head never splits: at 32B-class rows its 82-tile tail runs
    # as 163 tiles 128 wide (20864 entries)
    assert narrow_tiles(256, 5120, 151936, split=False) == (512, 163)
    # the 32B-class decode step (594 tiles: 2 rounds + 82) splits its tail
    # 3 ways; the 8B-class one (1188 tiles: 4 rounds + 164) does not split
    assert tail_part_bytes(256, 5120, 151936) == 82 * 3 * 256 * 256 * 4
    assert tail_part_bytes(512, 4096, 151936) == 0
    assert tail_part_bytes(256, 256, 76800) == 0      # too few hidden steps
    assert tail_part_bytes(256, 768, 66048) == 2 * 3 * 256 * 256 * 4   # 12 hidden steps: 3 parts
    assert rk.token_logprob_workspace_size(0, 64, 10) == 0
    with pytest.raises(rk.RLError):
        rk.token_logprob_workspace_size(4, 100, 10)


def test_binding_refuses_host_tensors():
    import torch
    x = torch.zeros(4, 64, dtype=torch.bfloat16)
    w = torch.zeros(8, 64, dtype=torch.bfloat16)
    t = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(ValueError, match="device tensor"):
        rk.token_logprob(x, w, t)


# ------------------------------------------------------------------ GRPO
def grpo_adv_call(P=4, G=8, r=FAKE, a=FAKE + 256):
    lib = rk.lib()
    st = lib.rl_grpo_advantage(P, G, r, a, None)
    return st, lib.rl_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(r=None), NULLP),
    (dict(a=None), NULLP),
    (dict(P=-1), SHAPE),
    (dict(G=0), SHAPE),
    (dict(G=-3), SHAPE),
    (dict(G=1025), UNSUP),
    (dict(r=FAKE + 2), MISAL),
    (dict(a=FAKE + 1), MISAL),
])
def test_grpo_advantage_validation(kw, expect):
    st, msg = grpo_adv_call(**kw)
    assert st == expect, (st, msg)
    assert msg


def test_grpo_advantage_empty_is_noop():
    st, msg = grpo_adv_call(P=0, r=None, a=None)
    assert st == OK and msg == ""


def grpo_sur_call(R=100, P=4, G=8, new=FAKE, old=FAKE + 1024, seq=FAKE + 2048, adv=FAKE + 4096,
                  eps=0.2, loss=FAKE + 8192, grad=FAKE + 8448, ws=FAKE + 16384, ws_bytes=1 << 20):
    lib = rk.lib()
    st = lib.rl_grpo_surrogate(R, P, G, new, old, seq, adv, eps, loss, grad, ws, ws_bytes, None)
    return st, lib.rl_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(new=None), NULLP),
    (dict(old=None), NULLP),
    (dict(seq=None), NULLP),
    (dict(adv=None), NULLP),
    (dict(loss=None), NULLP),
    (dict(grad=None), NULLP),
    (dict(R=-1), SHAPE),
    (dict(P=-2), SHAPE),
    (dict(G=0), SHAPE),
    (dict(eps=-0.1), SHAPE),
    (dict(eps=1.0), SHAPE),
    (dict(eps=float("inf")), SHAPE),
    (dict(eps=float("nan")), SHAPE),
    (dict(new=FAKE + 2), MISAL),
    (dict(seq=FAKE + 2049), MISAL),
    (dict(grad=FAKE + 8450), MISAL),
    (dict(ws=None), WSPACE),
    (dict(ws_bytes=16), WSPACE),
    (dict(ws=FAKE + 16388), MISAL),
])
def test_grpo_surrogate_validation(kw, expect):
    st, msg = grpo_sur_call(**kw)
    assert st == expect, (st, msg)
    assert msg


def test_grpo_surrogate_workspace_size():
    # one int32 count per candidate, one fp64 partial per 256 rows
    for R, P, G in [(262144, 4, 16), (0, 0, 1), (1, 1, 1), (1000, 4096, 16)]:
        n = rk.grpo_surrogate_workspace_size(R, P, G)
        assert n >= P * G * 4 + -(-R // 256) * 8
        assert n % 256 == 0 and n > 0
        assert n <= P * G * 4 + -(-R // 256) * 8 + 512
    with pytest.raises(rk.RLError):
        rk.grpo_surrogate_workspace_size(-1, 1, 1)
    with pytest.raises(rk.RLError):
        rk.grpo_surrogate_workspace_size(1, 1 << 30, 16)


# ------------------------------------------------------- log-prob backward
def logprob_bwd_call(R=8, H=256, V=1000, hs=FAKE, w=FAKE + 256, t=FAKE + 512, invT=1.0,
                     lse=FAKE + 768, g=FAKE + 1024, dh=FAKE + 2048, ws=FAKE, ws_bytes=1 << 30):
    lib = rk.lib()
    st = lib.rl_token_logprob_backward(R, H, V, hs, w, t, invT, lse, g, dh, ws, ws_bytes, None)
    return st, lib.rl_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(hs=None), NULLP),
    (dict(w=None), NULLP),
    (dict(t=None), NULLP),
    (dict(lse=None), NULLP),
    (dict(g=None), NULLP),
    (dict(dh=None), NULLP),
    (dict(R=-1), SHAPE),
    (dict(H=0), SHAPE),
    (dict(V=0), SHAPE),
    (dict(invT=0.0), SHAPE),
    (dict(invT=float("inf")), SHAPE),
    (dict(H=100), UNSUP),
    (dict(H=(1 << 22) + 64), UNSUP),      # 32-bit byte offsets within a tile's rows
    (dict(hs=FAKE + 8), MISAL),
    (dict(w=FAKE + 4), MISAL),
    (dict(dh=FAKE + 2056), MISAL),
    (dict(t=FAKE + 2), MISAL),
    (dict(lse=FAKE + 1), MISAL),
    (dict(g=FAKE + 2), MISAL),
    (dict(ws=None), WSPACE),
    (dict(ws_bytes=16), WSPACE),
    (dict(ws=FAKE + 4), MISAL),
])
def test_logprob_backward_validation(kw, expect):
    st, msg = logprob_bwd_call(**kw)
    assert st == expect, (st, msg)
    assert msg


def test_logprob_backward_empty_is_noop():
    st, msg = logprob_bwd_call(R=0, hs=None, w=None, t=None, lse=None, g=None, dh=None, ws=None, ws_bytes=0)
    assert st == OK and msg == ""


def test_logprob_backward_workspace_size():
    V = 151936
    vpad = -(-V // 256) * 256
    part = 256 * 256 * 4                 # one hidden-dimension part of a tail tile
    # one chunk of probabilities (at most 16384 rows, padded to 256) in bf16;
    # a full chunk has 594 x 64 tiles, whose last round of 128 tiles runs as
    # 2 hidden-dimension parts each
    for R, H in [(262144, 5120), (16384, 5120), (20000, 4096)]:
        n = rk.token_logprob_backward_workspace_size(R, H, V)
        assert n == 16384 * vpad * 2 + 128 * 2 * part
    # 8B-class rows: the vocabulary is split and fp32 partial sums follow
    # (1188 tiles, a last round of 164 runs whole: no tail parts)
    n = rk.token_logprob_backward_workspace_size(512, 4096, V)
    probs = 512 * vpad * 2
    assert n > probs and (n - probs) % (512 * 4096 * 4) == 0
    # 32B-class rows: the split sums (12 x 256 x 5120 fp32) and the tail
    # parts (82 tiles x 3) share one section, as large as the larger
    n = rk.token_logprob_backward_workspace_size(256, 5120, V)
    assert n == 256 * vpad * 2 + max(12 * 256 * 5120 * 4, 82 * 3 * part)
    assert rk.token_logprob_backward_workspace_size(0, 64, 10) == 0
    with pytest.raises(rk.RLError):
        rk.token_logprob_backward_workspace_size(4, 100, 10)


# ---------------------------------------------------------- sampling head
def sample_call(R=8, H=256, V=1000, hs=FAKE, w=FAKE + 256, it=FAKE + 512, top_p=0.9, u=FAKE + 768,
                tok=FAKE + 1024, lp=FAKE + 1280, ws=FAKE, ws_bytes=1 << 30):
    lib = rk.lib()
    st = lib.rl_sample_top_p(R, H, V, hs, w, it, top_p, u, tok, lp, ws, ws_bytes, None)
    return st, lib.rl_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(hs=None), NULLP),
    (dict(w=None), NULLP),
    (dict(it=None), NULLP),
    (dict(u=None), NULLP),
    (dict(tok=None), NULLP),
    (dict(R=-1), SHAPE),
    (dict(H=0), SHAPE),
    (dict(V=0), SHAPE),
    (dict(top_p=0.0), SHAPE),
    (dict(top_p=-0.5), SHAPE),
    (dict(top_p=1.5), SHAPE),
    (dict(top_p=float("nan")), SHAPE),
    (dict(H=100), UNSUP),
    (dict(H=(1 << 22) + 64), UNSUP),      # 32-bit byte offsets within a tile's rows
    (dict(V=(1 << 21) + 1), UNSUP),
    (dict(hs=FAKE + 8), MISAL),
    (dict(w=FAKE + 4), MISAL),
    (dict(it=FAKE + 2), MISAL),
    (dict(u=FAKE + 1), MISAL),
    (dict(tok=FAKE + 2), MISAL),
    (dict(lp=FAKE + 3), MISAL),
    (dict(ws=None), WSPACE),
    (dict(ws_bytes=16), WSPACE),
    (dict(ws=FAKE + 4), MISAL),
])
def test_sample_validation(kw, expect):
    st, msg = sample_call(**kw)
    assert st == expect, (st, msg)
    assert msg


def test_sample_logprob_optional_and_empty():
    st, msg = sample_call(R=0, hs=None, w=None, it=None, u=None, tok=None, lp=None, ws=None, ws_bytes=0)
    assert st == OK and msg == ""


def test_sample_workspace_size():
    V = 151936
    tiles = -(-V // 256)
    ld = (tiles + 1) * 256      # one tile of padding: narrow tiles end up to 191 entries past V
    # fp32 logits of up to 8192 rows (padded to 256) and their per-tile maxima;
    # at 512 rows the last round runs as 109 x 2 narrow tiles: 512 + 109 slots
    slots = 512 + 109
    assert narrow_tiles(512, 4096, V) == (512, 109)
    n = rk.sample_top_p_workspace_size(512, 4096, V)
    assert n >= 512 * ld * 4 + slots * 512 * 4 and n < 512 * ld * 4 + slots * 512 * 4 + 512
    # at 256 rows, 163 tiles 128 wide: 512 + 163 slots
    assert narrow_tiles(256, 5120, V, split=False) == (512, 163)
    n = rk.sample_top_p_workspace_size(256, 5120, V)
    slots = 512 + 163
    assert n >= 256 * ld * 4 + slots * 256 * 4 and n < 256 * ld * 4 + slots * 256 * 4 + 512
    assert rk.sample_top_p_workspace_size(100000, 4096, V) == rk.sample_top_p_workspace_size(8192, 4096, V)
    assert rk.sample_top_p_workspace_size(0, 64, 10) == 0


# -------------------------------------------------------------- KV append
def append_call(S=4, G=2, Hkv=2, D=128, ss=None, sl=None, cap=None, ns=None, nl=None, suffix_rows=64,
                new_rows=8, layout=0, ptrs=True, ws=FAKE, ws_bytes=1 << 20):
    lib = rk.lib()
    ss = np.arange(S, dtype=np.int64) * 16 if ss is None else np.asarray(ss, np.int64)
    sl = np.full(S, 3, np.int32) if sl is None else np.asarray(sl, np.int32)
    ns = np.arange(S, dtype=np.int64) * 2 if ns is None else np.asarray(ns, np.int64)
    nl = np.full(S, 2, np.int32) if nl is None else np.asarray(nl, np.int32)
    capa = None if cap is None else np.asarray(cap, np.int32)
    shape = rk.DecodeShape(S // G, G, 1, Hkv, D, 1.0, 0, layout)
    lens = rk.KvAppendLens(ss.ctypes.data, sl.ctypes.data, None if capa is None else capa.ctypes.data,
                           ns.ctypes.data, nl.ctypes.data, suffix_rows, new_rows)
    p = [FAKE, FAKE + 4096, FAKE + 8192, FAKE + 12288] if ptrs is True else ptrs
    st = lib.rl_kv_append(ctypes.byref(shape), ctypes.byref(lens), *p, ws, ws_bytes, None)
    return st, lib.rl_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(ptrs=[None, FAKE, FAKE, FAKE]), NULLP),
    (dict(ptrs=[FAKE, FAKE, FAKE, None]), NULLP),
    (dict(sl=[3, -1, 3, 3]), SHAPE),
    (dict(nl=[2, 2, -2, 2]), SHAPE),
    (dict(ss=[0, 16, 32, 62]), SHAPE),                 # 62 + 3 + 2 > 64 rows
    (dict(cap=[8, 8, 4, 8]), SHAPE),                   # 3 + 2 > 4
    (dict(ns=[0, 2, 4, 7]), SHAPE),                    # 7 + 2 > 8 new rows
    (dict(ss=[0, 1, 32, 48], sl=[3, 3, 3, 3]), SHAPE), # rows 3-4 and 4-5 overlap
    (dict(D=96), UNSUP),
    (dict(layout=2), SHAPE),
    (dict(ptrs=[FAKE + 8, FAKE, FAKE, FAKE]), MISAL),
    (dict(ws=None), WSPACE),
    (dict(ws_bytes=16), WSPACE),
    (dict(ws=FAKE + 4), MISAL),
])
def test_kv_append_validation(kw, expect):
    st, msg = append_call(**kw)
    assert st == expect, (st, msg)
    assert msg


def test_kv_append_nothing_to_do():
    st, msg = append_call(nl=[0, 0, 0, 0], ptrs=[None, None, None, None], ws=None, ws_bytes=0)
    assert st == OK and msg == ""


# ---------------------------------------------------------------- extend
def extend_call(P=2, G=2, Hq=4, Hkv=2, D=128, scale=0.125, lp=None, ls=None, nl=None, qs=None,
                prefix_rows=None, suffix_rows=None, q_rows=None, ptrs=None, ws=None, ws_bytes=1 << 30,
                null_shape=False, null_lens=False, null_ptrs=False, layout=0, size_only=False):
    lib = rk.lib()
    S = P * G
    lp = np.full(P, 5, np.int32) if lp is None else np.asarray(lp, np.int32)
    ls = np.full(S, 4, np.int32) if ls is None else np.asarray(ls, np.int32)
    nl = np.full(S, 2, np.int32) if nl is None else np.asarray(nl, np.int32)
    qs = (np.arange(S, dtype=np.int64) * 2) if qs is None else np.asarray(qs, np.int64)
    ps = np.arange(P, dtype=np.int64) * 5
    ss = np.arange(S, dtype=np.int64) * 4
    shape = rk.DecodeShape(P, G, Hq, Hkv, D, scale, 0, layout)
    lens = rk.ExtendLens(ps.ctypes.data, lp.ctypes.data, ss.ctypes.data, ls.ctypes.data, nl.ctypes.data,
                         qs.ctypes.data, 5 * P if prefix_rows is None else prefix_rows,
                         4 * S if suffix_rows is None else suffix_rows, 2 * S if q_rows is None else q_rows)
    if size_only:
        n = ctypes.c_size_t(0)
        st = lib.rl_extend_attn_workspace_size(ctypes.byref(shape), ctypes.byref(lens), ctypes.byref(n))
        return st, n.value
    p = dict(q=FAKE, k_prefix=FAKE + 256, v_prefix=FAKE + 512, k_suffix=FAKE + 768,
             v_suffix=FAKE + 1024, out=FAKE + 1280, lse=FAKE + 1536)
    p.update(ptrs or {})
    dp = rk.DecodePtrs(p["q"], p["k_prefix"], p["v_prefix"], p["k_suffix"], p["v_suffix"], p["out"], p["lse"])
    st = lib.rl_extend_attn(None if null_shape else ctypes.byref(shape), None if null_lens else ctypes.byref(lens),
                            None if null_ptrs else ctypes.byref(dp), ws, ws_bytes, None)
    return st, lib.rl_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(null_shape=True), NULLP),
    (dict(null_lens=True), NULLP),
    (dict(null_ptrs=True), NULLP),
    (dict(ptrs=dict(q=None)), NULLP),
    (dict(ptrs=dict(out=None)), NULLP),
    (dict(ptrs=dict(k_suffix=None)), NULLP),
    (dict(ptrs=dict(v_prefix=None)), NULLP),
    (dict(G=0), SHAPE),
    (dict(Hq=6, Hkv=4), SHAPE),
    (dict(scale=0.0), SHAPE),
    (dict(layout=3), SHAPE),
    (dict(nl=[2, 2, 5, 2]), SHAPE),          # more new tokens than the suffix holds
    (dict(nl=[2, -1, 2, 2]), SHAPE),
    (dict(qs=[0, 2, 3, 6]), SHAPE),          # candidates 1 and 2 share query row 3
    (dict(qs=[0, 2, 4, 7]), SHAPE),          # candidate 3 needs rows [7, 9) of 8
    (dict(qs=[-1, 2, 4, 6]), SHAPE),
    (dict(q_rows=-1), SHAPE),
    (dict(prefix_rows=9), SHAPE),
    (dict(suffix_rows=15), SHAPE),
    (dict(ls=[4, 4, -1, 4], nl=[2, 2, 0, 2]), SHAPE),
    (dict(D=96), UNSUP),
    (dict(ptrs=dict(q=FAKE + 8)), MISAL),
    (dict(ptrs=dict(k_prefix=FAKE + 4)), MISAL),
    (dict(ptrs=dict(lse=FAKE + 2)), MISAL),
    (dict(ws=None), WSPACE),
    (dict(ws=FAKE, ws_bytes=64), WSPACE),
    (dict(ws=FAKE + 8), MISAL),
])
def test_extend_validation(kw, expect):
    kw.setdefault("ws", FAKE)
    st, msg = extend_call(**kw)
    assert st == expect, (st, msg)
    assert msg, "a failing call must leave an error message"


def test_extend_noops_and_sizes():
    # no new tokens anywhere: valid, nothing enqueued, no workspace needed
    st, msg = extend_call(nl=[0, 0, 0, 0], ws=None, ptrs=dict(q=None, out=None))
    assert st == OK and msg == ""
    st, msg = extend_call(P=0, lp=[], ls=[], nl=[], qs=[], ws=None)
    assert st == OK and msg == ""
    # no prefix at all: the prefix pointers may be NULL
    st, n = extend_call(lp=[0, 0], prefix_rows=0, size_only=True)
    assert st == OK
    # 48 bytes per block of 256 query rows, rounded up to 256: 4 candidates x 2 kv heads x 1 block
    st, n = extend_call(size_only=True)
    assert st == OK and n == 512
    st, n = extend_call(Hq=8, Hkv=1, ls=[200] * 4, nl=[100] * 4, qs=[0, 100, 200, 300], suffix_rows=800,
                        q_rows=400, size_only=True)
    assert st == OK and n == ((4 * 4 * 48 + 255) // 256) * 256   # 100 tokens x 8 heads = 4 blocks each


# ---------------------------------------------------------------- no-alloc variant
def test_noalloc_validation_before_any_hip_call():
    lib = rk.lib()
    fake = ctypes.c_void_p(1 << 20)
    # rows 0: a valid no-op
    assert lib.rl_token_logprob_noalloc(0, 64, 100, None, None, None, 1.0, None, None, None) == 0
    # NULL target
    assert lib.rl_token_logprob_noalloc(4, 64, 100, fake, fake, None, 1.0, fake, None, None) == 1
    # hidden not a multiple of 64
    assert lib.rl_token_logprob_noalloc(4, 96, 100, fake, fake, fake, 1.0, fake, None, None) == 3
    # a workspace larger than the static scratch
    R, H, V = 65536, 64, 151936
    assert rk.token_logprob_workspace_size(R, H, V) > rk.NOALLOC_SCRATCH_BYTES
    assert lib.rl_token_logprob_noalloc(R, H, V, fake, fake, fake, 1.0, fake, fake, None) == 3
    assert b"scratch" in lib.rl_last_error()
    # the 8B-class and 32B-class decode-step rows fit
    assert rk.token_logprob_workspace_size(512, 4096, 151936) <= rk.NOALLOC_SCRATCH_BYTES
    assert rk.token_logprob_workspace_size(256, 5120, 151936) <= rk.NOALLOC_SCRATCH_BYTES


# ---------------------------------------------------------------- tile timeline (debug)
def test_timeline_size_query_and_validation():
    lib = rk.lib()
    n = ctypes.c_int64(-1)
    fake = ctypes.c_void_p(FAKE)
    # size query: no pointer but num_records is looked at, nothing launched
    for R, H, V in [(256, 5120, 151936), (512, 4096, 151936), (300, 128, 20000), (8, 256, 1024)]:
        assert lib.rl_debug_logprob_timeline(R, H, V, None, None, None, 1.0, None, None, None, 0, None, 0,
                                             ctypes.byref(n), None) == OK
        assert n.value > 0 and n.value % 8 == 0            # 8 waves per tile workgroup
        assert rk.logprob_timeline_records(R, H, V) == n.value
    # one 256-row tile per 256 vocab entries: every tile covered once, whole or in parts
    assert rk.logprob_timeline_records(256, 5120, 151936) >= 8 * 594
    assert lib.rl_debug_logprob_timeline(256, 5120, 151936, None, None, None, 1.0, None, None, None, 0, None, 0,
                                         None, None) == NULLP
    assert lib.rl_debug_logprob_timeline(8, 96, 1024, None, None, None, 1.0, None, None, None, 0, None, 0,
                                         ctypes.byref(n), None) == UNSUP
    need = rk.logprob_timeline_records(8, 256, 1024)
    ws = rk.token_logprob_workspace_size(8, 256, 1024)
    args = (8, 256, 1024, fake, fake, fake, 1.0, fake, fake, fake, ws)
    assert lib.rl_debug_logprob_timeline(*args, ctypes.c_void_p(FAKE), need - 1, ctypes.byref(n), None) == WSPACE
    assert lib.rl_debug_logprob_timeline(*args, ctypes.c_void_p(FAKE + 4), need, ctypes.byref(n), None) == MISAL
    assert lib.rl_debug_logprob_timeline(8, 256, 1024, fake, fake, None, 1.0, fake, fake, fake, ws,
                                         ctypes.c_void_p(FAKE), need, ctypes.byref(n), None) == NULLP


def test_decode_timeline_size_query_and_validation():
    lib = rk.lib()
    P, G, Hq, Hkv, D = 3, 8, 16, 2, 64
    lp = np.array([700, 0, 193], np.int32)
    ls = np.array([5, 0, 17, 64, 1, 65, 0, 30, 3, 9, 0, 2, 40, 1, 0, 12, 63, 0, 1, 2, 3, 4, 5, 6], np.int32)
    ps = np.concatenate([[0], np.cumsum(lp)[:-1]]).astype(np.int64)
    ss = np.concatenate([[0], np.cumsum(ls)[:-1]]).astype(np.int64)
    a = rk._DecodeArgs(P, G, Hq, Hkv, D, 0.125, 0, ps, lp, ss, ls, int(lp.sum()), int(ls.sum()))
    n = ctypes.c_int64(-1)
    # size query: planning only, no pointer looked at
    assert lib.rl_debug_decode_timeline(ctypes.byref(a.shape), ctypes.byref(a.lens), None, None, 0, None, 0,
                                        ctypes.byref(n), None) == OK
    items = rk.decode_plan(P, G, Hq, Hkv, D, ps, lp, ss, ls, int(lp.sum()), int(ls.sum()), scale=0.125)
    assert n.value == len(items) > 0
    assert lib.rl_debug_decode_timeline(ctypes.byref(a.shape), ctypes.byref(a.lens), None, None, 0, None, 0,
                                        None, None) == NULLP
    fake = ctypes.c_void_p(FAKE)
    ptrs = rk.DecodePtrs(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None)
    need = ctypes.c_size_t(0)
    assert lib.rl_decode_attn_workspace_size(ctypes.byref(a.shape), ctypes.byref(a.lens), ctypes.byref(need)) == OK
    call = lambda rec, cap: lib.rl_debug_decode_timeline(ctypes.byref(a.shape), ctypes.byref(a.lens),
                                                         ctypes.byref(ptrs), fake, need.value, rec, cap,
                                                         ctypes.byref(n), None)
    assert call(ctypes.c_void_p(FAKE), len(items) - 1) == WSPACE
    assert call(ctypes.c_void_p(FAKE + 4), len(items)) == MISAL
    bad = rk.DecodePtrs(FAKE, FAKE, FAKE, None, FAKE, FAKE, None)      # NULL k_suffix
    assert lib.rl_debug_decode_timeline(ctypes.byref(a.shape), ctypes.byref(a.lens), ctypes.byref(bad), fake,
                                        need.value, ctypes.c_void_p(FAKE), len(items), ctypes.byref(n),
                                        None) == NULLP
