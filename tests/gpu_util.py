"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import workloads as W

ATTN_OUT_TOL = 1e-2     # max-abs on the attention output (bf16 inputs, fp32 accumulation)
ATTN_LSE_TOL = 1e-3     # max-abs on the attention log-sum-exp
LOGPROB_TOL = 2e-3      # max-abs on log-probs and on their log-sum-exp


def say(*a):
    """Name the case before a GPU step, flushed, so a failing run shows what ran."""
    print(*a, flush=True)
    sys.stdout.flush()


def dev():
    return torch.device("cuda:0")


def to_dev(bits: np.ndarray) -> torch.Tensor:
    return W.bits_to_bf16(bits, dev())


def max_abs(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape
    if a.size == 0:
        return 0.0
    # equal infinities and NaN on both sides (e.g. an invalid target) agree
    same = (np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))) | (np.isnan(a) & np.isnan(b))
    with np.errstate(invalid="ignore"):
        d = np.where(same, 0.0, np.abs(a - b))
    return float(np.nan_to_num(d, nan=np.inf).max())


def decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=0, qmul=1.0, gap=0, poison=False):
    """Random bf16 decode inputs as host bit arrays with `gap` rows between sequences.

    With poison=True the gap rows (never part of any range) hold NaN, so a read
    outside a valid range shows up in the output.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    lp = np.asarray(lp, np.int32)
    ls = np.asarray(ls, np.int32)
    S = P * G
    ps = np.zeros(P, np.int64)
    ss = np.zeros(S, np.int64)
    pos = gap
    for p in range(P):
        ps[p] = pos
        pos += int(lp[p]) + gap
    prow = max(pos, 1)
    pos = gap
    for s in range(S):
        ss[s] = pos
        pos += int(ls[s]) + gap
    srow = max(pos, 1)

    def randbits(shape, mul=1.0):
        x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32) * mul)
        return W.bf16_bits(x.to(torch.bfloat16))

    q = randbits((S, Hq, D), qmul)
    kp, vp = randbits((prow, Hkv, D)), randbits((prow, Hkv, D))
    ks, vs = randbits((srow, Hkv, D)), randbits((srow, Hkv, D))
    if poison:
        nan = np.uint16(0x7FC0)
        for arr, starts, lens in ((kp, ps, lp), (vp, ps, lp), (ks, ss, ls), (vs, ss, ls)):
            mask = np.ones(arr.shape[0], bool)
            for a, n in zip(starts, lens):
                mask[a:a + n] = False
            arr[mask] = nan
    return dict(q=q, k_prefix=kp, v_prefix=vp, k_suffix=ks, v_suffix=vs,
                prefix_start=ps, prefix_len=lp, suffix_start=ss, suffix_len=ls, group_size=G)


def tile_sample(R: int, ntiles: int, seed: int = 0, tile: int = 256) -> np.ndarray:
    """Rows 0 and R - 1 plus one seeded row in each of ntiles distinct
    tile-row blocks (the last block included), ascending and distinct."""
    rng = np.random.Generator(np.random.PCG64(seed))
    nt = (R + tile - 1) // tile
    tiles = rng.choice(np.arange(nt - 1), size=min(ntiles, nt) - 1, replace=False) if nt > 1 else np.array([], int)
    tiles = np.concatenate([tiles, [nt - 1]])
    rows = [min(R - 1, int(t) * tile + int(rng.integers(0, tile))) for t in tiles]
    return np.unique(np.concatenate([[0, R - 1], rows]).astype(np.int64))
