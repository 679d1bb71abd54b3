"""Seeded random shapes through every GPU entry point, against the oracle.

The other GPU tests pick their shapes by hand to reach particular paths; here
each case draws its shape from its own seed (printed before the GPU step):
odd head ratios, zero-length prompts and suffixes, split sizes, both KV
layouts, ragged row and vocabulary counts, masked targets, temperatures,
nucleus sizes, append capacities, group sizes and clip ranges.  Every case applies the same bar as the hand-picked tests
(their check functions).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_20908_amd as rk
import workloads as W
from gpu_util import decode_host_case, say, to_dev
from test_decode_gpu import check as decode_check
from test_extend_gpu import check as extend_check
from test_extend_gpu import extend_host_case
from test_logprob_bwd_gpu import case as backward_case
from test_logprob_gpu import check as logprob_check
from test_logprob_gpu import rand_bits
from test_grpo_gpu import adv_close, check_surrogate
from test_sample_gpu import check as sample_check

pytestmark = pytest.mark.gpu

N = 25          # cases per entry point


def _rng(kind, i):
    return np.random.Generator(np.random.PCG64(1000 * kind + i))


def _lengths(rng, n, hi, p_zero=0.2):
    v = rng.integers(1, hi + 1, n)
    v[rng.random(n) < p_zero] = 0
    return v.astype(np.int32)


@pytest.mark.parametrize("i", range(N))
def test_decode_random_shapes(i):
    rng = _rng(1, i)
    P, G = int(rng.integers(1, 5)), int(rng.integers(1, 10))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    r = int(rng.choice([1, 2, 3, 4, 8, 16]))
    D = int(rng.choice([64, 128]))
    lp, ls = _lengths(rng, P, 700), _lengths(rng, P * G, 400, 0.15)
    split = int(rng.choice([0, 16, 48, 128]))
    layout = str(rng.choice(["token", "head"]))
    say(f"fuzz decode {i}: P={P} G={G} Hq={r * Hkv} Hkv={Hkv} D={D} split={split} layout={layout} "
        f"lp={lp.tolist()} sum ls={int(ls.sum())}")
    c = decode_host_case(P, G, r * Hkv, Hkv, D, lp, ls, seed=i, gap=int(rng.integers(0, 4)))
    decode_check(c, 1.0 / math.sqrt(D), split, f"fuzz {i}", layout)


@pytest.mark.parametrize("i", range(N))
def test_extend_random_shapes(i):
    rng = _rng(2, i)
    P, G = int(rng.integers(1, 4)), int(rng.integers(1, 6))
    Hkv = int(rng.choice([1, 2]))
    r = int(rng.choice([1, 2, 4]))
    D = int(rng.choice([64, 128]))
    lp, ls = _lengths(rng, P, 300), _lengths(rng, P * G, 200, 0.15)
    nl = np.array([int(rng.integers(0, x + 1)) for x in ls], np.int32)
    layout = str(rng.choice(["token", "head"]))
    say(f"fuzz extend {i}: P={P} G={G} Hq={r * Hkv} Hkv={Hkv} D={D} layout={layout} lp={lp.tolist()} "
        f"sum ls={int(ls.sum())} sum new={int(nl.sum())}")
    c = extend_host_case(P, G, r * Hkv, Hkv, D, lp, ls, nl, seed=100 + i)
    extend_check(c, 1.0 / math.sqrt(D), f"fuzz {i}", layout)


def _logprob_shape(rng):
    R = int(rng.integers(1, 700))
    H = 64 * int(rng.integers(1, 6))
    V = int(rng.integers(1, 5000))
    inv_T = float(rng.choice([1.0, 1 / 0.7, 1 / 0.2]))
    return R, H, V, inv_T


@pytest.mark.parametrize("i", range(N))
def test_logprob_random_shapes(i):
    rng = _rng(3, i)
    R, H, V, inv_T = _logprob_shape(rng)
    hb, wb = rand_bits(rng, (R, H)), rand_bits(rng, (V, H), float(rng.choice([0.02, 0.1, 0.3])))
    t = rng.integers(0, V, R).astype(np.int32)
    t[rng.random(R) < 0.1] = -1
    say(f"fuzz logprob {i}: R={R} H={H} V={V} inv_T={inv_T:.3f}")
    lp, _ = logprob_check(hb, wb, t, inv_T, f"fuzz {i}")
    assert (lp[t == -1] == 0).all()


@pytest.mark.parametrize("i", range(N))
def test_logprob_backward_random_shapes(i):
    rng = _rng(4, i)
    R, H, V, inv_T = _logprob_shape(rng)
    backward_case(R, H, V, seed=400 + i, wstd=float(rng.choice([0.02, 0.1])), inv_T=inv_T, mask_frac=0.1,
                  gzero=0.1, what=f"fuzz {i}")


@pytest.mark.parametrize("i", range(N))
def test_sample_random_shapes(i):
    rng = _rng(5, i)
    R = int(rng.integers(1, 400))
    H = 64 * int(rng.integers(1, 3))
    V = int(rng.integers(1, 3000))
    top_p = float(rng.choice([0.5, 0.9, 1.0]))
    hb, wb = rand_bits(rng, (R, H)), rand_bits(rng, (V, H), float(rng.choice([0.1, 0.3])))
    inv_t = rng.choice([1 / 0.2, 1 / 0.7, 1.0], R).astype(np.float32)
    say(f"fuzz sample {i}: R={R} H={H} V={V} top_p={top_p}")
    sample_check(hb, wb, inv_t, top_p, rng.random(R, dtype=np.float32), f"fuzz {i}")


@pytest.mark.parametrize("i", range(N))
def test_kv_append_random_shapes(i):
    rng = _rng(6, i)
    P, G = int(rng.integers(1, 5)), int(rng.integers(1, 9))
    Hkv, D = int(rng.choice([1, 2, 8])), int(rng.choice([64, 128]))
    S = P * G
    cap = int(rng.integers(1, 60))
    layout = str(rng.choice(["token", "head"]))
    pad = int(rng.integers(0, 4))
    ss = np.arange(S, dtype=np.int64) * (cap + pad) + pad
    sl = rng.integers(0, cap + 1, S).astype(np.int32)
    nl = np.array([int(rng.integers(0, cap - x + 1)) for x in sl], np.int32)
    ns = np.concatenate([[0], np.cumsum(nl)[:-1]]).astype(np.int64)
    rows = S * (cap + pad) + pad
    new_rows = max(int(nl.sum()), 1)
    shape = (Hkv, rows, D) if layout == "head" else (rows, Hkv, D)
    bits = lambda shp: rand_bits(rng, shp)
    kc, vc = bits(shape), bits(shape)
    kn, vn = bits((new_rows, Hkv, D)), bits((new_rows, Hkv, D))
    say(f"fuzz kv append {i}: P={P} G={G} Hkv={Hkv} D={D} cap={cap} layout={layout} new={int(nl.sum())}")
    kd, vd = to_dev(kc), to_dev(vc)
    rk.kv_append(to_dev(kn), to_dev(vn), kd, vd, ss, sl, ns, nl, G, suffix_capacity=np.full(S, cap),
                 kv_layout=layout)
    torch.cuda.synchronize()
    wk, wv = oracle.kv_append(kc, vc, kn, vn, ss, sl, ns, nl, kv_layout=layout)
    assert np.array_equal(W.bf16_bits(kd), wk) and np.array_equal(W.bf16_bits(vd), wv)


@pytest.mark.parametrize("i", range(N))
def test_grpo_random_shapes(i):
    rng = _rng(7, i)
    P, G = int(rng.integers(1, 9)), int(rng.integers(1, 70))
    T = int(rng.integers(2, 300))
    M = int(rng.integers(1, T + 1))
    cfg = W.GrpoConfig(f"fuzz{i}", P, G, T, M)
    say(f"fuzz grpo {i}: P={P} G={G} positions={T} max response={M}")
    x = W.make_grpo_inputs(cfg, "cuda:0", seed=700 + i, drift=float(rng.choice([0.05, 0.3, 1.0])),
                           reward_levels=int(rng.integers(1, 8)), eps=float(rng.choice([0.0, 0.2, 0.5])))
    adv = rk.grpo_advantage(x.reward, G)
    torch.cuda.synchronize()
    adv_close(adv.cpu().numpy(), oracle.grpo_advantage(x.reward.cpu().numpy(), G))
    check_surrogate(x, adv)
