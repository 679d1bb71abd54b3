"""Appending to the suffix KV cache on the GPU: bit-exact against the oracle's
copy, and a decode loop that appends one token per candidate per step into
fixed-capacity regions and checks every step's attention against the fp64
oracle (the cache never moves)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20908_amd as rk
import workloads as W
from gpu_util import ATTN_LSE_TOL, ATTN_OUT_TOL, dev, max_abs, say, to_dev

pytestmark = pytest.mark.gpu


def rand_bits(rng, shape):
    return W.bf16_bits(torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(torch.bfloat16))


@pytest.mark.parametrize("layout", ["token", "head"])
@pytest.mark.parametrize("D", [64, 128])
def test_append_bit_exact(layout, D):
    rng = np.random.Generator(np.random.PCG64(D))
    P, G, Hkv, cap = 3, 4, 2, 40
    S = P * G
    rows = S * cap + 7
    ss = np.arange(S, dtype=np.int64) * cap + 3
    sl = rng.integers(0, 20, S).astype(np.int32)
    nl = rng.integers(0, 6, S).astype(np.int32)
    nl[1] = 0
    ns = np.concatenate([[0], np.cumsum(nl)[:-1]]).astype(np.int64) + 1   # packed after one spare row
    new_rows = int(nl.sum()) + 3
    shape = (Hkv, rows, D) if layout == "head" else (rows, Hkv, D)
    kc, vc = rand_bits(rng, shape), rand_bits(rng, shape)
    kn, vn = rand_bits(rng, (new_rows, Hkv, D)), rand_bits(rng, (new_rows, Hkv, D))
    say(f"kv append {layout} D={D}")
    kd, vd = to_dev(kc), to_dev(vc)
    rk.kv_append(to_dev(kn), to_dev(vn), kd, vd, ss, sl, ns, nl, G, suffix_capacity=np.full(S, cap - 3),
                 kv_layout=layout)
    torch.cuda.synchronize()
    wk, wv = oracle.kv_append(kc, vc, kn, vn, ss, sl, ns, nl, kv_layout=layout)
    assert np.array_equal(W.bf16_bits(kd), wk) and np.array_equal(W.bf16_bits(vd), wv)


@pytest.mark.parametrize("layout", ["token", "head"])
def test_decode_loop_appends_in_place(layout):
    """12 decode steps: each appends one token per candidate, then attends."""
    rng = np.random.Generator(np.random.PCG64(17))
    P, G, Hq, Hkv, D, cap = 2, 4, 8, 2, 128, 48
    S = P * G
    Lp = np.array([300, 77], np.int32)
    ps = np.array([0, 300], np.int64)
    pshape = (Hkv, 377, D) if layout == "head" else (377, Hkv, D)
    kp, vp = rand_bits(rng, pshape), rand_bits(rng, pshape)
    rows = S * cap
    sshape = (Hkv, rows, D) if layout == "head" else (rows, Hkv, D)
    ks, vs = rand_bits(rng, sshape), rand_bits(rng, sshape)    # garbage past each suffix
    ss = np.arange(S, dtype=np.int64) * cap
    sl = rng.integers(0, 10, S).astype(np.int32)
    kpd, vpd, ksd, vsd = to_dev(kp), to_dev(vp), to_dev(ks), to_dev(vs)
    base = ksd.data_ptr()
    tm = lambda x: x.transpose(1, 0, 2).copy() if layout == "head" else x   # oracle wants token-major
    scale = float(np.float32(1 / np.sqrt(D)))
    for step in range(12):
        kn, vn = rand_bits(rng, (S, Hkv, D)), rand_bits(rng, (S, Hkv, D))
        q = rand_bits(rng, (S, Hq, D))
        rk.kv_append(to_dev(kn), to_dev(vn), ksd, vsd, ss, sl, np.arange(S), np.ones(S, np.int32), G,
                     suffix_capacity=np.full(S, cap), kv_layout=layout)
        ks, vs = oracle.kv_append(ks, vs, kn, vn, ss, sl, np.arange(S), np.ones(S, np.int32), kv_layout=layout)
        sl = sl + 1
        say(f"decode loop {layout} step {step}")
        out, lse = rk.decode_attn(to_dev(q), kpd, vpd, ksd, vsd, ps, Lp, ss, sl, G, scale=scale,
                                  return_lse=True, kv_layout=layout)
        torch.cuda.synchronize()
        assert ksd.data_ptr() == base
        ro, rl = oracle.decode_attn(q, tm(kp), tm(vp), tm(ks), tm(vs), ps, Lp, ss, sl, G, scale)
        e1 = max_abs(out.float().cpu().numpy(), ro)
        e2 = max_abs(lse.cpu().numpy(), rl)
        assert e1 <= ATTN_OUT_TOL and e2 <= ATTN_LSE_TOL, (step, e1, e2)
    assert np.array_equal(W.bf16_bits(ksd), ks) and np.array_equal(W.bf16_bits(vsd), vs)
