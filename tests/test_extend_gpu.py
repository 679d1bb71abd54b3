"""Extend (prefill) attention: the HIP path against the fp64 oracle on the same bits.

Bar (as for decode attention): output max-abs <= 1e-2 and lse max-abs <= 1e-3
for bf16 inputs with fp32 accumulation.  Rows of no candidate must stay
untouched; results must be bitwise reproducible across calls.  Gap rows
between sequences hold NaN, so a read outside a valid range shows up.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_20908_amd as rk
import workloads as W
from gpu_util import ATTN_LSE_TOL, ATTN_OUT_TOL, decode_host_case, dev, max_abs, say, to_dev

pytestmark = pytest.mark.gpu


def extend_host_case(P, G, Hq, Hkv, D, lp, ls, nl, seed=0, gap=3, qgap=2):
    """decode_host_case's poisoned caches plus new-token counts and packed queries
    (candidates in reverse order, `qgap` unused rows between them)."""
    c = decode_host_case(P, G, Hq, Hkv, D, lp, ls, seed=seed, gap=gap, poison=True)
    S = P * G
    nl = np.asarray(nl, np.int32)
    qs = np.zeros(S, np.int64)
    pos = qgap
    for s in reversed(range(S)):
        qs[s] = pos
        pos += int(nl[s]) + qgap
    rng = np.random.Generator(np.random.PCG64(seed + 77))
    q = W.bf16_bits(torch.from_numpy(rng.standard_normal((pos, Hq, D)).astype(np.float32)).to(torch.bfloat16))
    c.update(q=q, new_len=nl, q_start=qs)
    return c


def run_gpu(c, scale, layout="token", out_fill=None):
    def kv(bits):
        return to_dev(np.ascontiguousarray(np.transpose(bits, (1, 0, 2))) if layout == "head" else bits)
    t = {k: kv(c[k]) for k in ("k_prefix", "v_prefix", "k_suffix", "v_suffix")}
    q = to_dev(c["q"])
    out = lse = None
    if out_fill is not None:
        out = torch.full(q.shape, out_fill, dtype=torch.bfloat16, device=dev())
        lse = torch.full(q.shape[:2], out_fill, dtype=torch.float32, device=dev())
    out, lse = rk.extend_attn(q, t["k_prefix"], t["v_prefix"], t["k_suffix"], t["v_suffix"],
                              c["prefix_start"], c["prefix_len"], c["suffix_start"], c["suffix_len"],
                              c["new_len"], c["q_start"], c["group_size"], scale=scale, return_lse=True,
                              out=out, lse=lse, kv_layout=layout)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), lse.cpu().numpy(), W.bf16_bits(out)


def run_oracle(c, scale):
    return oracle.extend_attn(c["q"], c["k_prefix"], c["v_prefix"], c["k_suffix"], c["v_suffix"],
                              c["prefix_start"], c["prefix_len"], c["suffix_start"], c["suffix_len"],
                              c["new_len"], c["q_start"], c["group_size"], scale)


def owned_rows(c):
    rows = np.zeros(c["q"].shape[0], bool)
    for s in range(len(c["new_len"])):
        rows[c["q_start"][s]:c["q_start"][s] + c["new_len"][s]] = True
    return rows


def check(c, scale, what, layout="token"):
    say(f"extend parity {what} layout={layout}")
    o, l, _ = run_gpu(c, scale, layout, out_fill=-3.0)
    ro, rl = run_oracle(c, scale)
    rows = owned_rows(c)
    eo, el = max_abs(o[rows], ro[rows]), max_abs(l[rows], rl[rows])
    assert eo <= ATTN_OUT_TOL, f"{what}: out max-abs {eo}"
    assert el <= ATTN_LSE_TOL, f"{what}: lse max-abs {el}"
    assert (o[~rows] == -3.0).all() and (l[~rows] == -3.0).all(), f"{what}: wrote rows of no candidate"
    return eo, el


def test_tiny_config():
    cfg = W.DECODE_CONFIGS["tiny"]
    x = W.make_extend_inputs(cfg, "cpu")
    d = x.dec
    c = dict(q=W.bf16_bits(x.q), k_prefix=W.bf16_bits(d.k_prefix), v_prefix=W.bf16_bits(d.v_prefix),
             k_suffix=W.bf16_bits(d.k_suffix), v_suffix=W.bf16_bits(d.v_suffix),
             prefix_start=d.prefix_start, prefix_len=d.prefix_len, suffix_start=d.suffix_start,
             suffix_len=d.suffix_len, new_len=x.new_len, q_start=x.q_start, group_size=cfg.group_size)
    check(c, d.scale, "tiny config (all suffix tokens new)")


@pytest.mark.parametrize("layout", ["token", "head"])
@pytest.mark.parametrize("D", [64, 128])
def test_ragged_multi_block(D, layout):
    # several 64-token tiles and 256-row blocks, ragged tails, an empty prefix,
    # new tokens from none to the whole suffix
    P, G, Hq, Hkv = 2, 3, 16, 4
    lp = [300, 0]
    ls = [200, 1, 70, 65, 0, 131]
    nl = [130, 1, 70, 3, 0, 66]
    c = extend_host_case(P, G, Hq, Hkv, D, lp, ls, nl, seed=D)
    check(c, 1.0 / math.sqrt(D), f"ragged D={D}", layout)


@pytest.mark.parametrize("Hq,Hkv", [(64, 8),    # r = 8: 32 tokens per block
                                    (24, 2),    # r = 12: a block boundary splits a token's heads
                                    (4, 4),     # r = 1
                                    (6, 1)])    # r = 6, one kv head
def test_head_groups(Hq, Hkv):
    P, G, D = 2, 2, 128
    rng = np.random.Generator(np.random.PCG64(Hq * 10 + Hkv))
    lp = [190, 77]
    ls = rng.integers(40, 160, P * G).tolist()
    nl = [min(l, int(x)) for l, x in zip(ls, rng.integers(1, 120, P * G))]
    c = extend_host_case(P, G, Hq, Hkv, D, lp, ls, nl, seed=Hq + Hkv)
    check(c, 1.0 / math.sqrt(D), f"Hq={Hq} Hkv={Hkv}")


def _scaled_bits(bits, mul):
    """bf16 bits times a power of two (exact)."""
    f = torch.from_numpy((bits.astype(np.uint32) << 16).view(np.float32))
    return W.bf16_bits((f * mul).to(torch.bfloat16))


def test_peaky_scores_and_scale():
    # Large query norms: the running max moves often and exp underflows for
    # most tokens.  Each output is then nearly one value row, so V is halved to
    # keep |out| < 2: bf16 rounding of the output (half an ulp, 2^-8 there) and
    # of p ~ 1 (2^-9 relative) then stay inside the 1e-2 bar, as they do for
    # the averaged outputs of N(0, 1) inputs.
    P, G, Hq, Hkv, D = 1, 4, 8, 2, 128
    c = extend_host_case(P, G, Hq, Hkv, D, [150], [90, 64, 1, 200], [90, 10, 1, 129], seed=5)
    c["q"] = _scaled_bits(c["q"], 4.0)
    c["v_prefix"] = _scaled_bits(c["v_prefix"], 0.5)
    c["v_suffix"] = _scaled_bits(c["v_suffix"], 0.5)
    check(c, 0.3, "peaky")


def test_single_new_token_is_decode():
    # new_len = 1 everywhere: the same visible context as one decode step
    P, G, Hq, Hkv, D = 2, 4, 32, 8, 128
    ls = [100, 64, 1, 300, 17, 80, 200, 5]
    c = extend_host_case(P, G, Hq, Hkv, D, [129, 1000], ls, [1] * 8, seed=9)
    check(c, 1.0 / math.sqrt(D), "one new token per candidate")


def test_reproducible_and_no_new_tokens():
    P, G, Hq, Hkv, D = 1, 2, 16, 2, 128
    c = extend_host_case(P, G, Hq, Hkv, D, [300], [150, 90], [150, 40], seed=11)
    say("extend reproducibility")
    _, _, b1 = run_gpu(c, 0.1)
    _, _, b2 = run_gpu(c, 0.1)
    assert np.array_equal(b1, b2)
    c0 = dict(c, new_len=np.zeros(2, np.int32))
    say("extend with no new tokens")
    o, l, _ = run_gpu(c0, 0.1, out_fill=1.5)
    assert (o == 1.5).all() and (l == 1.5).all()


@pytest.mark.slow
@pytest.mark.parametrize("name,layout", [("longctx", "head"), ("longctx", "token"), ("8b", "head")])
def test_full_size_turn(name, layout):
    """The refinement-turn extend at full size, every candidate's whole
    suffix new: the long context (4 prompts x G=8, 64/8 heads, D=128, shared
    prefix 24576, suffixes geometric with mean 1024, cap 4096) in both
    layouts, and the 8B-class shape bench.py times (64 prompts x G=8, 32/8
    heads, prefix 1024, suffixes uniform in [256, 2048]: 609026 new tokens).
    The oracle checks the first, the last and a random new token of every
    candidate, at every head: a token is the call with that candidate's
    suffix ending at the token and one new token."""
    cfg = W.DECODE_CONFIGS[name]
    x = W.make_extend_inputs(cfg, dev(), kv_layout=layout)
    d = x.dec
    say(f"extend full size {name} layout={layout}: {int(x.new_len.sum())} new tokens")
    # outputs start as NaN: every new token's rows at every head must be
    # written, so a work block missing from the launch shows up
    out = torch.full(x.q.shape, float("nan"), dtype=torch.bfloat16, device=dev())
    lse = torch.full(x.q.shape[:2], float("nan"), dtype=torch.float32, device=dev())
    out, lse = rk.extend_attn(x.q, d.k_prefix, d.v_prefix, d.k_suffix, d.v_suffix, d.prefix_start,
                              d.prefix_len, d.suffix_start, d.suffix_len, x.new_len, x.q_start,
                              cfg.group_size, scale=d.scale, return_lse=True, out=out, lse=lse, kv_layout=layout)
    torch.cuda.synchronize()
    owned = torch.zeros(x.q.shape[0], dtype=torch.bool)
    for s in range(cfg.num_seqs):
        owned[int(x.q_start[s]):int(x.q_start[s]) + int(x.new_len[s])] = True
    owned = owned.to(dev())
    assert torch.isfinite(out[owned].float()).all() and torch.isfinite(lse[owned]).all()
    kp, vp, ks, vs = (W.bf16_bits(d.token_major(t)) for t in (d.k_prefix, d.v_prefix, d.k_suffix, d.v_suffix))
    rng = np.random.Generator(np.random.PCG64(3))
    S = cfg.num_seqs
    for rep in range(3):
        # one sampled new token per candidate (first, last, random)
        pick = [0 if rep == 0 else (int(x.new_len[s]) - 1 if rep == 1 else int(rng.integers(0, x.new_len[s])))
                for s in range(S)]
        sl = np.array([d.suffix_len[s] - x.new_len[s] + pick[s] + 1 for s in range(S)], np.int32)
        rows = np.array([x.q_start[s] + pick[s] for s in range(S)], np.int64)
        idx = torch.from_numpy(rows).to(dev())
        ro, rl = oracle.extend_attn(W.bf16_bits(x.q[idx]), kp, vp, ks, vs, d.prefix_start, d.prefix_len,
                                    d.suffix_start, sl, np.ones(S, np.int32), np.arange(S, dtype=np.int64),
                                    cfg.group_size, d.scale)
        eo = max_abs(out[idx].float().cpu().numpy(), ro)
        el = max_abs(lse[idx].cpu().numpy(), rl)
        say(f"  sample {rep}: out max-abs {eo:.2e} lse max-abs {el:.2e}")
        assert eo <= ATTN_OUT_TOL and el <= ATTN_LSE_TOL
