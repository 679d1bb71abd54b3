"""Calls on a stream other than torch's current one (stream=).

The binding allocates each call's workspace and outputs on the call's stream,
so after the call drops its workspace, torch's caching allocator reuses that
memory only for later work on the same stream.  Here every call is followed
by a default-stream allocation of the workspace's size that is filled with
garbage at once: were the workspace still owned by the default stream, the
fill could land in it while the side stream's kernels use it.  Every result
must equal the default-stream call's bit for bit.
"""
import math

import numpy as np
import pytest
import torch

import paper_2607_20908_amd as rk
from gpu_util import decode_host_case, dev, say, to_dev

pytestmark = pytest.mark.gpu


def test_side_stream_logprob_and_backward():
    rng = np.random.Generator(np.random.PCG64(31))
    R, H, V = 512, 1024, 20000
    h = torch.from_numpy(rng.standard_normal((R, H)).astype(np.float32)).to(torch.bfloat16).to(dev())
    w = torch.from_numpy((rng.standard_normal((V, H)) * 0.05).astype(np.float32)).to(torch.bfloat16).to(dev())
    t = torch.from_numpy(rng.integers(0, V, R).astype(np.int32)).to(dev())
    g = torch.from_numpy(rng.standard_normal(R).astype(np.float32)).to(dev())
    ref_lp, ref_lse = rk.token_logprob(h, w, t)
    ref_dh = rk.token_logprob_backward(h, w, t, ref_lse, g)
    torch.cuda.synchronize()
    n_fwd = rk.token_logprob_workspace_size(R, H, V)
    n_bwd = rk.token_logprob_backward_workspace_size(R, H, V)
    side = torch.cuda.Stream()
    say("log-prob forward and backward on a side stream")
    outs = []
    for _ in range(12):
        lp, lse = rk.token_logprob(h, w, t, stream=side)
        junk = torch.empty(n_fwd, dtype=torch.uint8, device=dev())
        junk.fill_(0xFF)
        dh = rk.token_logprob_backward(h, w, t, ref_lse, g, stream=side)
        junk = torch.empty(n_bwd, dtype=torch.uint8, device=dev())
        junk.fill_(0xFF)
        outs.append((lp, lse, dh))
    side.synchronize()
    torch.cuda.synchronize()
    for lp, lse, dh in outs:
        assert torch.equal(lp, ref_lp) and torch.equal(lse, ref_lse)
        assert torch.equal(dh, ref_dh)


def test_side_stream_decode():
    D = 128
    c = decode_host_case(4, 8, 16, 4, D, [300, 0, 77, 129], np.arange(32) * 23 % 400, seed=32, gap=2)
    scale = 1.0 / math.sqrt(D)
    t = {k: to_dev(c[k]) for k in ("q", "k_prefix", "v_prefix", "k_suffix", "v_suffix")}
    args = (t["q"], t["k_prefix"], t["v_prefix"], t["k_suffix"], t["v_suffix"], c["prefix_start"], c["prefix_len"],
            c["suffix_start"], c["suffix_len"], c["group_size"])
    ref_o, ref_l = rk.decode_attn(*args, scale=scale, return_lse=True)
    torch.cuda.synchronize()
    need = rk.decode_attn_workspace_size(4, 8, 16, 4, D, c["prefix_start"], c["prefix_len"], c["suffix_start"],
                                         c["suffix_len"], c["k_prefix"].shape[0], c["k_suffix"].shape[0], scale)
    side = torch.cuda.Stream()
    say("decode on a side stream")
    outs = []
    for _ in range(20):
        outs.append(rk.decode_attn(*args, scale=scale, return_lse=True, stream=side))
        junk = torch.empty(need, dtype=torch.uint8, device=dev())
        junk.fill_(0xFF)
    side.synchronize()
    torch.cuda.synchronize()
    for o, l in outs:
        assert torch.equal(o.view(torch.int16), ref_o.view(torch.int16))
        assert torch.equal(l, ref_l)
