"""rl_token_logprob_noalloc through the C ABI against rl_token_logprob.

The variant runs the same plan and kernels with its workspace in a static
device array, so its results must equal rl_token_logprob's bit for bit, on a
first call and on a second, smaller call that reuses the array (whatever the
first call left there).  Both are also held to the oracle's bar (log-prob and
lse max-abs <= 2e-3) on a sample of rows.  Sizes whose workspace exceeds the
array are refused before any launch, leaving the outputs untouched.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2607_20908_amd as rk
import workloads as W
from gpu_util import LOGPROB_TOL, dev, max_abs, say

pytestmark = pytest.mark.gpu


def inputs(R, H, V, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    h = W.bf16_bits(torch.from_numpy(rng.standard_normal((R, H)).astype(np.float32)).to(torch.bfloat16))
    w = W.bf16_bits(torch.from_numpy((rng.standard_normal((V, H)) * 0.02).astype(np.float32)).to(torch.bfloat16))
    t = rng.integers(0, V, R).astype(np.int32)
    t[::7] = -1                      # masked rows
    return h, w, t


def noalloc_call(h, w, t, lp, lse, inv_T):
    R, H = h.shape
    V = w.shape[0]
    lib = rk.lib()
    return lib.rl_token_logprob_noalloc(R, H, V, ctypes.c_void_p(h.data_ptr()), ctypes.c_void_p(w.data_ptr()),
                                        ctypes.c_void_p(t.data_ptr()), ctypes.c_float(inv_T),
                                        ctypes.c_void_p(lp.data_ptr()), ctypes.c_void_p(lse.data_ptr()), None)


# the 32B-class decode-step row (hidden-split tail, 66 MB of scratch), then a
# smaller call with narrow last-round tiles and another temperature
@pytest.mark.parametrize("shapes", [[(256, 5120, 151936, 1.0), (100, 256, 5000, 1.0 / 0.7)]])
def test_noalloc_matches_workspace_entry_point(shapes):
    for i, (R, H, V, inv_T) in enumerate(shapes):
        say(f"noalloc call {i}: {R} x {H} x {V}")
        hb, wb, tn = inputs(R, H, V, 17 + i)
        h, w = W.bits_to_bf16(hb, dev()), W.bits_to_bf16(wb, dev())
        t = torch.from_numpy(tn).to(dev())
        lp = torch.full((R,), float("nan"), dtype=torch.float32, device=dev())
        lse = torch.full((R,), float("nan"), dtype=torch.float32, device=dev())
        st = noalloc_call(h, w, t, lp, lse, inv_T)
        assert st == 0, rk.lib().rl_last_error().decode()
        ref_lp, ref_lse = rk.token_logprob(h, w, t, inv_T)
        torch.cuda.synchronize()
        assert torch.equal(lp, ref_lp), f"call {i}: logprob differs from rl_token_logprob"
        assert torch.equal(lse, ref_lse), f"call {i}: lse differs from rl_token_logprob"
        rows = np.unique(np.concatenate([[0, R - 1], np.random.Generator(np.random.PCG64(i)).integers(0, R, 14)]))
        olp, olse = oracle.token_logprob(hb[rows], wb, tn[rows], inv_T)
        assert max_abs(lp.cpu().numpy()[rows], olp) <= LOGPROB_TOL
        assert max_abs(lse.cpu().numpy()[rows], olse) <= LOGPROB_TOL
        assert np.all(lp.cpu().numpy()[tn == -1] == 0.0)
        del h, w


def test_noalloc_refuses_sizes_beyond_its_scratch():
    R, H, V = 65536, 64, 151936      # partials alone: 594 slots x 65536 rows x 8 B = 311 MB
    need = rk.token_logprob_workspace_size(R, H, V)
    assert need > rk.NOALLOC_SCRATCH_BYTES
    h = torch.zeros(R, H, dtype=torch.bfloat16, device=dev())
    w = torch.zeros(V, H, dtype=torch.bfloat16, device=dev())
    t = torch.zeros(R, dtype=torch.int32, device=dev())
    lp = torch.full((R,), 5.0, dtype=torch.float32, device=dev())
    lse = torch.full((R,), 5.0, dtype=torch.float32, device=dev())
    st = noalloc_call(h, w, t, lp, lse, 1.0)
    assert st == 3 and b"scratch" in rk.lib().rl_last_error()
    torch.cuda.synchronize()
    assert torch.all(lp == 5.0) and torch.all(lse == 5.0)
