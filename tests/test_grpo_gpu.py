"""GPU parity of the GRPO advantages and clipped surrogate (Sec. 3, Eq. grpo-loss)
against the fp64 oracle, through the C ABI.

Tolerances: both sides compute in fp64 from the same fp32 inputs and differ
only in summation order (relative ~1e-15) and in exp's last bit; the GPU
rounds its results to fp32 (half an ulp, 6e-8 relative).  Outputs are
compared at rtol 1e-6.  Which rows have a zero gradient (the clipped term is
the minimum) is a decision taken in fp64 on both sides from the same inputs,
compared exactly; the inputs keep ratios off the clip bounds by far more than
exp's error.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20908_amd as rk
import workloads as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
RTOL = 1e-6


def adv_close(got, want):
    np.testing.assert_allclose(got, want, rtol=RTOL, atol=1e-9)


def oracle_inputs(x):
    return (x.logp_new.cpu().numpy().astype(np.float64), x.logp_old.cpu().numpy().astype(np.float64),
            x.seq.cpu().numpy())


@pytest.mark.parametrize("P,G", [(1, 1), (3, 1), (2, 2), (4, 16), (7, 5), (2, 64), (3, 65), (5, 200),
                                 (2, 1024), (300, 8)])
def test_advantage_parity(P, G):
    rng = np.random.Generator(np.random.PCG64(P * 1000 + G))
    r = rng.normal(0.0, 3.0, P * G).astype(np.float32)
    if P > 1:
        r[G:2 * G] = r[G]                    # one group with zero variance
    adv = rk.grpo_advantage(torch.from_numpy(r).to(DEV), G)
    torch.cuda.synchronize()
    got = adv.cpu().numpy()
    want = oracle.grpo_advantage(r, G)
    adv_close(got, want)
    if G == 1:
        assert np.all(got == 0)
    if P > 1:
        assert np.all(got[G:2 * G] == 0)


def test_advantage_reward_levels():
    # rewards from a few levels: many ties, some groups all equal
    x = wl.make_grpo_inputs(wl.GRPO_CONFIGS["policy"], DEV, seed=3, reward_levels=3)
    G = x.cfg.group_size
    got = rk.grpo_advantage(x.reward, G).cpu().numpy()
    want = oracle.grpo_advantage(x.reward.cpu().numpy(), G)
    adv_close(got, want)
    assert np.all(got[:G] == 0)


def run_surrogate(x, adv, eps=None, workspace=None):
    eps = x.eps if eps is None else eps
    loss, grad = rk.grpo_surrogate(x.logp_new, x.logp_old, x.seq, adv, x.cfg.group_size, eps,
                                   workspace=workspace)
    torch.cuda.synchronize()
    return float(loss.cpu()[0]), grad.cpu().numpy()


def check_surrogate(x, adv_dev, eps=None):
    eps = x.eps if eps is None else eps
    loss, grad = run_surrogate(x, adv_dev, eps)
    new, old, seq = oracle_inputs(x)
    wl_, wg = oracle.grpo_surrogate(new, old, seq, adv_dev.cpu().numpy().astype(np.float64),
                                    x.cfg.group_size, eps)
    assert loss == pytest.approx(wl_, rel=RTOL, abs=1e-12), (loss, wl_)
    np.testing.assert_allclose(grad, wg, rtol=RTOL, atol=1e-12)
    np.testing.assert_array_equal(grad == 0, wg == 0)
    return loss, grad


@pytest.mark.parametrize("name,seed,drift", [("tiny", 0, 0.1), ("tiny", 1, 0.5), ("policy", 0, 0.1),
                                             ("policy", 2, 0.3)])
def test_surrogate_parity(name, seed, drift):
    x = wl.make_grpo_inputs(wl.GRPO_CONFIGS[name], DEV, seed=seed, drift=drift)
    adv = rk.grpo_advantage(x.reward, x.cfg.group_size)
    loss, grad = check_surrogate(x, adv)
    owned = x.seq.cpu().numpy() >= 0
    assert np.all(grad[~owned] == 0)
    assert np.count_nonzero(grad[owned]) > 0


def test_surrogate_chains_with_gpu_advantages():
    # the advantages the GPU computed feed the surrogate; the oracle recomputes
    # both from the rewards alone
    x = wl.make_grpo_inputs(wl.GRPO_CONFIGS["policy"], DEV, seed=5, drift=0.2)
    G = x.cfg.group_size
    adv = rk.grpo_advantage(x.reward, G)
    loss, grad = run_surrogate(x, adv)
    want_adv = oracle.grpo_advantage(x.reward.cpu().numpy(), G)
    new, old, seq = oracle_inputs(x)
    wl_, wg = oracle.grpo_surrogate(new, old, seq, want_adv, G, x.eps)
    assert loss == pytest.approx(wl_, rel=1e-5)
    np.testing.assert_allclose(grad, wg, rtol=1e-5, atol=1e-12)


def test_surrogate_bitwise_reproducible_and_workspace_reuse():
    x = wl.make_grpo_inputs(wl.GRPO_CONFIGS["policy"], DEV, seed=7)
    G = x.cfg.group_size
    adv = rk.grpo_advantage(x.reward, G)
    ws = torch.empty(rk.grpo_surrogate_workspace_size(x.seq.numel(), adv.numel() // G, G),
                     dtype=torch.uint8, device=DEV)
    a = run_surrogate(x, adv, workspace=ws)
    b = run_surrogate(x, adv, workspace=ws)      # counts left in the workspace are cleared
    assert a[0] == b[0]
    np.testing.assert_array_equal(a[1], b[1])
    # a smaller batch on the same workspace
    y = wl.make_grpo_inputs(wl.GRPO_CONFIGS["tiny"], DEV, seed=8)
    adv_y = rk.grpo_advantage(y.reward, y.cfg.group_size)
    loss, grad = run_surrogate(y, adv_y, workspace=ws)
    new, old, seq = oracle_inputs(y)
    wl_, wg = oracle.grpo_surrogate(new, old, seq, adv_y.cpu().numpy().astype(np.float64),
                                    y.cfg.group_size, y.eps)
    assert loss == pytest.approx(wl_, rel=RTOL)
    np.testing.assert_allclose(grad, wg, rtol=RTOL, atol=1e-12)


def test_surrogate_ratio_one_and_zero_eps():
    # new == old: every ratio is 1, the clip is inactive, ties go to the ratio term
    x = wl.make_grpo_inputs(wl.GRPO_CONFIGS["tiny"], DEV, seed=9)
    x.logp_new.copy_(x.logp_old)
    adv = torch.from_numpy(np.random.Generator(np.random.PCG64(9)).standard_normal(
        x.reward.numel()).astype(np.float32)).to(DEV)
    for eps in (0.0, x.eps):
        loss, grad = check_surrogate(x, adv, eps)
        owned = x.seq.cpu().numpy() >= 0
        assert np.all((grad[owned] != 0) == (adv.cpu().numpy()[x.seq.cpu().numpy()[owned]] != 0))


def test_surrogate_unowned_and_out_of_range_rows():
    x = wl.make_grpo_inputs(wl.GRPO_CONFIGS["tiny"], DEV, seed=10, drift=0.3)
    S = x.reward.numel()
    seq = x.seq.cpu().numpy()
    seq[::7] = S + 3                        # past the last candidate: ignored like -1
    seq[1::11] = -1
    x.seq.copy_(torch.from_numpy(seq))
    adv = rk.grpo_advantage(x.reward, x.cfg.group_size)
    loss, grad = check_surrogate(x, adv)
    assert np.all(grad[(seq < 0) | (seq >= S)] == 0)


def test_surrogate_all_rows_unowned():
    x = wl.make_grpo_inputs(wl.GRPO_CONFIGS["tiny"], DEV, seed=11)
    x.seq.fill_(-1)
    adv = rk.grpo_advantage(x.reward, x.cfg.group_size)
    loss, grad = run_surrogate(x, adv)
    assert loss == 0.0
    assert np.all(grad == 0)


def test_surrogate_empty():
    G = 4
    e = torch.empty(0, dtype=torch.float32, device=DEV)
    es = torch.empty(0, dtype=torch.int32, device=DEV)
    adv = torch.ones(8, dtype=torch.float32, device=DEV)
    loss, grad = rk.grpo_surrogate(e, e, es, adv, G)
    torch.cuda.synchronize()
    assert float(loss.cpu()[0]) == 0.0 and grad.numel() == 0
    # rows but no candidates
    x = wl.make_grpo_inputs(wl.GRPO_CONFIGS["tiny"], DEV, seed=12)
    x.seq.fill_(-1)
    loss, grad = rk.grpo_surrogate(x.logp_new, x.logp_old, x.seq, e, G)
    torch.cuda.synchronize()
    assert float(loss.cpu()[0]) == 0.0 and np.all(grad.cpu().numpy() == 0)


def test_surrogate_many_candidates():
    # 4096 prompts x 16: counts held per candidate, many term workgroups
    rng = np.random.Generator(np.random.PCG64(13))
    P, G = 4096, 16
    S = P * G
    seq = np.repeat(np.arange(S, dtype=np.int32), rng.integers(1, 9, S))
    rng.shuffle(seq)
    R = seq.size
    old = (-rng.exponential(1.0, R)).astype(np.float32)
    new = (old + rng.normal(0, 0.2, R)).astype(np.float32)
    adv = rng.standard_normal(S).astype(np.float32)
    d = lambda a: torch.from_numpy(a).to(DEV)
    loss, grad = rk.grpo_surrogate(d(new), d(old), d(seq), d(adv), G, float(np.float32(0.2)))
    torch.cuda.synchronize()
    wl_, wg = oracle.grpo_surrogate(new.astype(np.float64), old.astype(np.float64), seq,
                                    adv.astype(np.float64), G, float(np.float32(0.2)))
    assert float(loss.cpu()[0]) == pytest.approx(wl_, rel=RTOL)
    np.testing.assert_allclose(grad.cpu().numpy(), wg, rtol=RTOL, atol=1e-12)
