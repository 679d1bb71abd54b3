"""Token log-prob: the HIP path against the fp64 oracle on the same bits.

Bar: log-prob and lse max-abs <= 2e-3; the gathered target id bit-exact
(id probes), masked rows exactly 0, invalid targets NaN.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20908_amd as rk
import workloads as W
from gpu_util import LOGPROB_TOL, dev, max_abs, say, tile_sample, to_dev

pytestmark = pytest.mark.gpu


def rand_bits(rng, shape, std=1.0):
    x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32) * std)
    return W.bf16_bits(x.to(torch.bfloat16))


def run_gpu(h_bits, w_bits, target, inv_T=1.0):
    h, w = to_dev(h_bits), to_dev(w_bits)
    t = torch.from_numpy(np.ascontiguousarray(target, np.int32)).to(dev())
    lp, lse = rk.token_logprob(h, w, t, inv_T)
    torch.cuda.synchronize()
    return lp.cpu().numpy(), lse.cpu().numpy()


def check(h_bits, w_bits, target, inv_T=1.0, what=""):
    say(f"logprob parity {what}")
    lp, lse = run_gpu(h_bits, w_bits, target, inv_T)
    rlp, rlse = oracle.token_logprob(h_bits, w_bits, target, inv_T)
    e1, e2 = max_abs(lp, rlp), max_abs(lse, rlse)
    assert e1 <= LOGPROB_TOL, f"{what}: logprob max-abs {e1}"
    assert e2 <= LOGPROB_TOL, f"{what}: lse max-abs {e2}"
    return lp, lse


def test_tiny_config():
    x = W.make_logprob_inputs(W.LOGPROB_CONFIGS["tiny"], "cpu")
    check(W.bf16_bits(x.hidden), W.bf16_bits(x.w_lm), x.target.numpy(), what="tiny config")


@pytest.mark.parametrize("R,H,V", [(300, 128, 1000),    # ragged rows and vocab, 2x4 tiles
                                   (1, 64, 257),        # one row, one vocab entry past a tile
                                   (513, 192, 511),
                                   (256, 4096, 2048),
                                   # more than 8 row tiles: the two-stage weight ring
                                   (2305, 64, 700),     # one hidden stage, ragged rows and vocab
                                   (2049, 192, 300),    # three hidden stages, one row past a tile
                                   # the combine: one workgroup per row up to 4096 rows,
                                   # one wave per row above
                                   (4096, 64, 1500),
                                   (5000, 64, 1500)])
def test_ragged_shapes(R, H, V):
    rng = np.random.Generator(np.random.PCG64(R + H + V))
    h = rand_bits(rng, (R, H))
    w = rand_bits(rng, (V, H), 0.05)
    t = rng.integers(0, V, R).astype(np.int32)
    check(h, w, t, what=f"{R}x{H}x{V}")


@pytest.mark.parametrize("R,H,V", [(200, 1024, 75739),    # 296 vocab tiles: 256 whole, 40 in 4 hidden parts
                                   (300, 1024, 38395),    # 2 x 150 tiles: 256 whole, 44 in 4 parts
                                   (256, 768, 66048)])    # 258 tiles: 256 whole, 2 in 3 parts
def test_split_tail(R, H, V):
    """A short last round of tiles runs as hidden-dimension parts summed by a
    reduce kernel; the tail holds the highest vocab tiles, so targets there
    (the last ids included), masks and invalid ids go through it."""
    rng = np.random.Generator(np.random.PCG64(R * 7 + V))
    h = rand_bits(rng, (R, H))
    w = rand_bits(rng, (V, H), 0.05)
    t = rng.integers(0, V, R).astype(np.int32)
    t[: R // 4] = rng.integers(V - 40 * 256, V, R // 4)
    t[[0, 1, 2, 3]] = [V - 1, V - 256, -1, V]
    lp, lse = check(h, w, t, 1.0 / 0.7, f"split tail {R}x{H}x{V}")
    assert lp[2] == 0 and np.isnan(lp[3])


@pytest.mark.parametrize("R,H,V,vt0,n,width", [(300, 512, 51001, 128, 95, 192),     # 2 row tiles, ragged rows
                                               (600, 512, 35700, 85, 73, 192),      # 3 row tiles: 255 whole tiles
                                               (1000, 512, 25500, 64, 48, 192),     # 4 row tiles
                                               (256, 256, 76800, 256, 88, 128),     # too few hidden steps to split
                                               (400, 64, 40000, 128, 57, 128)])     # 2 row tiles, past the vocabulary
def test_narrow_last_round(R, H, V, vt0, n, width):
    """A partial last round that cannot be split over the hidden dimension
    runs as tiles 128 (if they fit one round) or 192 entries wide over vocab
    [256 vt0, V), each with its own partial slot; targets on both sides of
    the boundary, on narrow-tile edges, in the ragged last narrow tile, a
    masked row and an invalid id go through it."""
    rng = np.random.Generator(np.random.PCG64(R * 11 + V))
    h = rand_bits(rng, (R, H))
    w = rand_bits(rng, (V, H), 0.05)
    t = rng.integers(0, V, R).astype(np.int32)
    v0 = vt0 * 256
    t[: R // 3] = rng.integers(v0, V, R // 3)
    edges = [v0 - 1, v0, v0 + width - 1, v0 + width, v0 + width // 2, v0 + width // 2 - 1, v0 + width * (n - 1),
             V - 1, -1, V]
    t[: len(edges)] = edges
    lp, lse = check(h, w, t, 1.0 / 0.9, f"narrow last round {R}x{H}x{V}")
    assert lp[8] == 0 and np.isnan(lp[9])


def test_temperature_masking_and_invalid_targets():
    rng = np.random.Generator(np.random.PCG64(7))
    R, H, V = 400, 256, 1500
    h = rand_bits(rng, (R, H))
    w = rand_bits(rng, (V, H), 0.08)
    t = rng.integers(0, V, R).astype(np.int32)
    t[rng.random(R) < 0.1] = -1
    t[[3, 50, 399]] = [V, -2, 1 << 30]
    lp, lse = check(h, w, t, 1.0 / 0.7, "temperature+mask")
    assert (lp[t == -1] == 0).all()
    assert np.isnan(lp[[3, 50, 399]]).all() and np.isfinite(lse).all()


def test_probabilities_sum_to_one():
    x = W.make_logprob_inputs(W.LOGPROB_CONFIGS["tiny"], "cpu", w_std=0.5)
    V = x.cfg.vocab
    h = W.bf16_bits(x.hidden)
    hh = np.repeat(h, V, axis=0)
    t = np.tile(np.arange(V, dtype=np.int32), x.cfg.rows)
    say("logprob sum to one")
    lp, _ = run_gpu(hh, W.bf16_bits(x.w_lm), t)
    sums = np.exp(lp.astype(np.float64).reshape(x.cfg.rows, V)).sum(1)
    assert np.abs(sums - 1).max() <= 1e-3, sums


def test_id_probe_bit_exact():
    """Logits that encode the vocabulary id: the gathered logit names the target exactly."""
    R, H, V = 700, 64, 151936
    rng = np.random.Generator(np.random.PCG64(8))
    t = rng.integers(0, V, R).astype(np.int32)
    t[:4] = [0, V - 1, 255, 256]
    for col, code in ((0, lambda v: (v % 251) / 16.0), (1, lambda v: (v // 251 % 256) / 16.0)):
        h = np.zeros((R, H), np.float32); h[:, col] = 1.0
        w = np.zeros((V, H), np.float32); w[:, col] = code(np.arange(V))
        bits = lambda a: W.bf16_bits(torch.from_numpy(a).to(torch.bfloat16))
        say(f"logprob id probe col {col}")
        lp, lse = run_gpu(bits(h), bits(w), t)
        z = (lp.astype(np.float64) + lse.astype(np.float64)) * 16.0
        assert np.array_equal(np.rint(z), code(t) * 16.0), "gathered the wrong id"
        assert np.abs(z - np.rint(z)).max() < 0.05


def test_row_permutation_bitwise():
    rng = np.random.Generator(np.random.PCG64(9))
    R, H, V = 600, 128, 3000
    h = rand_bits(rng, (R, H))
    w = rand_bits(rng, (V, H), 0.05)
    t = rng.integers(0, V, R).astype(np.int32)
    perm = rng.permutation(R)
    say("logprob permutation")
    lp1, lse1 = run_gpu(h, w, t)
    lp2, lse2 = run_gpu(h[perm], w, t[perm])
    assert np.array_equal(lp1[perm].view(np.uint32), lp2.view(np.uint32))
    assert np.array_equal(lse1[perm].view(np.uint32), lse2.view(np.uint32))
    lp3, _ = run_gpu(h, w, t)
    assert np.array_equal(lp1.view(np.uint32), lp3.view(np.uint32)), "not deterministic"


def test_many_rows_every_row():
    """40000 rows (more than 32768: the one-thread-per-row combine; 157 row
    tiles: the two-stage weight ring), small hidden size and vocabulary, so
    the oracle checks every row."""
    rng = np.random.Generator(np.random.PCG64(12))
    R, H, V = 40000, 64, 700
    h = rand_bits(rng, (R, H))
    w = rand_bits(rng, (V, H), 0.1)
    t = rng.integers(0, V, R).astype(np.int32)
    t[rng.random(R) < 0.05] = -1
    lp, _ = check(h, w, t, 1.0, "40000 rows, every row")
    assert (lp[t == -1] == 0).all()


@pytest.mark.slow
@pytest.mark.parametrize("name,ntiles", [("8b", 64), ("32b", 64), ("policy", 126)])
def test_full_size_workloads(name, ntiles):
    """Full-size runs; the oracle recomputes rows 0 and R - 1 and one seeded
    row in each of `ntiles` distinct 256-row tiles (the last included; all the
    tiles of the 8B- and 32B-class rows, 127 of the policy pass's 1024 tiles:
    128 rows, about 4 s of oracle time on 16 cores)."""
    cfg = W.LOGPROB_CONFIGS[name]
    say(f"logprob full-size {name}: generating")
    x = W.make_logprob_inputs(cfg, dev())
    say(f"logprob full-size {name}: gpu")
    lp, lse = rk.token_logprob(x.hidden, x.w_lm, x.target, x.inv_temperature)
    torch.cuda.synchronize()
    rows = tile_sample(cfg.rows, ntiles, seed=11)
    if cfg.rows <= 512:
        rows = np.unique(np.concatenate([rows, np.arange(0, cfg.rows, 8)]))   # a row in every 8
    idx = torch.from_numpy(rows).to(dev())
    say(f"logprob full-size {name}: oracle on {len(rows)} rows")
    rlp, rlse = oracle.token_logprob(W.bf16_bits(x.hidden[idx]), W.bf16_bits(x.w_lm),
                                     x.target[idx].cpu().numpy(), x.inv_temperature)
    e1 = max_abs(lp[idx].cpu().numpy(), rlp)
    e2 = max_abs(lse[idx].cpu().numpy(), rlse)
    say(f"logprob full-size {name}: logprob max-abs {e1:.3g}, lse max-abs {e2:.3g}")
    assert e1 <= LOGPROB_TOL and e2 <= LOGPROB_TOL
    assert torch.isfinite(lp).all() and torch.isfinite(lse).all()


@pytest.mark.parametrize("R,H,V", [(256, 5120, 151936), (512, 4096, 151936), (300, 128, 20000)])
def test_timeline_same_outputs_and_complete_records(R, H, V):
    """rl_debug_logprob_timeline: the same log-prob and lse as rl_token_logprob
    bit for bit (the instrumented kernels do the same arithmetic), and one
    record per wave of every tile launch, with ordered timestamps.  The shapes:
    32B-class rows (whole tiles + tail parts), 8B-class rows (whole tiles +
    narrow last round) and a ragged small shape."""
    say(f"timeline {R}x{H}x{V}")
    x = W.make_logprob_inputs(W.LogprobConfig("t", R, H, V), dev())
    lp0, lse0 = rk.token_logprob(x.hidden, x.w_lm, x.target, x.inv_temperature)
    lp, lse, rec = rk.token_logprob_timeline(x.hidden, x.w_lm, x.target, x.inv_temperature)
    torch.cuda.synchronize()
    assert torch.equal(lp, lp0) and torch.equal(lse, lse0)
    r = rec.cpu().numpy()
    assert len(r) == rk.logprob_timeline_records(R, H, V)
    kind, wave, blk = (r[:, 0] >> 40) & 0xFF, (r[:, 0] >> 48) & 0xFF, r[:, 7] & 0xFFFFFFFF
    xcc = (r[:, 0] >> 32) & 0xFF
    assert set(kind.tolist()) <= {0, 1, 2} and (xcc < 8).all()
    # record 8 b + w of each launch is workgroup b, wave w (8 waves per tile workgroup)
    for k in set(kind.tolist()):
        m = kind == k
        n = int(m.sum())
        assert n % 8 == 0
        assert (blk[m] == np.arange(n) // 8).all() and (wave[m] == np.arange(n) % 8).all()
    st, l0, l1, en = (r[:, i] for i in range(1, 5))
    assert (st > 0).all() and (st <= l0).all() and (l0 <= l1).all() and (l1 <= en).all()
    assert (r[:, 5] <= r[:, 6]).all() and (r[:, 6] > 0).all()     # stage-end waits within the loop's cycles
    stages, samples = (r[:, 7] >> 32) & 0xFFFF, r[:, 7] >> 48
    assert (stages > 0).all() and (samples == (stages + 4) // 8).all()   # stages 3, 11, 19, ... sampled
    if R == 256:
        assert {0, 2} <= set(kind.tolist())
    if R == 512:
        assert {0, 1} <= set(kind.tolist())


def test_vocabulary_of_two_million():
    """vocab = 2^21: 8192 vocabulary tiles, so each row's combine merges 8192
    partial slots; targets include a masked row and the last id."""
    rng = np.random.Generator(np.random.PCG64(2021))
    R, H, V = 8, 64, 1 << 21
    h, w = rand_bits(rng, (R, H)), rand_bits(rng, (V, H), 0.05)
    t = rng.integers(0, V, R).astype(np.int32)
    t[0], t[-1] = -1, V - 1
    lp, _ = check(h, w, t, 1.0, "vocab 2^21")
    assert lp[0] == 0.0
