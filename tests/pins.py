"""Pins of the fp64 oracle against things other than itself.

Each function takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with what the mathematics fixes:

* independent library routines on tiny inputs: torch's fp64 CPU
  scaled_dot_product_attention (with its own grouped-query head expansion),
  torch.logsumexp and torch.log_softmax;
* closed forms (one token, zero query, equal keys, zero weights);
* invariants (prefix sharing == concatenation, token permutation, vocab
  chunking with a log-sum-exp merge, constant shift, sum of probabilities);
* exact probes (one-hot attention returns one value row bit for bit; uniform
  attention recovers the context length; an id probe recovers the target);
* hand-derived worked examples under tests/golden/;
* for the GRPO pieces and the backward: hand-worked regimes of the clipped
  objective, the statistics that define the advantages, central finite
  differences of the oracle's own loss / forward, the two-class logistic
  gradient, and torch autograd in fp64;
* for nucleus sampling: the top_p = 1 reduction to numpy's inverse CDF of
  torch's softmax, the greedy limit (torch argmax), sample frequencies over a
  uniform grid against the renormalised nucleus, ties broken by id, the
  temperature / hidden-scale equivalence, the log-prob against torch's
  log_softmax, and hand-worked cases.

The same battery runs against deliberately broken copies of the oracle
(test_oracle_mutants.py) to show that each plausible mistake is caught.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch
import torch.nn.functional as F

import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------- helpers
def f64(bits: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bits -> float64 tensor (exact)."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).double()


def bf16_bits_of(x: np.ndarray) -> np.ndarray:
    """float64 values -> bf16 bit patterns (RNE); exact for bf16-representable values."""
    return W.bf16_bits(torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16))


def decode_case(P=2, G=3, Hq=4, Hkv=2, D=8, lp=None, ls=None, seed=0, qmul=1.0):
    """Small random decode input as bf16 bit arrays + host length arrays."""
    rng = np.random.Generator(np.random.PCG64(seed))
    S = P * G
    lp = np.asarray(rng.integers(0, 7, P) if lp is None else lp, dtype=np.int32)
    ls = np.asarray(rng.integers(0, 6, S) if ls is None else ls, dtype=np.int32)
    # leave gaps between sequences so a wrong start index reads other rows
    ps = np.cumsum(np.concatenate([[1], lp[:-1] + 2])).astype(np.int64)
    ss = np.cumsum(np.concatenate([[2], ls[:-1] + 1])).astype(np.int64)
    prow = int(ps[-1] + lp[-1] + 3) if P else 1
    srow = int(ss[-1] + ls[-1] + 3) if S else 1
    def rn(*shape, mul=1.0):
        return bf16_bits_of(rng.standard_normal(shape) * mul)
    return dict(q=rn(S, Hq, D, mul=qmul), k_prefix=rn(prow, Hkv, D), v_prefix=rn(prow, Hkv, D),
                k_suffix=rn(srow, Hkv, D), v_suffix=rn(srow, Hkv, D),
                prefix_start=ps, prefix_len=lp, suffix_start=ss, suffix_len=ls,
                group_size=G, scale=float(np.float32(1.0 / math.sqrt(D))))


def torch_attention(c):
    """Reference via torch's fp64 SDPA on the concatenated context of each candidate."""
    q = f64(c["q"]); kp = f64(c["k_prefix"]); vp = f64(c["v_prefix"])
    ks = f64(c["k_suffix"]); vs = f64(c["v_suffix"])
    S, Hq, D = q.shape
    Hkv = kp.shape[1]
    G = c["group_size"]
    sigma = float(np.float32(c["scale"]))
    out = torch.zeros(S, Hq, D, dtype=torch.float64)
    lse = torch.full((S, Hq), -math.inf, dtype=torch.float64)
    for s in range(S):
        p = s // G
        a, n = int(c["prefix_start"][p]), int(c["prefix_len"][p])
        b, m = int(c["suffix_start"][s]), int(c["suffix_len"][s])
        K = torch.cat([kp[a:a + n], ks[b:b + m]])          # [T, Hkv, D]
        V = torch.cat([vp[a:a + n], vs[b:b + m]])
        if K.shape[0] == 0:
            continue
        o = F.scaled_dot_product_attention(q[s][None, :, None, :], K.permute(1, 0, 2)[None],
                                           V.permute(1, 0, 2)[None], scale=sigma, enable_gqa=True)
        out[s] = o[0, :, 0, :]
        Krep = K.repeat_interleave(Hq // Hkv, dim=1)         # [T, Hq, D]
        scores = sigma * (Krep.permute(1, 0, 2) @ q[s][:, :, None])[..., 0]   # [Hq, T]
        lse[s] = torch.logsumexp(scores, dim=1)
    return out.numpy(), lse.numpy()


def logprob_case(R=5, H=16, V=37, seed=0, w_std=0.3, targets=None):
    rng = np.random.Generator(np.random.PCG64(seed))
    hidden = bf16_bits_of(rng.standard_normal((R, H)))
    w = bf16_bits_of(rng.standard_normal((V, H)) * w_std)
    t = rng.integers(0, V, R).astype(np.int32) if targets is None else np.asarray(targets, np.int32)
    return hidden, w, t


def torch_logprob(hidden, w, target, inv_T):
    z = float(np.float32(inv_T)) * (f64(hidden) @ f64(w).T)
    ls = torch.log_softmax(z, dim=1)
    lse = torch.logsumexp(z, dim=1)
    out = torch.zeros(len(target), dtype=torch.float64)
    for r, t in enumerate(target):
        out[r] = 0.0 if t == -1 else (ls[r, t] if 0 <= t < w.shape[0] else math.nan)
    return out.numpy(), lse.numpy()


def close(a, b, tol, what):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    same_inf = (np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))) | (np.isnan(a) & np.isnan(b))
    with np.errstate(invalid="ignore"):
        err = np.where(same_inf, 0.0, np.abs(a - b))
    err = np.where(np.isnan(err), np.inf, err)
    assert err.max(initial=0.0) <= tol, f"{what}: max err {err.max()} > {tol}"


# ------------------------------------------------------------ attention pins
def pin_attention_vs_torch(orc):
    """A1: brute force by an independent library routine on small shapes."""
    cases = [
        dict(P=2, G=4, Hq=4, Hkv=1, D=64, lp=[128, 128], ls=[32] * 8, seed=0),   # tiny-config shape
        dict(P=3, G=2, Hq=4, Hkv=2, D=8, seed=1),
        dict(P=2, G=3, Hq=6, Hkv=3, D=16, seed=2),
        dict(P=1, G=5, Hq=2, Hkv=2, D=8, lp=[0], seed=3),              # no prefix
        dict(P=2, G=2, Hq=8, Hkv=1, D=8, ls=[0, 0, 0, 0], seed=4),      # no suffix
        dict(P=2, G=2, Hq=4, Hkv=2, D=8, lp=[0, 3], ls=[0, 2, 0, 0], seed=5, qmul=4.0),  # empty contexts, peaky
    ]
    for cs in cases:
        c = decode_case(**cs)
        o, l = orc.decode_attn(**c)
        ro, rl = torch_attention(c)
        close(o, ro, 1e-12, f"out {cs}")
        close(l, rl, 1e-12, f"lse {cs}")


def pin_prefix_sharing(orc):
    """A2: a shared prefix equals concatenating it into every candidate's suffix."""
    c = decode_case(P=2, G=3, Hq=4, Hkv=2, D=8, lp=[5, 3], ls=[2, 0, 4, 1, 3, 2], seed=7)
    o, l = orc.decode_attn(**c)
    S, G = 6, 3
    kp, vp, ks, vs = c["k_prefix"], c["v_prefix"], c["k_suffix"], c["v_suffix"]
    krows, vrows, starts, lens = [], [], [], []
    pos = 0
    for s in range(S):
        p = s // G
        a, n = c["prefix_start"][p], c["prefix_len"][p]
        b, m = c["suffix_start"][s], c["suffix_len"][s]
        krows.append(np.concatenate([kp[a:a + n], ks[b:b + m]]))
        vrows.append(np.concatenate([vp[a:a + n], vs[b:b + m]]))
        starts.append(pos); lens.append(n + m); pos += n + m
    c2 = dict(c, k_prefix=kp[:1], v_prefix=vp[:1], prefix_start=np.zeros(2, np.int64),
              prefix_len=np.zeros(2, np.int32), k_suffix=np.concatenate(krows),
              v_suffix=np.concatenate(vrows), suffix_start=np.array(starts, np.int64),
              suffix_len=np.array(lens, np.int32))
    o2, l2 = orc.decode_attn(**c2)
    close(o, o2, 1e-12, "prefix sharing out")
    close(l, l2, 1e-12, "prefix sharing lse")


def pin_attention_closed_forms(orc):
    """A3: one token -> that value row; zero query -> mean of values, lse = ln T."""
    # one prefix token, no suffix
    c = decode_case(P=1, G=2, Hq=2, Hkv=1, D=8, lp=[1], ls=[0, 0], seed=11)
    o, l = orc.decode_attn(**c)
    v0 = f64(c["v_prefix"])[c["prefix_start"][0], 0].numpy()
    k0 = f64(c["k_prefix"])[c["prefix_start"][0], 0].numpy()
    q = f64(c["q"]).numpy()
    for s in range(2):
        for h in range(2):
            close(o[s, h], v0, 0.0, "T=1 out")
            close(l[s, h], float(np.float32(c["scale"])) * float(q[s, h] @ k0), 1e-13, "T=1 lse")
    # zero query: uniform weights
    c = decode_case(P=2, G=2, Hq=4, Hkv=2, D=8, lp=[3, 2], ls=[1, 4, 0, 2], seed=12)
    c["q"] = np.zeros_like(c["q"])
    o, l = orc.decode_attn(**c)
    vp, vs = f64(c["v_prefix"]).numpy(), f64(c["v_suffix"]).numpy()
    for s in range(4):
        p = s // 2
        a, n = c["prefix_start"][p], c["prefix_len"][p]
        b, m = c["suffix_start"][s], c["suffix_len"][s]
        for h in range(4):
            kh = h // 2
            V = np.concatenate([vp[a:a + n, kh], vs[b:b + m, kh]])
            close(o[s, h], V.mean(0), 1e-14, "q=0 mean")
            close(l[s, h], math.log(n + m), 1e-14, "q=0 lse")


def pin_permutation(orc):
    """A5: permuting the suffix tokens of a candidate changes nothing."""
    c = decode_case(P=1, G=2, Hq=4, Hkv=2, D=8, lp=[4], ls=[6, 5], seed=13)
    o, l = orc.decode_attn(**c)
    c2 = dict(c)
    ks, vs = c["k_suffix"].copy(), c["v_suffix"].copy()
    rng = np.random.Generator(np.random.PCG64(1))
    for s in range(2):
        b, m = c["suffix_start"][s], c["suffix_len"][s]
        perm = b + rng.permutation(m)
        ks[b:b + m] = c["k_suffix"][perm]
        vs[b:b + m] = c["v_suffix"][perm]
    c2["k_suffix"], c2["v_suffix"] = ks, vs
    o2, l2 = orc.decode_attn(**c2)
    close(o, o2, 1e-13, "perm out")
    close(l, l2, 1e-13, "perm lse")


def pin_one_hot_probe(orc):
    """A6: a single dominant key returns its value row exactly (indexing, bit-exact).

    Every key is zero except one per (sequence, kv head), which equals the query
    direction scaled so its score beats all others by >= 200: every other weight
    is exp(-200) relative, far below the resolution of the sum, so the output is
    that token's value row up to fp64 rounding of a weight of 1.  Value rows
    encode (prefix/suffix, kv head, position) as small integers.
    """
    P, G, Hq, Hkv, D = 2, 2, 4, 2, 8
    S, r = P * G, Hq // Hkv
    lp, ls = np.array([5, 7], np.int32), np.array([3, 0, 4, 6], np.int32)
    c = decode_case(P=P, G=G, Hq=Hq, Hkv=Hkv, D=D, lp=lp, ls=ls, seed=14)
    q = np.zeros((S, Hq, D)); q[:, :, 0] = 1.0
    kp = np.zeros((len(c["k_prefix"]), Hkv, D)); ks = np.zeros((len(c["k_suffix"]), Hkv, D))
    vp = np.zeros_like(kp); vs = np.zeros_like(ks)
    for arr, tag in ((vp, 1), (vs, 2)):
        for row in range(arr.shape[0]):
            for kh in range(Hkv):
                arr[row, kh, :4] = [tag, kh, row % 16, row // 16]
    rng = np.random.Generator(np.random.PCG64(5))
    expect = np.zeros((S, Hq, D))
    chosen = {}
    for p in range(P):
        for kh in range(Hkv):
            j = int(rng.integers(0, lp[p]))
            chosen[(p, kh)] = ("p", int(c["prefix_start"][p] + j))
    for s in range(S):
        p = s // G
        for kh in range(Hkv):
            if ls[s] and (s % 2 == 0):
                j = int(rng.integers(0, ls[s]))
                row = int(c["suffix_start"][s] + j)
                ks[row, kh, 0] = 2048.0
                src = vs[row, kh]
            else:
                kind, row = chosen[(p, kh)]
                src = vp[row, kh]
            for h in range(kh * r, (kh + 1) * r):
                expect[s, h] = src
    for (p, kh), (_, row) in chosen.items():
        kp[row, kh, 0] = 1024.0
    c.update(q=bf16_bits_of(q), k_prefix=bf16_bits_of(kp), k_suffix=bf16_bits_of(ks),
             v_prefix=bf16_bits_of(vp), v_suffix=bf16_bits_of(vs), scale=1.0)
    o, _ = orc.decode_attn(**c)
    close(o, expect, 1e-9, "one-hot probe")
    assert np.array_equal(np.rint(o), expect), "one-hot probe indices"


def pin_length_probe(orc):
    """A7: zero keys -> uniform weights -> exp(lse) is the context length."""
    c = decode_case(P=3, G=2, Hq=2, Hkv=1, D=8, lp=[0, 9, 4], ls=[3, 0, 1, 5, 0, 0], seed=15)
    c["k_prefix"] = np.zeros_like(c["k_prefix"])
    c["k_suffix"] = np.zeros_like(c["k_suffix"])
    o, l = orc.decode_attn(**c)
    T = np.array([c["prefix_len"][s // 2] + c["suffix_len"][s] for s in range(6)])
    for s in range(6):
        for h in range(2):
            if T[s] == 0:
                assert l[s, h] == -math.inf and not o[s, h].any(), "empty context"
            else:
                assert round(math.exp(l[s, h])) == T[s], "length probe"


def pin_attention_golden(orc):
    """Hand-derived worked examples (tests/golden/attention_hand.json)."""
    with open(os.path.join(GOLDEN, "attention_hand.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        c = dict(q=bf16_bits_of(np.array(case["q"], np.float64)),
                 k_prefix=bf16_bits_of(np.array(case["k_prefix"], np.float64)),
                 v_prefix=bf16_bits_of(np.array(case["v_prefix"], np.float64)),
                 k_suffix=bf16_bits_of(np.array(case["k_suffix"], np.float64)),
                 v_suffix=bf16_bits_of(np.array(case["v_suffix"], np.float64)),
                 prefix_start=np.array(case["prefix_start"], np.int64),
                 prefix_len=np.array(case["prefix_len"], np.int32),
                 suffix_start=np.array(case["suffix_start"], np.int64),
                 suffix_len=np.array(case["suffix_len"], np.int32),
                 group_size=case["group_size"], scale=case["scale"])
        o, l = orc.decode_attn(**c)
        close(o, np.array(case["out"]), 1e-15, case["name"] + " out")
        close(l, np.array(case["lse"]), 1e-15, case["name"] + " lse")


# -------------------------------------------------------------- log-prob pins
def pin_logprob_vs_torch(orc):
    """L1: brute force by torch.log_softmax on materialised fp64 logits."""
    for (R, H, V, seed, invT, tg) in [
        (5, 16, 37, 0, 1.0, None),
        (8, 256, 1024, 1, 1.0, None),                  # tiny-config shape
        (6, 32, 50, 2, 1.0 / 0.7, [3, -1, 49, 0, -1, 7]),  # temperature, masked rows
        (3, 8, 11, 3, 1.0, [11, -2, 5]),               # invalid ids -> NaN
    ]:
        h, w, t = logprob_case(R, H, V, seed, targets=tg)
        lp, lse = orc.token_logprob(h, w, t, invT)
        rlp, rlse = torch_logprob(h, w, t, invT)
        close(lp, rlp, 1e-12, f"logprob {R}x{H}x{V}")
        close(lse, rlse, 1e-12, f"lse {R}x{H}x{V}")


def pin_logprob_sum_to_one(orc):
    """L2: exp(logprob) over every vocabulary id sums to 1."""
    h, w, _ = logprob_case(4, 24, 300, seed=4, w_std=1.0)
    V = w.shape[0]
    hh = np.repeat(h, V, axis=0)
    t = np.tile(np.arange(V, dtype=np.int32), 4)
    lp, _ = orc.token_logprob(hh, w, t, 1.0)
    sums = np.exp(lp.reshape(4, V)).sum(1)
    close(sums, np.ones(4), 1e-12, "sum of probabilities")


def pin_logprob_closed_forms(orc):
    """L3: zero weights -> every logit 0 -> logprob = -ln V and lse = ln V."""
    h, w, t = logprob_case(3, 16, 1024, seed=5)
    lp, lse = orc.token_logprob(h, np.zeros_like(w), t, 1.0)
    close(lp, np.full(3, -math.log(1024)), 1e-15, "W=0 logprob")
    close(lse, np.full(3, math.log(1024)), 1e-15, "W=0 lse")


def pin_logprob_shift(orc):
    """L4: a constant extra hidden column times a constant W column shifts every logit alike."""
    h, w, t = logprob_case(4, 15, 40, seed=6)
    lp, lse = orc.token_logprob(h, w, t, 1.0)
    h2 = np.concatenate([h, bf16_bits_of(np.full((4, 1), 2.0))], 1)
    w2 = np.concatenate([w, bf16_bits_of(np.full((40, 1), 1.5))], 1)
    lp2, lse2 = orc.token_logprob(h2, w2, t, 1.0)
    close(lp2, lp, 1e-12, "shift logprob")
    close(lse2, lse + 3.0, 1e-12, "shift lse")


def pin_logprob_chunks(orc):
    """L5: per-vocab-chunk results merged by log-sum-exp equal one full pass."""
    h, w, t = logprob_case(6, 32, 100, seed=7)
    lp, lse = orc.token_logprob(h, w, t, 1.0 / 0.7)
    bounds = [0, 17, 50, 64, 100]
    lses, zt = [], np.zeros(6)
    for a, b in zip(bounds[:-1], bounds[1:]):
        tt = np.where((t >= a) & (t < b), t - a, -1).astype(np.int32)
        lpc, lsec = orc.token_logprob(h, w[a:b], tt, 1.0 / 0.7)
        lses.append(lsec)
        zt += np.where(tt >= 0, lpc + lsec, 0.0)     # the target's logit, from its own chunk
    merged = torch.logsumexp(torch.tensor(np.stack(lses)), dim=0).numpy()
    close(merged, lse, 1e-12, "chunked lse")
    close(zt - merged, lp, 1e-12, "chunked logprob")


def pin_logprob_id_probe(orc):
    """L6: logits that encode the vocabulary id recover the gathered id exactly."""
    R, H, V = 6, 8, 1000
    rng = np.random.Generator(np.random.PCG64(8))
    t = rng.integers(0, V, R).astype(np.int32)
    for col, code in ((0, lambda v: (v % 251) / 16.0), (1, lambda v: (v // 251) / 16.0)):
        h = np.zeros((R, H)); h[:, col] = 1.0
        w = np.zeros((V, H)); w[:, col] = [code(v) for v in range(V)]
        lp, lse = orc.token_logprob(bf16_bits_of(h), bf16_bits_of(w), t, 1.0)
        got = (lp + lse) * 16.0
        assert np.array_equal(np.rint(got), np.array([code(v) * 16 for v in t])), "id probe"
        close(got, np.rint(got), 1e-9, "id probe exactness")


def pin_logprob_golden(orc):
    """Hand-derived worked examples (tests/golden/logprob_hand.json)."""
    with open(os.path.join(GOLDEN, "logprob_hand.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        lp, lse = orc.token_logprob(bf16_bits_of(np.array(case["hidden"], np.float64)),
                                    bf16_bits_of(np.array(case["w_lm"], np.float64)),
                                    np.array(case["target"], np.int32), case["inv_temperature"])
        close(lp, np.array(case["logprob"], dtype=np.float64), 1e-15, case["name"] + " logprob")
        close(lse, np.array(case["lse"]), 1e-15, case["name"] + " lse")


# ------------------------------------------------------------ GRPO pins
# (Sec. 3, Eq. grpo-loss and the advantage definition under it)
def pin_advantage_closed_form(orc):
    """G1: rewards 1, 2, 3, 4: mean 2.5, sample variance 5/3 -> (r - 2.5) / sqrt(5/3);
    a group of equal rewards and a group of one give 0."""
    sd = math.sqrt(5.0 / 3.0)
    got = orc.grpo_advantage([1.0, 2.0, 3.0, 4.0, 7.0, 7.0, 7.0, 7.0], 4)
    close(got, [-1.5 / sd, -0.5 / sd, 0.5 / sd, 1.5 / sd, 0, 0, 0, 0], 1e-15, "advantage 1..4")
    close(orc.grpo_advantage([3.0, -2.0], 1), [0.0, 0.0], 0.0, "group of one")


def pin_advantage_invariants(orc):
    """G2: per group the advantages sum to 0 and have sample variance 1; they do not
    change under r -> a r + b (a > 0) and follow a permutation of the candidates."""
    rng = np.random.Generator(np.random.PCG64(11))
    P, G = 5, 16
    r = rng.standard_normal(P * G) * 3.0 + 1.0
    a = orc.grpo_advantage(r, G).reshape(P, G)
    close(a.sum(1), np.zeros(P), 1e-12, "advantage sum")
    close((a * a).sum(1) / (G - 1), np.ones(P), 1e-12, "advantage variance")
    close(orc.grpo_advantage(2.5 * r + 7.0, G).reshape(P, G), a, 1e-12, "affine invariance")
    perm = rng.permutation(G)
    close(orc.grpo_advantage(r.reshape(P, G)[:, perm].reshape(-1), G).reshape(P, G), a[:, perm], 1e-15,
          "permutation")


def surrogate_case(seed=12, P=3, G=4, lo=1, hi=9, spread=0.15):
    """Random token rows of P*G candidates (some rows belong to none) with ratios
    exp(logp_new - logp_old) kept away from the clip bounds 0.8 and 1.2."""
    rng = np.random.Generator(np.random.PCG64(seed))
    S = P * G
    counts = rng.integers(lo, hi, S)
    seq = np.repeat(np.arange(S, dtype=np.int32), counts)
    seq = np.concatenate([seq, np.full(5, -1, np.int32)])
    rng.shuffle(seq)
    R = len(seq)
    old = rng.uniform(-6.0, -0.1, R)
    d = rng.uniform(-spread, spread, R)
    log_bounds = np.log([0.8, 1.2])
    for b in log_bounds:                                  # at least 1e-3 from each bound
        near = np.abs(d - b) < 1e-3
        d[near] += 3e-3
    adv = random_advantages(rng, P, G)
    return old + d, old, seq, adv


def random_advantages(rng, P, G):
    a = rng.standard_normal((P, G))
    return a.reshape(-1)


def pin_surrogate_finite_differences(orc):
    """G3: the returned gradient is the derivative of the returned loss (central
    differences, every row, ratios inside, below and above the clip range)."""
    for seed, spread in ((12, 0.1), (13, 0.6)):
        new, old, seq, adv = surrogate_case(seed, spread=spread)
        loss, grad = orc.grpo_surrogate(new, old, seq, adv, 4, 0.2)
        h = 1e-6
        fd = np.zeros_like(new)
        for r in range(len(new)):
            e = np.zeros_like(new); e[r] = h
            lp, _ = orc.grpo_surrogate(new + e, old, seq, adv, 4, 0.2)
            lm, _ = orc.grpo_surrogate(new - e, old, seq, adv, 4, 0.2)
            fd[r] = (lp - lm) / (2 * h)
        close(grad, fd, 1e-8, f"surrogate gradient (spread {spread})")


def pin_surrogate_closed_forms(orc):
    """G4: hand-worked cases.
    * ratio 1 everywhere: L = -(1/(P G)) sum_i A_i (each candidate's token mean is A_i),
      dL/dlogp = -A_i / (P G |o_i|);
    * one candidate with one token per regime (A = +-1, ratio e^{+-0.5}, eps = 0.2):
      A=+1, ratio 1.6487 -> clipped 1.2, gradient 0; A=-1, ratio 0.6065 -> clipped -0.8,
      gradient 0; A=-1, ratio 1.6487 -> the ratio term -1.6487 is the minimum; A=+1,
      ratio 0.6065 -> the ratio term 0.6065 is the minimum."""
    P, G = 2, 3
    seq = np.array([0, 0, 1, 2, 2, 2, 3, 5, 5, -1], np.int32)        # candidate 4 has no tokens
    adv = np.array([1.0, -0.5, 2.0, 0.25, 3.0, -1.0])
    z = np.full(len(seq), -2.0)
    loss, grad = orc.grpo_surrogate(z, z, seq, adv, G, 0.2)
    counts = np.bincount(seq[seq >= 0], minlength=6)
    close(loss, -(adv[counts > 0].sum()) / (P * G), 1e-15, "ratio-1 loss")
    want = np.array([-adv[i] / (P * G * counts[i]) if i >= 0 else 0.0 for i in seq])
    close(grad, want, 1e-15, "ratio-1 gradient")
    e = math.exp(0.5)
    for a, d, term, g in ((1.0, 0.5, 1.2, 0.0), (-1.0, -0.5, -0.8, 0.0),
                          (-1.0, 0.5, -e, e), (1.0, -0.5, 1 / e, -1 / e)):
        loss, grad = orc.grpo_surrogate([d], [0.0], [0], [a], 1, 0.2)
        close(loss, -term, 1e-15, f"regime A={a} d={d}")
        close(grad, [g], 1e-15, f"regime gradient A={a} d={d}")


def pin_surrogate_unowned_rows(orc):
    """G5: rows of no candidate (seq = -1) change neither the loss nor the other
    rows' gradients, and get gradient 0."""
    new, old, seq, adv = surrogate_case(14)
    keep = seq >= 0
    l1, g1 = orc.grpo_surrogate(new, old, seq, adv, 4, 0.2)
    l2, g2 = orc.grpo_surrogate(new[keep], old[keep], seq[keep], adv, 4, 0.2)
    close(l1, l2, 1e-15, "loss without unowned rows")
    close(g1[keep], g2, 1e-15, "gradients without unowned rows")
    close(g1[~keep], np.zeros((~keep).sum()), 0.0, "unowned rows")


# --------------------------------------------------------- backward pins
def pin_backward_vs_torch(orc):
    """B1: torch autograd in fp64 on the CPU (log_softmax, gather, sum g * logprob)."""
    for R, H, V, seed, invT in ((4, 16, 37, 20, 1.0), (3, 24, 90, 21, 1 / 0.7)):
        h, w, t = logprob_case(R, H, V, seed)
        t[0] = -1
        rng = np.random.Generator(np.random.PCG64(seed + 1))
        g = rng.standard_normal(R)
        dh = orc.token_logprob_backward(h, w, t, g, invT)
        ht = f64(h).clone().requires_grad_(True)
        z = float(np.float32(invT)) * (ht @ f64(w).T)
        ls = torch.log_softmax(z, dim=1)
        keep = torch.tensor(t >= 0)
        tt = torch.tensor(np.where(t >= 0, t, 0).astype(np.int64))
        picked = ls.gather(1, tt[:, None])[:, 0] * keep
        (picked * torch.tensor(g)).sum().backward()
        close(dh, ht.grad.numpy(), 1e-12, f"backward vs torch {R}x{H}x{V}")


def pin_backward_finite_differences(orc):
    """B2: central differences of sum_r g_r logprob_r with respect to every hidden entry."""
    R, H, V = 3, 6, 13
    h, w, t = logprob_case(R, H, V, seed=22)
    g = np.array([0.7, -1.3, 2.0])
    dh = orc.token_logprob_backward(h, w, t, g, 1.0 / 0.9)
    hd = f64(h).numpy()
    step = 1e-6
    fd = np.zeros_like(hd)
    for r in range(R):
        for k in range(H):
            e = np.zeros_like(hd); e[r, k] = step
            lp, _ = orc.token_logprob_f64(hd + e, w, t, 1.0 / 0.9)
            lm, _ = orc.token_logprob_f64(hd - e, w, t, 1.0 / 0.9)
            fd[r, k] = (g * (lp - lm)).sum() / (2 * step)
    close(dh, fd, 1e-7, "backward finite differences")


def pin_backward_closed_forms(orc):
    """B3: two classes: dlogp_t/dh = inv_T (1 - p_t)(W_t - W_o) with p_t the logistic
    of the logit gap (the textbook logistic-regression gradient); equal weight rows give
    0; a masked row gives 0 and an invalid target NaN."""
    h, w, _ = logprob_case(2, 8, 2, seed=23, w_std=1.0)
    t = np.array([0, 1], np.int32)
    invT = 1.5
    dh = orc.token_logprob_backward(h, w, t, np.ones(2), invT)
    H, W2 = f64(h).numpy(), f64(w).numpy()
    for r in range(2):
        o = 1 - t[r]
        gap = invT * (H[r] @ (W2[t[r]] - W2[o]))
        pt = 1.0 / (1.0 + math.exp(-gap))
        close(dh[r], invT * (1 - pt) * (W2[t[r]] - W2[o]), 1e-13, "two-class gradient")
    weq = np.tile(w[:1], (9, 1))
    h3, _, t3 = logprob_case(3, 8, 9, seed=24)
    close(orc.token_logprob_backward(h3, weq, t3, np.ones(3), 1.0), np.zeros((3, 8)), 1e-14, "equal rows")
    t4 = np.array([-1, 9, 4], np.int32)
    dh4 = orc.token_logprob_backward(h3, weq, t4, np.ones(3), 1.0)
    assert np.all(dh4[0] == 0.0) and np.all(np.isnan(dh4[1])), "masked / invalid rows"


# ------------------------------------------------------- nucleus sampling
# (Sec. 3, Multi-turn RL Training: candidates drawn by nucleus sampling with
# p = 0.9 at temperatures 0.2 and 0.7)
def sampling_case(R, H, V, seed, hstd=1.0, wstd=0.3):
    rng = np.random.Generator(np.random.PCG64(seed))
    h = bf16_bits_of(rng.standard_normal((R, H)) * hstd)
    w = bf16_bits_of(rng.standard_normal((V, H)) * wstd)
    return h, w, rng


def torch_probs(h, w, inv_t):
    """softmax(inv_T * h W^T) in fp64 by torch (independent of the oracle)."""
    z = f64(h) @ f64(w).T
    return torch.softmax(z * torch.tensor(np.asarray(inv_t, np.float64))[:, None], dim=1).numpy()


def pin_sampling_full_distribution(orc):
    """S1: with top_p = 1 the nucleus is the whole vocabulary, so the sample is
    the plain inverse CDF of softmax in id order: numpy searchsorted on the
    cumulative sum of torch's softmax."""
    R, H, V = 12, 16, 40
    h, w, rng = sampling_case(R, H, V, seed=41)
    it = np.float32(1 / 0.7) * np.ones(R, np.float32)
    u = rng.random(R)
    tok, _, _ = orc.sample_top_p(h, w, it, 1.0, u)
    p = torch_probs(h, w, it)
    want = np.array([np.searchsorted(np.cumsum(p[r]), u[r] * p[r].sum(), side="right") for r in range(R)])
    assert np.array_equal(tok, want), (tok, want)


def pin_sampling_greedy_limit(orc):
    """S2: a tiny top_p keeps only the most probable token, whatever u is
    (torch argmax; random logits have no ties)."""
    R, H, V = 10, 16, 50
    h, w, rng = sampling_case(R, H, V, seed=42)
    it = np.full(R, 1 / 0.2, np.float32)
    want = torch.argmax(f64(h) @ f64(w).T, dim=1).numpy()
    for u in (np.zeros(R), rng.random(R), np.full(R, 0.999999)):
        tok, _, _ = orc.sample_top_p(h, w, it, 1e-9, u)
        assert np.array_equal(tok, want)


def pin_sampling_frequencies(orc):
    """S3: over a grid of M uniform values the oracle's samples follow the
    renormalised nucleus: token v appears within 1 of M p_v / Z_N times, tokens
    outside the nucleus never.  The nucleus (from torch's softmax) is the
    shortest most-probable prefix reaching top_p: its mass reaches top_p and
    dropping its least probable member falls short."""
    R, H, V, M = 3, 16, 30, 4000
    h, w, _ = sampling_case(R, H, V, seed=43)
    it = np.array([1 / 0.7, 1 / 0.2, 1.0], np.float32)
    p = torch_probs(h, w, it)
    grid = (np.arange(M) + 0.5) / M
    for top_p in (0.9, 0.5):
        for r in range(R):
            tok, _, _ = orc.sample_top_p(np.repeat(h[r:r + 1], M, 0), w, np.full(M, it[r], np.float32),
                                         top_p, grid)
            counts = np.bincount(tok, minlength=V)
            members = np.flatnonzero(counts)
            mass = p[r, members].sum()
            assert mass >= top_p and mass - p[r, members].min() < top_p, "nucleus not minimal"
            order = np.argsort(-p[r], kind="stable")
            assert set(members) == set(order[:len(members)].tolist()), "nucleus not the most probable"
            assert np.all(np.abs(counts[members] - M * p[r, members] / mass) <= 1.0), "frequencies"


def pin_sampling_ties(orc):
    """S4: ten equal logits (identical weight rows), top_p = 0.35: each token
    has p = 0.1, so the nucleus is the four smallest ids (0.3 < 0.35 <= 0.4);
    u = 0.6 puts the target at 0.24 of the nucleus mass 0.4: the third id."""
    h = bf16_bits_of(np.array([[1.0, 2.0]]))
    w = bf16_bits_of(np.tile([[0.5, -0.25]], (10, 1)))
    for u, want in ((0.6, 2), (0.0, 0), (0.99, 3), (0.26, 1)):
        tok, lp, _ = orc.sample_top_p(h, w, np.ones(1, np.float32), 0.35, np.array([u]))
        assert tok[0] == want, (u, tok[0], want)
        close(lp, [-math.log(10.0)], 1e-15, "tie log-prob")


def pin_sampling_temperature_scale(orc):
    """S5: inv_T = 2 on hidden h samples as inv_T = 1 on hidden 2h (the
    doubling is exact in bf16), for the same u."""
    R, H, V = 16, 8, 60
    h, w, rng = sampling_case(R, H, V, seed=44, hstd=0.5)
    u = rng.random(R)
    a = orc.sample_top_p(h, w, np.full(R, 2.0, np.float32), 0.9, u)
    b = orc.sample_top_p(bf16_bits_of(f64(h).numpy() * 2.0), w, np.ones(R, np.float32), 0.9, u)
    assert np.array_equal(a[0], b[0])
    close(a[1], b[1], 1e-12, "temperature scale log-prob")


def pin_sampling_logprob(orc):
    """S6: the returned log-prob is the full-vocabulary log-prob of the sampled
    token (the pinned token_logprob, and torch's log_softmax)."""
    R, H, V = 9, 16, 70
    h, w, rng = sampling_case(R, H, V, seed=45)
    inv_t = np.float32(1 / 0.7)
    tok, lp, _ = orc.sample_top_p(h, w, np.full(R, inv_t, np.float32), 0.9, rng.random(R))
    want, _ = orc.token_logprob(h, w, tok, float(inv_t))
    close(lp, want, 1e-12, "sample log-prob vs token_logprob")
    ls = torch.log_softmax(f64(h) @ f64(w).T * float(inv_t), dim=1).numpy()
    close(lp, ls[np.arange(R), tok], 1e-12, "sample log-prob vs log_softmax")


def pin_sampling_intervals(orc):
    """S7: the intervals of u that map to each token tile [0, 1) in id order,
    one per nucleus member, each as long as the member's share of the
    nucleus mass (torch's softmax); the sampled token's interval holds u."""
    H, V = 16, 40
    h, w, rng = sampling_case(1, H, V, seed=46)
    for inv_t, top_p in ((1 / 0.7, 0.9), (1 / 0.2, 0.9), (1.0, 0.5), (1.0, 1.0)):
        it = np.float32(inv_t)
        lo, hi = orc.top_p_interval(np.repeat(h, V, 0), w, np.full(V, it, np.float32), top_p,
                                    np.arange(V, dtype=np.int32))
        members = np.flatnonzero(lo >= 0)
        p = torch_probs(h, w, [it])[0]
        share = p[members] / p[members].sum()
        close(hi[members] - lo[members], share, 1e-12, "interval lengths")
        close(lo[members], np.concatenate([[0.0], np.cumsum(share)[:-1]]), 1e-12, "intervals in id order")
        assert np.all(hi[lo < 0] == -1.0)
        u = rng.random(8)
        tok, _, _ = orc.sample_top_p(np.repeat(h, 8, 0), w, np.full(8, it, np.float32), top_p, u)
        assert np.all((lo[tok] <= u) & (u < hi[tok])), "sample outside its interval"


# ------------------------------------------------------------ KV append
def pin_kv_append_hand(orc=None):
    """A1: two candidates, one kv head, D = 2, caches of 8 rows holding -1.
    Candidate 0 (region from row 0, 2 tokens there) appends new rows 1 and 2;
    candidate 1 (region from row 4, 1 token) appends new row 0: rows 2, 3 and
    5 change, nothing else.  In the head-major cache the same rows change."""
    import oracle as _o
    new = np.array([[[10, 11]], [[20, 21]], [[30, 31]]], np.int64)      # [3, 1, 2]
    cache = -np.ones((8, 1, 2), np.int64)
    k, v = _o.kv_append(cache, cache, new, new + 100, [0, 4], [2, 1], [1, 0], [2, 1])
    want = cache.copy()
    want[2], want[3], want[5] = new[1], new[2], new[0]
    assert np.array_equal(k, want) and np.array_equal(v, np.where(want == -1, -1, want + 100))
    kh, _ = _o.kv_append(cache.transpose(1, 0, 2).copy(), cache.transpose(1, 0, 2).copy(), new, new,
                         [0, 4], [2, 1], [1, 0], [2, 1], kv_layout="head")
    assert np.array_equal(kh, want.transpose(1, 0, 2))


def pin_sampling_golden(orc):
    """Hand-worked cases (tests/golden/sampling_hand.json)."""
    with open(os.path.join(GOLDEN, "sampling_hand.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        n = len(case["uniform"])
        h = bf16_bits_of(np.tile(np.array(case["hidden"], np.float64), (n, 1)))
        tok, _, _ = orc.sample_top_p(h, bf16_bits_of(np.array(case["w_lm"], np.float64)),
                                     np.full(n, case["inv_temperature"], np.float32), case["top_p"],
                                     np.array(case["uniform"], np.float64))
        assert tok.tolist() == case["token"], (case["name"], tok.tolist(), case["token"])


ATTENTION_PINS = [pin_attention_vs_torch, pin_prefix_sharing, pin_attention_closed_forms,
                  pin_permutation, pin_one_hot_probe, pin_length_probe, pin_attention_golden]
LOGPROB_PINS = [pin_logprob_vs_torch, pin_logprob_sum_to_one, pin_logprob_closed_forms,
                pin_logprob_shift, pin_logprob_chunks, pin_logprob_id_probe, pin_logprob_golden]
GRPO_PINS = [pin_advantage_closed_form, pin_advantage_invariants, pin_surrogate_finite_differences,
             pin_surrogate_closed_forms, pin_surrogate_unowned_rows]
BACKWARD_PINS = [pin_backward_vs_torch, pin_backward_finite_differences, pin_backward_closed_forms]
SAMPLING_PINS = [pin_sampling_full_distribution, pin_sampling_greedy_limit, pin_sampling_frequencies,
                 pin_sampling_ties, pin_sampling_temperature_scale, pin_sampling_logprob, pin_sampling_intervals,
                 pin_sampling_golden]
APPEND_PINS = [pin_kv_append_hand]
ALL_PINS = ATTENTION_PINS + LOGPROB_PINS + GRPO_PINS + BACKWARD_PINS + SAMPLING_PINS + APPEND_PINS


# --------------------------------------------------------------- extend pins
def extend_case(P=2, G=2, Hq=4, Hkv=2, D=8, lp=None, ls=None, nl=None, seed=0, qmul=1.0):
    """Small random extend input: decode_case's caches plus the new-token counts
    and a packed query array whose candidates come in reverse order, with gaps."""
    c = decode_case(P=P, G=G, Hq=Hq, Hkv=Hkv, D=D, lp=lp, ls=ls, seed=seed, qmul=qmul)
    rng = np.random.Generator(np.random.PCG64(seed + 1000))
    S = P * G
    ls_ = c["suffix_len"]
    nl = np.asarray([int(rng.integers(0, l + 1)) for l in ls_] if nl is None else nl, np.int32)
    qs = np.zeros(S, np.int64)
    pos = 1
    for s in reversed(range(S)):
        qs[s] = pos
        pos += int(nl[s]) + 1
    q = bf16_bits_of(rng.standard_normal((pos + 1, Hq, D)) * qmul)
    c.update(q=q, new_len=nl, q_start=qs)
    return c


def torch_extend(c):
    """Reference via torch's fp64 SDPA with a lower-triangular boolean mask over
    each candidate's concatenated sequence, keeping the rows of its last n tokens."""
    q = f64(c["q"]); kp = f64(c["k_prefix"]); vp = f64(c["v_prefix"])
    ks = f64(c["k_suffix"]); vs = f64(c["v_suffix"])
    Q, Hq, D = q.shape
    Hkv = kp.shape[1]
    G = c["group_size"]
    sigma = float(np.float32(c["scale"]))
    out = torch.zeros(Q, Hq, D, dtype=torch.float64)
    lse = torch.zeros(Q, Hq, dtype=torch.float64)
    for s in range(len(c["suffix_len"])):
        n = int(c["new_len"][s])
        if n == 0:
            continue
        p = s // G
        a, lp = int(c["prefix_start"][p]), int(c["prefix_len"][p])
        b, ls = int(c["suffix_start"][s]), int(c["suffix_len"][s])
        K = torch.cat([kp[a:a + lp], ks[b:b + ls]])          # [T, Hkv, D]
        V = torch.cat([vp[a:a + lp], vs[b:b + ls]])
        T = K.shape[0]
        mask = torch.ones(T, T, dtype=torch.bool).tril()[T - n:]   # [n, T]
        qs = int(c["q_start"][s])
        Qs = q[qs:qs + n].permute(1, 0, 2)[None]              # [1, Hq, n, D]
        o = F.scaled_dot_product_attention(Qs, K.permute(1, 0, 2)[None], V.permute(1, 0, 2)[None],
                                           attn_mask=mask, scale=sigma, enable_gqa=True)
        out[qs:qs + n] = o[0].permute(1, 0, 2)
        Krep = K.repeat_interleave(Hq // Hkv, dim=1).permute(1, 0, 2)   # [Hq, T, D]
        scores = sigma * (Qs[0] @ Krep.transpose(1, 2))                  # [Hq, n, T]
        scores = scores.masked_fill(~mask, -math.inf)
        lse[qs:qs + n] = torch.logsumexp(scores, dim=2).T
    return out.numpy(), lse.numpy()


def _extend_args(c):
    return {k: c[k] for k in ("q", "k_prefix", "v_prefix", "k_suffix", "v_suffix", "prefix_start",
                              "prefix_len", "suffix_start", "suffix_len", "new_len", "q_start",
                              "group_size", "scale")}


def pin_extend_vs_torch(orc):
    """E1: brute force by torch's masked SDPA over the concatenated sequence."""
    cases = [
        dict(P=2, G=3, Hq=4, Hkv=2, D=8, seed=21),
        dict(P=1, G=4, Hq=6, Hkv=3, D=16, lp=[9], ls=[7, 3, 5, 1], nl=[7, 1, 2, 0], seed=22),  # n = Ls, n = 0
        dict(P=2, G=2, Hq=2, Hkv=2, D=8, lp=[0, 4], ls=[5, 3, 6, 2], nl=[5, 2, 1, 2], seed=23),  # no prefix
        dict(P=2, G=2, Hq=8, Hkv=1, D=8, lp=[3, 6], ls=[4, 4, 5, 2], nl=[4, 3, 5, 1], seed=24, qmul=4.0),
    ]
    for cs in cases:
        c = extend_case(**cs)
        o, l = orc.extend_attn(**_extend_args(c))
        ro, rl = torch_extend(c)
        close(o, ro, 1e-12, f"extend out {cs}")
        close(l, rl, 1e-12, f"extend lse {cs}")


def pin_extend_decode_steps(orc):
    """E2: new token i equals a decode step whose suffix ends at that token (a
    decode loop that appends one token per step), through the pinned decode
    definition; a single new token is exactly one decode step."""
    c = extend_case(P=2, G=2, Hq=4, Hkv=2, D=8, lp=[5, 2], ls=[6, 4, 3, 5], nl=[6, 1, 3, 2], seed=25)
    o, l = orc.extend_attn(**_extend_args(c))
    S = 4
    Hq, D = c["q"].shape[1:]
    for i in range(int(c["new_len"].max())):
        qd = np.zeros((S, Hq, D), np.uint16)
        sl = c["suffix_len"].copy()
        live = [s for s in range(S) if i < c["new_len"][s]]
        for s in live:
            qd[s] = c["q"][c["q_start"][s] + i]
            sl[s] = c["suffix_len"][s] - c["new_len"][s] + i + 1
        od, ld = orc.decode_attn(qd, c["k_prefix"], c["v_prefix"], c["k_suffix"], c["v_suffix"],
                                 c["prefix_start"], c["prefix_len"], c["suffix_start"], sl,
                                 c["group_size"], c["scale"])
        for s in live:
            row = c["q_start"][s] + i
            close(o[row], od[s], 1e-13, f"extend step {i} out s={s}")
            close(l[row], ld[s], 1e-13, f"extend step {i} lse s={s}")


def pin_extend_future_independence(orc):
    """E3: a new token's result does not depend on the tokens after it, and
    does depend on the ones up to it (causality both ways)."""
    c = extend_case(P=1, G=2, Hq=2, Hkv=1, D=8, lp=[3], ls=[6, 5], nl=[5, 4], seed=26)
    o, l = orc.extend_attn(**_extend_args(c))
    for s, cut in ((0, 2), (1, 1)):            # perturb suffix positions after new token `cut`
        ks, vs = c["k_suffix"].copy(), c["v_suffix"].copy()
        b, ls, n = int(c["suffix_start"][s]), int(c["suffix_len"][s]), int(c["new_len"][s])
        first = b + ls - n + cut + 1
        rng = np.random.Generator(np.random.PCG64(s))
        ks[first:b + ls] = bf16_bits_of(rng.standard_normal(ks[first:b + ls].shape) * 3)
        vs[first:b + ls] = bf16_bits_of(rng.standard_normal(vs[first:b + ls].shape) * 3)
        o2, l2 = orc.extend_attn(**dict(_extend_args(c), k_suffix=ks, v_suffix=vs))
        q0 = int(c["q_start"][s])
        assert np.array_equal(o2[q0:q0 + cut + 1], o[q0:q0 + cut + 1]), "a later token leaked into an earlier one"
        assert np.array_equal(l2[q0:q0 + cut + 1], l[q0:q0 + cut + 1])
        assert not np.allclose(o2[q0 + cut + 1:q0 + n], o[q0 + cut + 1:q0 + n]), "later tokens must see the change"


def pin_extend_prefix_sharing(orc):
    """E4: a shared prefix equals concatenating it into every candidate's suffix."""
    c = extend_case(P=2, G=3, Hq=4, Hkv=2, D=8, lp=[5, 3], ls=[2, 1, 4, 1, 3, 2], nl=[2, 0, 3, 1, 1, 2], seed=27)
    o, l = orc.extend_attn(**_extend_args(c))
    krows, vrows, starts, lens = [], [], [], []
    pos = 0
    for s in range(6):
        p = s // 3
        a, n = c["prefix_start"][p], c["prefix_len"][p]
        b, m = c["suffix_start"][s], c["suffix_len"][s]
        krows.append(np.concatenate([c["k_prefix"][a:a + n], c["k_suffix"][b:b + m]]))
        vrows.append(np.concatenate([c["v_prefix"][a:a + n], c["v_suffix"][b:b + m]]))
        starts.append(pos); lens.append(n + m); pos += n + m
    c2 = dict(_extend_args(c), k_prefix=c["k_prefix"][:1], v_prefix=c["v_prefix"][:1],
              prefix_start=np.zeros(2, np.int64), prefix_len=np.zeros(2, np.int32),
              k_suffix=np.concatenate(krows), v_suffix=np.concatenate(vrows),
              suffix_start=np.array(starts, np.int64), suffix_len=np.array(lens, np.int32))
    o2, l2 = orc.extend_attn(**c2)
    close(o, o2, 1e-12, "extend prefix sharing out")
    close(l, l2, 1e-12, "extend prefix sharing lse")


def pin_extend_golden(orc):
    """Hand-derived worked examples (tests/golden/extend_hand.json)."""
    with open(os.path.join(GOLDEN, "extend_hand.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        c = {k: bf16_bits_of(np.array(case[k], np.float64))
             for k in ("q", "k_prefix", "v_prefix", "k_suffix", "v_suffix")}
        c.update(prefix_start=np.array(case["prefix_start"], np.int64),
                 prefix_len=np.array(case["prefix_len"], np.int32),
                 suffix_start=np.array(case["suffix_start"], np.int64),
                 suffix_len=np.array(case["suffix_len"], np.int32),
                 new_len=np.array(case["new_len"], np.int32), q_start=np.array(case["q_start"], np.int64),
                 group_size=case["group_size"], scale=case["scale"])
        o, l = orc.extend_attn(**c)
        close(o, np.array(case["out"]), 1e-15, case["name"] + " out")
        close(l, np.array(case["lse"]), 1e-15, case["name"] + " lse")


EXTEND_PINS = [pin_extend_vs_torch, pin_extend_decode_steps, pin_extend_future_independence,
               pin_extend_prefix_sharing, pin_extend_golden]
ALL_PINS = ALL_PINS + EXTEND_PINS
