"""Seeded synthetic inputs for the rollout hot path.

This module draws random tensors and lengths and lays them out in memory. It
holds none of the method's arithmetic: it computes no scores, softmax, logits
or log-probs. Both the fp64 oracle's tests and the GPU path's tests and bench
take their inputs from here, so both sides see the same bits.

Workload shapes follow the method's setting: each input program x gets a group
of g sampled candidates that share the prompt (Sec. 2.2.1, Problem Setup),
16 candidates per turn with up to 1536 generated tokens and a masked log-prob
window for the policy update (Sec. 3, Multi-turn RL Training), and refinement
turns that grow the shared prompt (same paragraph, Structured Feedback and
Iterative Refinement). The concrete sizes are those of the five named configs
below; the paper's own datasets are not used (they stand in only as shapes).

Layout conventions (shared with the C ABI):
  q        bf16 [S, Hq, D]            S = P*G, sequence s = p*G + g
  k/v_pfx  bf16 [prefix_rows, Hkv, D] prompt p owns rows [prefix_start[p], +Lp[p])
           (or [Hkv, prefix_rows, D] with kv_layout="head")
  k/v_sfx  bf16 [suffix_rows, Hkv, D] candidate s owns rows [suffix_start[s], +Ls[s])
           (or [Hkv, suffix_rows, D] with kv_layout="head")
  hidden   bf16 [R, H]
  w_lm     bf16 [V, H]                row v produces logit v (nn.Linear layout)
  target   int32 [R]                  -1 masks a row
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class DecodeConfig:
    name: str
    num_prompts: int          # P
    group_size: int           # G
    num_q_heads: int          # Hq
    num_kv_heads: int         # Hkv
    head_dim: int             # D
    prefix_len: int           # Lp (same for every prompt)
    suffix_kind: str          # "const", "uniform" or "geometric"
    suffix_a: int             # const value / uniform low / unused
    suffix_b: int             # unused / uniform high (inclusive) / cap
    suffix_mean: float = 0.0  # geometric mean before the cap

    @property
    def num_seqs(self) -> int:
        return self.num_prompts * self.group_size

    @property
    def softmax_scale(self) -> float:
        # fp32(1/sqrt(D)): the exact float32 value both sides receive.
        return float(np.float32(1.0 / math.sqrt(self.head_dim)))


@dataclasses.dataclass(frozen=True)
class LogprobConfig:
    name: str
    rows: int      # R
    hidden: int    # H
    vocab: int     # V


# The five workloads: a tiny case the oracle finishes instantly, an 8B-class and
# a 32B-class single-layer decode step, a multi-turn long-context step and the
# policy-update log-prob pass over 64 sequences x 4096 positions.
DECODE_CONFIGS = {
    "tiny": DecodeConfig("tiny", 2, 4, 4, 1, 64, 128, "const", 32, 32),
    "8b": DecodeConfig("8b", 64, 8, 32, 8, 128, 1024, "uniform", 256, 2048),
    "32b": DecodeConfig("32b", 16, 16, 64, 8, 128, 2048, "uniform", 512, 8192),
    "longctx": DecodeConfig("longctx", 4, 8, 64, 8, 128, 24576, "geometric", 0, 4096, 1024.0),
}

LOGPROB_CONFIGS = {
    "tiny": LogprobConfig("tiny", 8, 256, 1024),
    "8b": LogprobConfig("8b", 512, 4096, 151936),
    "32b": LogprobConfig("32b", 256, 5120, 151936),
    "policy": LogprobConfig("policy", 262144, 5120, 151936),
}

# Sub-seeds per tensor: base seed + k.
_SUB = {"q": 1, "kp": 2, "vp": 3, "ks": 4, "vs": 5, "hidden": 6, "w": 7}


def suffix_lengths(cfg: DecodeConfig, seed: int = 0) -> np.ndarray:
    """Per-candidate generated-token counts, int32 [P*G]."""
    S = cfg.num_seqs
    if cfg.suffix_kind == "const":
        return np.full(S, cfg.suffix_a, dtype=np.int32)
    rng = np.random.Generator(np.random.PCG64(seed))
    if cfg.suffix_kind == "uniform":
        # integers, inclusive at both ends
        return rng.integers(cfg.suffix_a, cfg.suffix_b + 1, S).astype(np.int32)
    if cfg.suffix_kind == "geometric":
        # support {1, 2, ...} with success prob 1/mean, then capped
        draw = rng.geometric(1.0 / cfg.suffix_mean, S)
        return np.minimum(draw, cfg.suffix_b).astype(np.int32)
    raise ValueError(cfg.suffix_kind)


def _randn_bf16(shape, seed: int, device, std: float = 1.0) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(torch.bfloat16)   # round-to-nearest-even


@dataclasses.dataclass
class DecodeInputs:
    cfg: DecodeConfig
    q: torch.Tensor
    k_prefix: torch.Tensor
    v_prefix: torch.Tensor
    k_suffix: torch.Tensor
    v_suffix: torch.Tensor
    prefix_start: np.ndarray   # int64 [P]
    prefix_len: np.ndarray     # int32 [P]
    suffix_start: np.ndarray   # int64 [S]
    suffix_len: np.ndarray     # int32 [S]
    scale: float
    kv_layout: str = "token"

    def token_major(self, t: torch.Tensor) -> torch.Tensor:
        """A KV tensor of this input as [rows, Hkv, D]."""
        return t.transpose(0, 1).contiguous() if self.kv_layout == "head" else t

    @property
    def P(self): return self.cfg.num_prompts

    @property
    def G(self): return self.cfg.group_size


def packed_starts(lengths: np.ndarray) -> np.ndarray:
    """Densest packing: sequence i starts where sequence i-1 ends."""
    starts = np.zeros(len(lengths), dtype=np.int64)
    if len(lengths) > 1:
        starts[1:] = np.cumsum(lengths.astype(np.int64))[:-1]
    return starts


def make_decode_inputs(cfg: DecodeConfig, device="cpu", seed: int = 0,
                       suffix_len: Optional[np.ndarray] = None,
                       prefix_len: Optional[np.ndarray] = None,
                       kv_layout: str = "token") -> DecodeInputs:
    """kv_layout "token": KV tensors [rows, Hkv, D]; "head": [Hkv, rows, D] holding
    the same values (the token-major draw, transposed)."""
    P, G, Hq, Hkv, D = cfg.num_prompts, cfg.group_size, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    S = P * G
    lp = (np.full(P, cfg.prefix_len, dtype=np.int32) if prefix_len is None
          else np.asarray(prefix_len, dtype=np.int32))
    ls = suffix_lengths(cfg, seed) if suffix_len is None else np.asarray(suffix_len, dtype=np.int32)
    ps, ss = packed_starts(lp), packed_starts(ls)
    prow, srow = int(lp.sum()), int(ls.sum())
    q = _randn_bf16((S, Hq, D), seed + _SUB["q"], device)
    kp = _randn_bf16((prow, Hkv, D), seed + _SUB["kp"], device)
    vp = _randn_bf16((prow, Hkv, D), seed + _SUB["vp"], device)
    ks = _randn_bf16((srow, Hkv, D), seed + _SUB["ks"], device)
    vs = _randn_bf16((srow, Hkv, D), seed + _SUB["vs"], device)
    if kv_layout == "head":
        kp, vp, ks, vs = (t.transpose(0, 1).contiguous() for t in (kp, vp, ks, vs))
    elif kv_layout != "token":
        raise ValueError(kv_layout)
    return DecodeInputs(cfg, q, kp, vp, ks, vs, ps, lp, ss, ls, cfg.softmax_scale, kv_layout)


@dataclasses.dataclass
class LogprobInputs:
    cfg: LogprobConfig
    hidden: torch.Tensor    # bf16 [R, H]
    w_lm: torch.Tensor      # bf16 [V, H]
    target: torch.Tensor    # int32 [R]
    inv_temperature: float


def make_targets(rows: int, vocab: int, seed: int = 0, mask_frac: float = 0.0) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    t = rng.integers(0, vocab, rows).astype(np.int32)
    if mask_frac > 0:
        m = np.random.Generator(np.random.PCG64(seed + 100)).random(rows) < mask_frac
        t[m] = -1
    return t


def make_logprob_inputs(cfg: LogprobConfig, device="cpu", seed: int = 0,
                        inv_temperature: float = 1.0, mask_frac: float = 0.0,
                        w_std: float = 0.02) -> LogprobInputs:
    R, H, V = cfg.rows, cfg.hidden, cfg.vocab
    hidden = _randn_bf16((R, H), seed + _SUB["hidden"], device)
    w = _randn_bf16((V, H), seed + _SUB["w"], device, std=w_std)
    t = torch.from_numpy(make_targets(R, V, seed, mask_frac)).to(device)
    return LogprobInputs(cfg, hidden, w, t, float(np.float32(inv_temperature)))


def bf16_bits(x: torch.Tensor) -> np.ndarray:
    """Raw bf16 bit patterns as a host uint16 array (no rounding)."""
    return x.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def bits_to_bf16(bits: np.ndarray, device="cpu") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


# ----------------------------------------------------------------- GRPO update
@dataclasses.dataclass(frozen=True)
class GrpoConfig:
    name: str
    num_prompts: int     # P
    group_size: int      # G
    positions: int       # token positions per sequence (row r = s * positions + t)
    max_response: int    # longest generated response; the rest of a row is prompt or padding


# The policy-update pass as 4 prompts x 16 candidates = 64 sequences of 4096
# positions (the log-prob pass's 262144 rows), each candidate with up to 1536
# generated tokens; a small case of the same structure for exhaustive checks.
GRPO_CONFIGS = {
    "tiny": GrpoConfig("tiny", 3, 4, 48, 32),
    "policy": GrpoConfig("policy", 4, 16, 4096, 1536),
}


@dataclasses.dataclass
class GrpoInputs:
    cfg: GrpoConfig
    reward: torch.Tensor     # fp32 [P*G]
    logp_old: torch.Tensor   # fp32 [R]  log-probs under the sampling policy
    logp_new: torch.Tensor   # fp32 [R]  log-probs under the current policy
    seq: torch.Tensor        # int32 [R] candidate of each row, -1 = prompt or padding
    eps: float               # clip range, an exact float32 value


def make_grpo_inputs(cfg: GrpoConfig, device="cpu", seed: int = 0, eps: float = 0.2,
                     drift: float = 0.1, reward_levels: int = 5,
                     equal_group: bool = True) -> GrpoInputs:
    """Rows of P*G sequences laid end to end, `positions` rows each.  Sequence s
    holds its prompt in the first positions - max_response rows (masked), then a
    response of uniform length in [1, max_response] (rows tagged s), then
    padding (masked).  Rewards are drawn from `reward_levels` evenly spaced
    values in [0, 1], so ties occur; with equal_group, prompt 0's candidates all
    get the same reward.  Old log-probs are -Exp(1); new ones add N(0, drift^2),
    so ratios fall inside and on both sides of the clip range."""
    P, G, T, M = cfg.num_prompts, cfg.group_size, cfg.positions, cfg.max_response
    S = P * G
    rng = np.random.Generator(np.random.PCG64(seed))
    levels = np.linspace(0.0, 1.0, max(reward_levels, 1))
    reward = levels[rng.integers(0, len(levels), S)].astype(np.float32)
    if equal_group and P > 0 and G > 1:
        reward[:G] = reward[0]
    lens = rng.integers(1, M + 1, S)
    seq = np.full((S, T), -1, np.int32)
    start = T - M
    for s in range(S):
        seq[s, start:start + lens[s]] = s
    seq = seq.reshape(-1)
    R = seq.size
    old = (-rng.exponential(1.0, R)).astype(np.float32)
    new = (old + rng.normal(0.0, drift, R)).astype(np.float32)
    dev = lambda a: torch.from_numpy(a).to(device)
    return GrpoInputs(cfg, dev(reward), dev(old), dev(new), dev(seq), float(np.float32(eps)))


# ------------------------------------------------------------ sampling head
# The rollout draws each turn's candidates by nucleus sampling with p = 0.9
# at temperatures 0.2 and 0.7 (Sec. 3, Multi-turn RL Training); the rows of a
# decode step alternate between the two.
SAMPLE_TEMPERATURES = (0.2, 0.7)
SAMPLE_TOP_P = 0.9


@dataclasses.dataclass
class SampleInputs:
    cfg: LogprobConfig
    hidden: torch.Tensor            # bf16 [R, H]
    w_lm: torch.Tensor              # bf16 [V, H]
    inv_temperature: torch.Tensor   # fp32 [R], 1/T per row
    uniform: torch.Tensor           # fp32 [R], in [0, 1)
    top_p: float


def make_sample_inputs(cfg: LogprobConfig, device="cpu", seed: int = 0, top_p: float = SAMPLE_TOP_P,
                       w_std: float = 0.02) -> SampleInputs:
    """Hidden rows and lm-head weight as for the log-prob pass (same seeds);
    row r samples at temperature SAMPLE_TEMPERATURES[r % 2]; one uniform draw
    per row (PCG64, float32 in [0, 1))."""
    R, H, V = cfg.rows, cfg.hidden, cfg.vocab
    hidden = _randn_bf16((R, H), seed + _SUB["hidden"], device)
    w = _randn_bf16((V, H), seed + _SUB["w"], device, std=w_std)
    inv_t = np.array([1.0 / SAMPLE_TEMPERATURES[r % 2] for r in range(R)], dtype=np.float32)
    u = np.random.Generator(np.random.PCG64(seed + 200)).random(R, dtype=np.float32)
    return SampleInputs(cfg, hidden, w, torch.from_numpy(inv_t).to(device), torch.from_numpy(u).to(device),
                        float(np.float32(top_p)))


@dataclasses.dataclass
class ExtendInputs:
    """A refinement turn's extend: the caches of a DecodeInputs (each candidate's
    suffix already holds its new tokens' K/V at its end) plus the new tokens'
    queries, packed [sum(new_len), Hq, D] with candidate s at rows
    [q_start[s], +new_len[s])."""
    dec: DecodeInputs
    q: torch.Tensor
    new_len: np.ndarray   # int32 [S], 0 <= new_len <= suffix_len
    q_start: np.ndarray   # int64 [S]


def make_extend_inputs(cfg: DecodeConfig, device="cpu", seed: int = 0,
                       new_len: Optional[np.ndarray] = None,
                       suffix_len: Optional[np.ndarray] = None,
                       prefix_len: Optional[np.ndarray] = None,
                       kv_layout: str = "token") -> ExtendInputs:
    """Default new_len: the whole suffix is new (the turn's summary, feedback and
    previous code are read in one pass against the shared prefix)."""
    dec = make_decode_inputs(cfg, device, seed, suffix_len=suffix_len, prefix_len=prefix_len,
                             kv_layout=kv_layout)
    n = dec.suffix_len.copy() if new_len is None else np.asarray(new_len, dtype=np.int32)
    qs = packed_starts(n)
    q = _randn_bf16((int(n.sum()), cfg.num_q_heads, cfg.head_dim), seed + 8, device)
    return ExtendInputs(dec, q, n, qs)
