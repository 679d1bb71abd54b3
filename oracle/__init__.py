"""ctypes wrapper of the fp64 CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY.  The tests, ``__graft_entry__.smoke()`` and the
bench's CPU-baseline leg may call it; the GPU library and its Python binding
never import it.  It takes host numpy arrays (bf16 inputs as raw uint16 bit
patterns) and returns float64 results.

The definitions it computes are stated at the top of oracle.c: grouped-query
decode attention over a shared prompt prefix followed by each candidate's own
suffix (Sec. 2.2.1, Problem Setup) and the causal extend (prefill) of a
refinement turn's new tokens over that context (Sec. 3, Structured Feedback
and Iterative Refinement), the full-vocabulary token log-prob of
the sampled token that the GRPO ratio needs (Sec. 3, Eq. grpo-loss; masked
positions per Sec. 3, Multi-turn RL Training), the group-relative advantages
and the clipped surrogate of Eq. grpo-loss with its gradient, and the
gradient of the log-prob with respect to the hidden rows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")
# Plain IEEE double arithmetic: no -ffast-math, no FMA contraction.
CFLAGS = ["-O2", "-std=c99", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared"]


def compile_c(src_path: str, out_path: str) -> str:
    """Compile an oracle C source into a shared library with gcc."""
    tmp = out_path + ".tmp"
    subprocess.run(["gcc", *CFLAGS, src_path, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, out_path)
    return out_path


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (plain C99 + OpenMP)."""
    if force or not os.path.exists(LIB_PATH):
        compile_c(SRC_PATH, LIB_PATH)
    return LIB_PATH


def _bind(path: str):
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.oracle_decode_attn.restype = ctypes.c_int
    lib.oracle_decode_attn.argtypes = [ctypes.c_int32] * 5 + [ctypes.c_float] + [P] * 11
    lib.oracle_token_logprob.restype = ctypes.c_int
    lib.oracle_token_logprob.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                         P, P, P, ctypes.c_float, P, P]
    lib.oracle_token_logprob_f64.restype = ctypes.c_int
    lib.oracle_token_logprob_f64.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                             P, P, P, ctypes.c_float, P, P]
    lib.oracle_grpo_advantage.restype = ctypes.c_int
    lib.oracle_grpo_advantage.argtypes = [ctypes.c_int64, ctypes.c_int32, P, P]
    lib.oracle_grpo_surrogate.restype = ctypes.c_int
    lib.oracle_grpo_surrogate.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                          P, P, P, P, ctypes.c_double, P, P]
    lib.oracle_sample_top_p.restype = ctypes.c_int
    lib.oracle_sample_top_p.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, P, P, P,
                                        ctypes.c_double, P, P, P, P]
    lib.oracle_top_p_interval.restype = ctypes.c_int
    lib.oracle_top_p_interval.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, P, P, P,
                                          ctypes.c_double, P, P, P]
    lib.oracle_token_logprob_backward.restype = ctypes.c_int
    lib.oracle_token_logprob_backward.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                                  P, P, P, ctypes.c_float, P, P]
    lib.oracle_extend_attn.restype = ctypes.c_int
    lib.oracle_extend_attn.argtypes = [ctypes.c_int32] * 5 + [ctypes.c_float] + [P] * 13
    return lib


_default = None


def _load():
    global _default
    if _default is None:
        if not os.path.exists(LIB_PATH):
            build()
        _default = _bind(LIB_PATH)
    return _default


def _u16(a, shape=None):
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 inputs are passed as uint16 bit patterns")
    if shape is not None and a.shape != tuple(shape):
        raise ValueError(f"shape {a.shape} != {tuple(shape)}")
    return a


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def decode_attn(q, k_prefix, v_prefix, k_suffix, v_suffix,
                prefix_start, prefix_len, suffix_start, suffix_len,
                group_size: int, scale: float, _lib=None):
    """Oracle decode attention.

    q: uint16 [S, Hq, D]; k/v_prefix: uint16 [rows_p, Hkv, D];
    k/v_suffix: uint16 [rows_s, Hkv, D]; lengths/starts host ints.
    Returns (out float64 [S, Hq, D], lse float64 [S, Hq]).
    """
    q = _u16(q)
    S, Hq, D = q.shape
    G = int(group_size)
    if G <= 0 or S % G:
        raise ValueError("S must be a positive multiple of group_size")
    P = S // G
    kp, vp, ks, vs = (_u16(t) for t in (k_prefix, v_prefix, k_suffix, v_suffix))
    Hkv = kp.shape[1]
    if Hq % Hkv or any(t.shape[1:] != (Hkv, D) for t in (kp, vp, ks, vs)):
        raise ValueError("bad head layout")
    ps = np.ascontiguousarray(prefix_start, dtype=np.int64)
    pl = np.ascontiguousarray(prefix_len, dtype=np.int32)
    ss = np.ascontiguousarray(suffix_start, dtype=np.int64)
    sl = np.ascontiguousarray(suffix_len, dtype=np.int32)
    if ps.shape != (P,) or pl.shape != (P,) or ss.shape != (S,) or sl.shape != (S,):
        raise ValueError("length arrays")
    if (pl < 0).any() or (sl < 0).any():
        raise ValueError("negative length")
    if P and ((ps < 0).any() or (ps + pl > kp.shape[0]).any() or kp.shape != vp.shape):
        raise ValueError("prefix range")
    if S and ((ss < 0).any() or (ss + sl > ks.shape[0]).any() or ks.shape != vs.shape):
        raise ValueError("suffix range")
    out = np.zeros((S, Hq, D), dtype=np.float64)
    lse = np.zeros((S, Hq), dtype=np.float64)
    if S == 0:
        return out, lse
    rc = (_lib or _load()).oracle_decode_attn(
        P, G, Hq, Hkv, D, float(np.float32(scale)),
        _ptr(ps), _ptr(pl), _ptr(ss), _ptr(sl),
        _ptr(q), _ptr(kp), _ptr(vp), _ptr(ks), _ptr(vs), _ptr(out), _ptr(lse))
    if rc:
        raise MemoryError("oracle_decode_attn scratch allocation failed")
    return out, lse


def extend_attn(q, k_prefix, v_prefix, k_suffix, v_suffix,
                prefix_start, prefix_len, suffix_start, suffix_len, new_len, q_start,
                group_size: int, scale: float, _lib=None):
    """Oracle extend (prefill) attention of a refinement turn.

    The last new_len[s] tokens of candidate s's suffix are new; new token i
    attends causally to the prompt's prefix and the candidate's suffix up to
    and including itself.  q: uint16 [Q, Hq, D], its query rows q_start[s] + i;
    k/v_prefix, k/v_suffix as in decode_attn (token-major).
    Returns (out float64 [Q, Hq, D], lse float64 [Q, Hq]); rows of no
    candidate stay 0.
    """
    q = _u16(q)
    Q, Hq, D = q.shape
    G = int(group_size)
    S = len(suffix_len)
    if G <= 0 or S % G:
        raise ValueError("the number of candidates must be a positive multiple of group_size")
    P = S // G
    kp, vp, ks, vs = (_u16(t) for t in (k_prefix, v_prefix, k_suffix, v_suffix))
    Hkv = kp.shape[1]
    if Hq % Hkv or any(t.shape[1:] != (Hkv, D) for t in (kp, vp, ks, vs)):
        raise ValueError("bad head layout")
    ps = np.ascontiguousarray(prefix_start, dtype=np.int64)
    pl = np.ascontiguousarray(prefix_len, dtype=np.int32)
    ss = np.ascontiguousarray(suffix_start, dtype=np.int64)
    sl = np.ascontiguousarray(suffix_len, dtype=np.int32)
    nl = np.ascontiguousarray(new_len, dtype=np.int32)
    qs = np.ascontiguousarray(q_start, dtype=np.int64)
    if ps.shape != (P,) or pl.shape != (P,) or any(a.shape != (S,) for a in (ss, sl, nl, qs)):
        raise ValueError("length arrays")
    if (pl < 0).any() or (sl < 0).any() or (nl < 0).any() or (nl > sl).any():
        raise ValueError("lengths: need 0 <= new_len <= suffix_len")
    if P and ((ps < 0).any() or (ps + pl > kp.shape[0]).any() or kp.shape != vp.shape):
        raise ValueError("prefix range")
    if S and ((ss < 0).any() or (ss + sl > ks.shape[0]).any() or ks.shape != vs.shape):
        raise ValueError("suffix range")
    if S and ((qs < 0).any() or (qs + nl > Q).any()):
        raise ValueError("query range")
    out = np.zeros((Q, Hq, D), dtype=np.float64)
    lse = np.zeros((Q, Hq), dtype=np.float64)
    if S == 0:
        return out, lse
    rc = (_lib or _load()).oracle_extend_attn(
        P, G, Hq, Hkv, D, float(np.float32(scale)),
        _ptr(ps), _ptr(pl), _ptr(ss), _ptr(sl), _ptr(nl), _ptr(qs),
        _ptr(q), _ptr(kp), _ptr(vp), _ptr(ks), _ptr(vs), _ptr(out), _ptr(lse))
    if rc == 1:
        raise MemoryError("oracle_extend_attn scratch allocation failed")
    if rc:
        raise ValueError("oracle_extend_attn: new_len exceeds suffix_len")
    return out, lse


def token_logprob(hidden, w_lm, target, inv_temperature: float = 1.0, _lib=None):
    """Oracle token log-prob.

    hidden: uint16 [R, H]; w_lm: uint16 [V, H]; target: int32 [R].
    Returns (logprob float64 [R], lse float64 [R]).
    """
    hidden = _u16(hidden)
    w = _u16(w_lm)
    R, H = hidden.shape
    V, H2 = w.shape
    if H2 != H or V <= 0 or H <= 0:
        raise ValueError("shape")
    t = np.ascontiguousarray(target, dtype=np.int32)
    if t.shape != (R,):
        raise ValueError("target shape")
    logprob = np.zeros(R, dtype=np.float64)
    lse = np.zeros(R, dtype=np.float64)
    if R == 0:
        return logprob, lse
    rc = (_lib or _load()).oracle_token_logprob(
        R, H, V, _ptr(hidden), _ptr(w), _ptr(t),
        float(np.float32(inv_temperature)), _ptr(logprob), _ptr(lse))
    if rc:
        raise MemoryError("oracle_token_logprob scratch allocation failed")
    return logprob, lse


def token_logprob_f64(hidden, w_lm, target, inv_temperature: float = 1.0, _lib=None):
    """Oracle token log-prob with float64 hidden rows (for finite differences).

    hidden: float64 [R, H]; w_lm: uint16 [V, H]; target: int32 [R].
    """
    hidden = np.ascontiguousarray(hidden, dtype=np.float64)
    w = _u16(w_lm)
    R, H = hidden.shape
    V, H2 = w.shape
    if H2 != H or V <= 0 or H <= 0:
        raise ValueError("shape")
    t = np.ascontiguousarray(target, dtype=np.int32)
    if t.shape != (R,):
        raise ValueError("target shape")
    logprob = np.zeros(R, dtype=np.float64)
    lse = np.zeros(R, dtype=np.float64)
    if R == 0:
        return logprob, lse
    rc = (_lib or _load()).oracle_token_logprob_f64(
        R, H, V, _ptr(hidden), _ptr(w), _ptr(t),
        float(np.float32(inv_temperature)), _ptr(logprob), _ptr(lse))
    if rc:
        raise MemoryError("oracle_token_logprob_f64 scratch allocation failed")
    return logprob, lse


def grpo_advantage(reward, group_size: int, _lib=None):
    """Group-relative advantages: reward [P*G] -> float64 [P*G]."""
    r = np.ascontiguousarray(reward, dtype=np.float64).reshape(-1)
    G = int(group_size)
    if G <= 0 or r.size % G:
        raise ValueError("reward length must be a multiple of group_size")
    adv = np.zeros_like(r)
    if r.size:
        (_lib or _load()).oracle_grpo_advantage(r.size // G, G, _ptr(r), _ptr(adv))
    return adv


def grpo_surrogate(logp_new, logp_old, seq, adv, group_size: int, eps: float = 0.2, _lib=None):
    """Clipped GRPO surrogate loss and its gradient with respect to logp_new.

    logp_new, logp_old: [R] (float64 values); seq: int32 [R], the candidate of
    each token row or -1; adv: [P*G].  Returns (loss float, grad float64 [R]).
    """
    ln = np.ascontiguousarray(logp_new, dtype=np.float64)
    lo = np.ascontiguousarray(logp_old, dtype=np.float64)
    sq = np.ascontiguousarray(seq, dtype=np.int32)
    a = np.ascontiguousarray(adv, dtype=np.float64)
    G = int(group_size)
    R = ln.shape[0]
    if lo.shape != (R,) or sq.shape != (R,) or G <= 0 or a.size % G:
        raise ValueError("shapes")
    loss = np.zeros(1, dtype=np.float64)
    grad = np.zeros(R, dtype=np.float64)
    rc = (_lib or _load()).oracle_grpo_surrogate(R, a.size // G, G, _ptr(ln), _ptr(lo), _ptr(sq),
                                                 _ptr(a), float(eps), _ptr(loss), _ptr(grad))
    if rc:
        raise MemoryError("oracle_grpo_surrogate scratch allocation failed")
    return float(loss[0]), grad


def token_logprob_backward(hidden, w_lm, target, grad_logprob, inv_temperature: float = 1.0, _lib=None):
    """d(sum_r g_r logprob_r)/d hidden: float64 [R, H]."""
    hidden = _u16(hidden)
    w = _u16(w_lm)
    R, H = hidden.shape
    V, H2 = w.shape
    if H2 != H or V <= 0 or H <= 0:
        raise ValueError("shape")
    t = np.ascontiguousarray(target, dtype=np.int32)
    g = np.ascontiguousarray(grad_logprob, dtype=np.float64)
    if t.shape != (R,) or g.shape != (R,):
        raise ValueError("target / grad shape")
    dh = np.zeros((R, H), dtype=np.float64)
    if R == 0:
        return dh
    rc = (_lib or _load()).oracle_token_logprob_backward(
        R, H, V, _ptr(hidden), _ptr(w), _ptr(t), float(np.float32(inv_temperature)), _ptr(g), _ptr(dh))
    if rc:
        raise MemoryError("oracle_token_logprob_backward scratch allocation failed")
    return dh


def sample_top_p(hidden, w_lm, inv_temperature, top_p: float, uniform, _lib=None):
    """Nucleus sampling of one token per row.

    hidden [R, H] and w_lm [V, H] bf16 bits; inv_temperature [R] (float32
    values, one temperature per row); top_p in (0, 1]; uniform [R] in [0, 1).
    Returns (token int32 [R], logprob float64 [R], margin float64 [R, 3]); the
    margin columns are the inverse-CDF margin, the nucleus margin and the mass
    a nucleus change could move (see oracle.c).
    """
    hidden = _u16(hidden)
    w = _u16(w_lm)
    R, H = hidden.shape
    V, H2 = w.shape
    if H2 != H or V <= 0 or H <= 0:
        raise ValueError("shape")
    it = np.ascontiguousarray(inv_temperature, dtype=np.float32)
    u = np.ascontiguousarray(uniform, dtype=np.float64)
    if it.shape != (R,) or u.shape != (R,):
        raise ValueError("inv_temperature / uniform shape")
    token = np.zeros(R, dtype=np.int32)
    lp = np.zeros(R, dtype=np.float64)
    margin = np.zeros((R, 3), dtype=np.float64)
    if R == 0:
        return token, lp, margin
    rc = (_lib or _load()).oracle_sample_top_p(R, H, V, _ptr(hidden), _ptr(w), _ptr(it), float(top_p),
                                               _ptr(u), _ptr(token), _ptr(lp), _ptr(margin))
    if rc:
        raise MemoryError("oracle_sample_top_p scratch allocation failed")
    return token, lp, margin


def top_p_interval(hidden, w_lm, inv_temperature, top_p: float, token, _lib=None):
    """For a given token per row, the range [lo, hi) of u that nucleus sampling
    maps to it; (-1, -1) when the token is outside the nucleus."""
    hidden = _u16(hidden)
    w = _u16(w_lm)
    R, H = hidden.shape
    V, H2 = w.shape
    if H2 != H or V <= 0 or H <= 0:
        raise ValueError("shape")
    it = np.ascontiguousarray(inv_temperature, dtype=np.float32)
    t = np.ascontiguousarray(token, dtype=np.int32)
    if it.shape != (R,) or t.shape != (R,):
        raise ValueError("inv_temperature / token shape")
    lo = np.zeros(R, dtype=np.float64)
    hi = np.zeros(R, dtype=np.float64)
    if R == 0:
        return lo, hi
    rc = (_lib or _load()).oracle_top_p_interval(R, H, V, _ptr(hidden), _ptr(w), _ptr(it), float(top_p),
                                                 _ptr(t), _ptr(lo), _ptr(hi))
    if rc:
        raise MemoryError("oracle_top_p_interval scratch allocation failed")
    return lo, hi


def kv_append(k_suffix, v_suffix, k_new, v_new, suffix_start, suffix_len, new_start, new_len,
              kv_layout: str = "token"):
    """The suffix caches after appending: rows new_start[s] + i of k_new / v_new
    ([new_rows, Hkv, D], token-major) become suffix rows suffix_start[s] +
    suffix_len[s] + i, i < new_len[s], at every kv head; every other row is
    unchanged.  Caches are [rows, Hkv, D] (token) or [Hkv, rows, D] (head);
    any dtype (the copy moves bits).  Returns new arrays."""
    ks, vs = np.array(k_suffix, copy=True), np.array(v_suffix, copy=True)
    kn, vn = np.asarray(k_new), np.asarray(v_new)
    for s in range(len(suffix_start)):
        for i in range(int(new_len[s])):
            src = int(new_start[s]) + i
            dst = int(suffix_start[s]) + int(suffix_len[s]) + i
            if kv_layout == "head":
                ks[:, dst, :] = kn[src]
                vs[:, dst, :] = vn[src]
            else:
                ks[dst] = kn[src]
                vs[dst] = vn[src]
    return ks, vs


def num_threads() -> int:
    """Threads OpenMP will use (OMP_NUM_THREADS, else the CPUs this process may run on)."""
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.strip().isdigit() and int(env) > 0:
        return int(env)
    return len(os.sched_getaffinity(0))


class Oracle:
    """The oracle's functions bound to one compiled library.

    The default instance uses liboracle.so; the mutation tests bind a copy
    compiled from a deliberately altered source to show the pins catch it.
    """

    def __init__(self, lib_path: str = LIB_PATH):
        self.lib_path = lib_path
        self._lib = _bind(lib_path) if lib_path != LIB_PATH else _load()

    def decode_attn(self, *args, **kw):
        return decode_attn(*args, **kw, _lib=self._lib)

    def extend_attn(self, *args, **kw):
        return extend_attn(*args, **kw, _lib=self._lib)

    def token_logprob(self, *args, **kw):
        return token_logprob(*args, **kw, _lib=self._lib)

    def token_logprob_f64(self, *args, **kw):
        return token_logprob_f64(*args, **kw, _lib=self._lib)

    def grpo_advantage(self, *args, **kw):
        return grpo_advantage(*args, **kw, _lib=self._lib)

    def grpo_surrogate(self, *args, **kw):
        return grpo_surrogate(*args, **kw, _lib=self._lib)

    def token_logprob_backward(self, *args, **kw):
        return token_logprob_backward(*args, **kw, _lib=self._lib)

    def sample_top_p(self, *args, **kw):
        return sample_top_p(*args, **kw, _lib=self._lib)

    def top_p_interval(self, *args, **kw):
        return top_p_interval(*args, **kw, _lib=self._lib)
