"""Python binding of librlkern.so, the MI355X rollout hot path.

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C ABI (include/rl_kernels.h).  PyTorch provides device
memory and the current stream.  There is no fallback: if the library is not
built, importing this package raises.

    decode_attn(...)    prefix-shared grouped-query decode attention for a
                        batch of prompts with G candidates each (Sec. 2.2.1,
                        Problem Setup)
    extend_attn(...)    causal prefill of each candidate's new tokens over
                        the shared prefix and its own suffix (Sec. 3,
                        Structured Feedback and Iterative Refinement)
    token_logprob(...)  log-prob of each sampled token over the full
                        vocabulary, through the lm-head, without storing the
                        logits (the GRPO ratio's factor, Sec. 3, Eq. grpo-loss)
"""
from __future__ import annotations

import ctypes
import functools
import math
import os
from typing import Optional

import numpy as np
import torch  # imported first so its HIP runtime is the one the library binds to

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librlkern.so")

RL_OK = 0
STATUS_NAMES = {0: "RL_OK", 1: "RL_ERR_NULL_POINTER", 2: "RL_ERR_INVALID_SHAPE",
                3: "RL_ERR_UNSUPPORTED", 4: "RL_ERR_MISALIGNED", 5: "RL_ERR_WORKSPACE",
                6: "RL_ERR_HIP"}


class RLError(RuntimeError):
    """A non-OK status from librlkern; ``status`` is the rl_status value."""

    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {detail}")


class DecodeShape(ctypes.Structure):
    _fields_ = [("num_prompts", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("split_tokens", ctypes.c_int32), ("kv_layout", ctypes.c_int32)]


KV_LAYOUTS = {"token": 0, "head": 1}   # [rows, Hkv, D] / [Hkv, rows, D]


class DecodeLens(ctypes.Structure):
    _fields_ = [("prefix_start", ctypes.c_void_p), ("prefix_len", ctypes.c_void_p),
                ("suffix_start", ctypes.c_void_p), ("suffix_len", ctypes.c_void_p),
                ("prefix_rows", ctypes.c_int64), ("suffix_rows", ctypes.c_int64)]


class ExtendLens(ctypes.Structure):
    _fields_ = [("prefix_start", ctypes.c_void_p), ("prefix_len", ctypes.c_void_p),
                ("suffix_start", ctypes.c_void_p), ("suffix_len", ctypes.c_void_p),
                ("new_len", ctypes.c_void_p), ("q_start", ctypes.c_void_p),
                ("prefix_rows", ctypes.c_int64), ("suffix_rows", ctypes.c_int64), ("q_rows", ctypes.c_int64)]


class KvAppendLens(ctypes.Structure):
    _fields_ = [("suffix_start", ctypes.c_void_p), ("suffix_len", ctypes.c_void_p),
                ("suffix_capacity", ctypes.c_void_p), ("new_start", ctypes.c_void_p),
                ("new_len", ctypes.c_void_p), ("suffix_rows", ctypes.c_int64), ("new_rows", ctypes.c_int64)]


class DecodePtrs(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k_prefix", ctypes.c_void_p),
                ("v_prefix", ctypes.c_void_p), ("k_suffix", ctypes.c_void_p),
                ("v_suffix", ctypes.c_void_p), ("out", ctypes.c_void_p), ("lse", ctypes.c_void_p)]


class PlanItem(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("unit", ctypes.c_int32), ("kv_head", ctypes.c_int32),
                ("chunk", ctypes.c_int32), ("tok_begin", ctypes.c_int64),
                ("tok_count", ctypes.c_int32), ("row_begin", ctypes.c_int32),
                ("row_count", ctypes.c_int32), ("split_variant", ctypes.c_int32)]


class BoundsReport(ctypes.Structure):
    _fields_ = [("accesses", ctypes.c_uint64), ("violations", ctypes.c_uint64), ("launches", ctypes.c_int32),
                ("regions", ctypes.c_int32), ("first_violation", ctypes.c_char * 256)]


EXPORTS = ["rl_decode_attn_workspace_size", "rl_decode_attn", "rl_token_logprob_workspace_size",
           "rl_token_logprob", "rl_status_string", "rl_last_error", "rl_abi_version",
           "rl_decode_plan_debug", "rl_grpo_advantage", "rl_grpo_surrogate_workspace_size",
           "rl_grpo_surrogate", "rl_token_logprob_backward_workspace_size", "rl_token_logprob_backward",
           "rl_sample_top_p_workspace_size", "rl_sample_top_p", "rl_kv_append_workspace_size",
           "rl_kv_append", "rl_extend_attn_workspace_size", "rl_extend_attn", "rl_debug_logprob_bounds",
           "rl_token_logprob_noalloc", "rl_debug_logprob_timeline", "rl_debug_decode_timeline",
           "rl_debug_extend_bounds", "rl_debug_decode_bounds"]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() or "
                          "python paper_2607_20908_amd/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.rl_abi_version.restype = ctypes.c_int
    lib.rl_status_string.restype = ctypes.c_char_p
    lib.rl_status_string.argtypes = [ctypes.c_int]
    lib.rl_last_error.restype = ctypes.c_char_p
    lib.rl_decode_attn_workspace_size.restype = ctypes.c_int
    lib.rl_decode_attn_workspace_size.argtypes = [P, P, ctypes.POINTER(SZ)]
    lib.rl_decode_attn.restype = ctypes.c_int
    lib.rl_decode_attn.argtypes = [P, P, P, P, SZ, P]
    lib.rl_token_logprob_workspace_size.restype = ctypes.c_int
    lib.rl_token_logprob_workspace_size.argtypes = [I64, I32, I32, ctypes.POINTER(SZ)]
    lib.rl_token_logprob.restype = ctypes.c_int
    lib.rl_token_logprob.argtypes = [I64, I32, I32, P, P, P, ctypes.c_float, P, P, P, SZ, P]
    lib.rl_decode_plan_debug.restype = ctypes.c_int
    lib.rl_decode_plan_debug.argtypes = [P, P, P, I64, ctypes.POINTER(I64)]
    lib.rl_grpo_advantage.restype = ctypes.c_int
    lib.rl_grpo_advantage.argtypes = [I64, I32, P, P, P]
    lib.rl_grpo_surrogate_workspace_size.restype = ctypes.c_int
    lib.rl_grpo_surrogate_workspace_size.argtypes = [I64, I64, I32, ctypes.POINTER(SZ)]
    lib.rl_grpo_surrogate.restype = ctypes.c_int
    lib.rl_grpo_surrogate.argtypes = [I64, I64, I32, P, P, P, P, ctypes.c_float, P, P, P, SZ, P]
    lib.rl_token_logprob_backward_workspace_size.restype = ctypes.c_int
    lib.rl_token_logprob_backward_workspace_size.argtypes = [I64, I32, I32, ctypes.POINTER(SZ)]
    lib.rl_token_logprob_backward.restype = ctypes.c_int
    lib.rl_token_logprob_backward.argtypes = [I64, I32, I32, P, P, P, ctypes.c_float, P, P, P, P, SZ, P]
    lib.rl_sample_top_p_workspace_size.restype = ctypes.c_int
    lib.rl_sample_top_p_workspace_size.argtypes = [I64, I32, I32, ctypes.POINTER(SZ)]
    lib.rl_sample_top_p.restype = ctypes.c_int
    lib.rl_sample_top_p.argtypes = [I64, I32, I32, P, P, P, ctypes.c_float, P, P, P, P, SZ, P]
    lib.rl_kv_append_workspace_size.restype = ctypes.c_int
    lib.rl_kv_append_workspace_size.argtypes = [P, P, ctypes.POINTER(SZ)]
    lib.rl_kv_append.restype = ctypes.c_int
    lib.rl_kv_append.argtypes = [P, P, P, P, P, P, P, SZ, P]
    lib.rl_extend_attn_workspace_size.restype = ctypes.c_int
    lib.rl_extend_attn_workspace_size.argtypes = [P, P, ctypes.POINTER(SZ)]
    lib.rl_extend_attn.restype = ctypes.c_int
    lib.rl_extend_attn.argtypes = [P, P, P, P, SZ, P]
    lib.rl_debug_logprob_bounds.restype = ctypes.c_int
    lib.rl_debug_logprob_bounds.argtypes = [I32, I64, I32, I32, I32, I32, ctypes.POINTER(BoundsReport)]
    lib.rl_debug_extend_bounds.restype = ctypes.c_int
    lib.rl_debug_extend_bounds.argtypes = [P, P, I32, I32, ctypes.POINTER(BoundsReport)]
    lib.rl_debug_decode_bounds.restype = ctypes.c_int
    lib.rl_debug_decode_bounds.argtypes = [P, P, I32, ctypes.POINTER(BoundsReport)]
    lib.rl_token_logprob_noalloc.restype = ctypes.c_int
    lib.rl_token_logprob_noalloc.argtypes = [I64, I32, I32, P, P, P, ctypes.c_float, P, P, P]
    lib.rl_debug_decode_timeline.restype = ctypes.c_int
    lib.rl_debug_decode_timeline.argtypes = [P, P, P, P, ctypes.c_size_t, P, I64, ctypes.POINTER(ctypes.c_int64), P]
    lib.rl_debug_logprob_timeline.restype = ctypes.c_int
    lib.rl_debug_logprob_timeline.argtypes = [I64, I32, I32, P, P, P, ctypes.c_float, P, P, P, ctypes.c_size_t, P, I64,
                                              ctypes.POINTER(ctypes.c_int64), P]
    if lib.rl_abi_version() != 13:
        raise ImportError("librlkern ABI version mismatch")
    return lib


_lib = _load()


def lib() -> ctypes.CDLL:
    return _lib


def hip_runtimes_mapped() -> list[str]:
    """Paths of every libamdhip64 mapped into this process (should be exactly one)."""
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            parts = line.split()
            if len(parts) >= 6 and "libamdhip64" in parts[5]:
                paths.add(os.path.realpath(parts[5]))
    return sorted(paths)


def _check(st: int, where: str):
    if st != RL_OK:
        raise RLError(st, where, _lib.rl_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        if torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
        return None
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _on_call_stream(fn):
    """Runs a wrapper whose caller passed stream= with that stream current, so
    the workspace and outputs it allocates belong to that stream in torch's
    caching allocator: once dropped, they are reused only by later work on the
    same stream, never while the library's kernels there may still use them."""
    @functools.wraps(fn)
    def call(*args, stream=None, **kw):
        if stream is None:
            return fn(*args, stream=None, **kw)
        s = stream if isinstance(stream, torch.cuda.Stream) else torch.cuda.ExternalStream(_stream_handle(stream))
        with torch.cuda.stream(s):
            return fn(*args, stream=stream, **kw)
    return call


def _on_device(t: torch.Tensor, name: str) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor (the kernels read it on the GPU)")
    return t


def _bf16_dev(t: torch.Tensor, name: str) -> torch.Tensor:
    _on_device(t, name)
    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


class _DecodeArgs:
    """Host-side ctypes structures for one decode call (kept alive by the caller)."""

    def __init__(self, P, G, Hq, Hkv, D, scale, split_tokens, prefix_start, prefix_len,
                 suffix_start, suffix_len, prefix_rows, suffix_rows, kv_layout="token"):
        self.ps = np.ascontiguousarray(prefix_start, dtype=np.int64)
        self.pl = np.ascontiguousarray(prefix_len, dtype=np.int32)
        self.ss = np.ascontiguousarray(suffix_start, dtype=np.int64)
        self.sl = np.ascontiguousarray(suffix_len, dtype=np.int32)
        if self.ps.shape != (P,) or self.pl.shape != (P,) or self.ss.shape != (P * G,) \
                or self.sl.shape != (P * G,):
            raise ValueError("length arrays must be [P] (prefix) and [P*G] (suffix)")
        if kv_layout not in KV_LAYOUTS:
            raise ValueError(f"kv_layout must be one of {sorted(KV_LAYOUTS)}")
        self.shape = DecodeShape(P, G, Hq, Hkv, D, float(np.float32(scale)), int(split_tokens),
                                 KV_LAYOUTS[kv_layout])
        self.lens = DecodeLens(self.ps.ctypes.data, self.pl.ctypes.data, self.ss.ctypes.data,
                               self.sl.ctypes.data, int(prefix_rows), int(suffix_rows))


def decode_attn_workspace_size(P, G, Hq, Hkv, D, prefix_start, prefix_len, suffix_start,
                               suffix_len, prefix_rows, suffix_rows, scale=None,
                               split_tokens: int = 0, kv_layout: str = "token") -> int:
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    a = _DecodeArgs(P, G, Hq, Hkv, D, scale, split_tokens, prefix_start, prefix_len,
                    suffix_start, suffix_len, prefix_rows, suffix_rows, kv_layout)
    n = ctypes.c_size_t(0)
    _check(_lib.rl_decode_attn_workspace_size(ctypes.byref(a.shape), ctypes.byref(a.lens),
                                              ctypes.byref(n)), "rl_decode_attn_workspace_size")
    return n.value


def decode_bounds(P, G, Hq, Hkv, D, prefix_start, prefix_len, suffix_start, suffix_len, prefix_rows, suffix_rows,
                  split_tokens: int = 0, kv_layout: str = "token", shrink_region: int = -1) -> "BoundsReport":
    """Host replay of the global accesses of rl_decode_attn for these lengths
    (no device access)."""
    a = _DecodeArgs(P, G, Hq, Hkv, D, 1.0 / math.sqrt(D), split_tokens, prefix_start, prefix_len,
                    suffix_start, suffix_len, prefix_rows, suffix_rows, kv_layout)
    rep = BoundsReport()
    _check(_lib.rl_debug_decode_bounds(ctypes.byref(a.shape), ctypes.byref(a.lens), shrink_region,
                                       ctypes.byref(rep)), "rl_debug_decode_bounds")
    return rep


def decode_plan(P, G, Hq, Hkv, D, prefix_start, prefix_len, suffix_start, suffix_len,
                prefix_rows, suffix_rows, scale=None, split_tokens: int = 0) -> np.ndarray:
    """The split-K work list (host-only), as a numpy structured array in launch order."""
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    a = _DecodeArgs(P, G, Hq, Hkv, D, scale, split_tokens, prefix_start, prefix_len,
                    suffix_start, suffix_len, prefix_rows, suffix_rows)
    n = ctypes.c_int64(0)
    _check(_lib.rl_decode_plan_debug(ctypes.byref(a.shape), ctypes.byref(a.lens), None, 0,
                                     ctypes.byref(n)), "rl_decode_plan_debug")
    buf = (PlanItem * max(1, n.value))()
    _check(_lib.rl_decode_plan_debug(ctypes.byref(a.shape), ctypes.byref(a.lens), buf, n.value,
                                     ctypes.byref(n)), "rl_decode_plan_debug")
    dt = np.dtype([("kind", np.int32), ("unit", np.int32), ("kv_head", np.int32),
                   ("chunk", np.int32), ("tok_begin", np.int64), ("tok_count", np.int32),
                   ("row_begin", np.int32), ("row_count", np.int32), ("split_variant", np.int32)])
    return np.frombuffer(bytes(buf), dtype=dt, count=n.value).copy()


class _AppendArgs:
    """Host-side marshalling of rl_kv_append's shape and lengths (keeps the arrays alive)."""

    def __init__(self, P, G, Hkv, D, suffix_start, suffix_len, new_start, new_len, suffix_rows, new_rows,
                 suffix_capacity=None, kv_layout: str = "token"):
        self.ss = np.ascontiguousarray(suffix_start, dtype=np.int64)
        self.sl = np.ascontiguousarray(suffix_len, dtype=np.int32)
        self.ns = np.ascontiguousarray(new_start, dtype=np.int64)
        self.nl = np.ascontiguousarray(new_len, dtype=np.int32)
        self.cap = None if suffix_capacity is None else np.ascontiguousarray(suffix_capacity, dtype=np.int32)
        S = P * G
        for arr, n in ((self.ss, "suffix_start"), (self.sl, "suffix_len"), (self.ns, "new_start"),
                       (self.nl, "new_len")) + (((self.cap, "suffix_capacity"),) if self.cap is not None else ()):
            if arr.shape != (S,):
                raise ValueError(f"{n} must have P*G = {S} entries")
        if kv_layout not in KV_LAYOUTS:
            raise ValueError(f"kv_layout must be one of {sorted(KV_LAYOUTS)}")
        self.shape = DecodeShape(P, G, 1, Hkv, D, 1.0, 0, KV_LAYOUTS[kv_layout])
        self.lens = KvAppendLens(self.ss.ctypes.data, self.sl.ctypes.data,
                                 None if self.cap is None else self.cap.ctypes.data,
                                 self.ns.ctypes.data, self.nl.ctypes.data, int(suffix_rows), int(new_rows))


@_on_call_stream
def kv_append(k_new: torch.Tensor, v_new: torch.Tensor, k_suffix: torch.Tensor, v_suffix: torch.Tensor,
              suffix_start, suffix_len, new_start, new_len, group_size: int, suffix_capacity=None,
              kv_layout: str = "token", workspace: Optional[torch.Tensor] = None, stream=None):
    """Writes rows new_start[s] + i of k_new / v_new ([new_rows, Hkv, D]) to suffix rows
    suffix_start[s] + suffix_len[s] + i of the caches, for i < new_len[s]."""
    for t, n in ((k_new, "k_new"), (v_new, "v_new"), (k_suffix, "k_suffix"), (v_suffix, "v_suffix")):
        _bf16_dev(t, n)
    if k_new.dim() != 3 or v_new.shape != k_new.shape:
        raise ValueError("k_new / v_new must be [new_rows, Hkv, D]")
    new_rows, Hkv, D = k_new.shape
    if k_suffix.shape != v_suffix.shape or k_suffix.dim() != 3:
        raise ValueError("k_suffix / v_suffix must have the same 3-d shape")
    rdim = 1 if kv_layout == "head" else 0
    hdim = 0 if kv_layout == "head" else 1
    if k_suffix.shape[hdim] != Hkv or k_suffix.shape[2] != D:
        raise ValueError("suffix caches do not match k_new's heads / head_dim")
    G = int(group_size)
    S = len(np.asarray(suffix_start))
    if G <= 0 or S % G:
        raise ValueError("the number of candidates must be a multiple of group_size")
    a = _AppendArgs(S // G, G, Hkv, D, suffix_start, suffix_len, new_start, new_len, k_suffix.shape[rdim],
                    new_rows, suffix_capacity, kv_layout)
    n = ctypes.c_size_t(0)
    _check(_lib.rl_kv_append_workspace_size(ctypes.byref(a.shape), ctypes.byref(a.lens), ctypes.byref(n)),
           "rl_kv_append_workspace_size")
    if workspace is None:
        workspace = torch.empty(max(n.value, 1), dtype=torch.uint8, device=k_new.device)
    _on_device(workspace, "workspace")
    _check(_lib.rl_kv_append(ctypes.byref(a.shape), ctypes.byref(a.lens), _ptr(k_new), _ptr(v_new),
                             _ptr(k_suffix), _ptr(v_suffix), ctypes.c_void_p(workspace.data_ptr()),
                             workspace.numel(), _stream_handle(stream)), "rl_kv_append")


def _decode_prepare(q, k_prefix, v_prefix, k_suffix, v_suffix, prefix_start, prefix_len, suffix_start, suffix_len,
                    group_size, scale, split_tokens, return_lse, out, lse, workspace, kv_layout):
    """Validation and marshalling shared by decode_attn and decode_attn_timeline."""
    for t, n in ((q, "q"), (k_prefix, "k_prefix"), (v_prefix, "v_prefix"),
                 (k_suffix, "k_suffix"), (v_suffix, "v_suffix")):
        _bf16_dev(t, n)
    S, Hq, D = q.shape
    G = int(group_size)
    if G <= 0 or S % G:
        raise ValueError("q.shape[0] must be a positive multiple of group_size")
    P = S // G
    head_major = kv_layout == "head"
    hdim, rdim = (0, 1) if head_major else (1, 0)
    Hkv = k_prefix.shape[hdim]
    for t in (k_prefix, v_prefix, k_suffix, v_suffix):
        if t.dim() != 3 or t.shape[hdim] != Hkv or t.shape[2] != D:
            raise ValueError("KV tensors must be [rows, Hkv, D] (token) or [Hkv, rows, D] (head)")
    if k_prefix.shape != v_prefix.shape or k_suffix.shape != v_suffix.shape:
        raise ValueError("K and V shapes differ")
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    a = _DecodeArgs(P, G, Hq, Hkv, D, scale, split_tokens, prefix_start, prefix_len,
                    suffix_start, suffix_len, k_prefix.shape[rdim], k_suffix.shape[rdim], kv_layout)
    if out is None:
        out = torch.empty((S, Hq, D), dtype=torch.bfloat16, device=q.device)
    if return_lse and lse is None:
        lse = torch.empty((S, Hq), dtype=torch.float32, device=q.device)
    _bf16_dev(out, "out")
    if out.shape != (S, Hq, D):
        raise ValueError("out must be [P*G, Hq, D]")
    if lse is not None:
        _on_device(lse, "lse")
        if lse.dtype != torch.float32 or lse.shape != (S, Hq) or not lse.is_contiguous():
            raise ValueError("lse must be a contiguous fp32 [P*G, Hq] tensor")
    need = ctypes.c_size_t(0)
    _check(_lib.rl_decode_attn_workspace_size(ctypes.byref(a.shape), ctypes.byref(a.lens),
                                              ctypes.byref(need)), "rl_decode_attn_workspace_size")
    if workspace is None:
        workspace = torch.empty(max(need.value, 1), dtype=torch.uint8, device=q.device)
    _on_device(workspace, "workspace")
    ptrs = DecodePtrs(q.data_ptr(), k_prefix.data_ptr() if k_prefix.numel() else None,
                      v_prefix.data_ptr() if v_prefix.numel() else None,
                      k_suffix.data_ptr() if k_suffix.numel() else None,
                      v_suffix.data_ptr() if v_suffix.numel() else None,
                      out.data_ptr(), lse.data_ptr() if lse is not None else None)
    return a, out, lse, workspace, ptrs


@_on_call_stream
def decode_attn(q: torch.Tensor, k_prefix: torch.Tensor, v_prefix: torch.Tensor,
                k_suffix: torch.Tensor, v_suffix: torch.Tensor,
                prefix_start, prefix_len, suffix_start, suffix_len, group_size: int,
                scale: Optional[float] = None, split_tokens: int = 0, return_lse: bool = False,
                out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, stream=None, kv_layout: str = "token"):
    """Decode attention of P*G candidates over their prompt's prefix KV ++ own suffix KV.

    q [P*G, Hq, D] bf16; k/v_prefix and k/v_suffix bf16 device tensors laid out
    [rows, Hkv, D] (kv_layout="token") or [Hkv, rows, D] (kv_layout="head");
    prefix_start/len [P], suffix_start/len [P*G] host integers.
    Returns out [P*G, Hq, D] bf16 (and lse [P*G, Hq] fp32 natural log).
    """
    a, out, lse, workspace, ptrs = _decode_prepare(q, k_prefix, v_prefix, k_suffix, v_suffix, prefix_start,
                                                   prefix_len, suffix_start, suffix_len, group_size, scale,
                                                   split_tokens, return_lse, out, lse, workspace, kv_layout)
    _check(_lib.rl_decode_attn(ctypes.byref(a.shape), ctypes.byref(a.lens), ctypes.byref(ptrs),
                               ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                               _stream_handle(stream)), "rl_decode_attn")
    return (out, lse) if return_lse else out


@_on_call_stream
def decode_attn_timeline(q: torch.Tensor, k_prefix: torch.Tensor, v_prefix: torch.Tensor,
                         k_suffix: torch.Tensor, v_suffix: torch.Tensor,
                         prefix_start, prefix_len, suffix_start, suffix_len, group_size: int,
                         scale: Optional[float] = None, split_tokens: int = 0,
                         workspace: Optional[torch.Tensor] = None, stream=None, kv_layout: str = "token"):
    """decode_attn through rl_debug_decode_timeline: returns (out, lse,
    records), records an int64 [n_items, TIMELINE_WORDS] device tensor, one
    timeline record per work item of the split kernel (layout in rl_kernels.h)."""
    a, out, lse, workspace, ptrs = _decode_prepare(q, k_prefix, v_prefix, k_suffix, v_suffix, prefix_start,
                                                   prefix_len, suffix_start, suffix_len, group_size, scale,
                                                   split_tokens, True, None, None, workspace, kv_layout)
    n = ctypes.c_int64(0)
    _check(_lib.rl_debug_decode_timeline(ctypes.byref(a.shape), ctypes.byref(a.lens), None, None, 0, None, 0,
                                         ctypes.byref(n), None), "rl_debug_decode_timeline")
    records = torch.zeros((max(n.value, 1), TIMELINE_WORDS), dtype=torch.int64, device=q.device)
    _check(_lib.rl_debug_decode_timeline(ctypes.byref(a.shape), ctypes.byref(a.lens), ctypes.byref(ptrs),
                                         ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                         ctypes.c_void_p(records.data_ptr()), n.value, ctypes.byref(n),
                                         _stream_handle(stream)), "rl_debug_decode_timeline")
    return out, lse, records[:n.value]


class _ExtendArgs:
    """Host-side ctypes structures for one extend call (kept alive by the caller)."""

    def __init__(self, P, G, Hq, Hkv, D, scale, prefix_start, prefix_len, suffix_start, suffix_len,
                 new_len, q_start, prefix_rows, suffix_rows, q_rows, kv_layout="token"):
        self.ps = np.ascontiguousarray(prefix_start, dtype=np.int64)
        self.pl = np.ascontiguousarray(prefix_len, dtype=np.int32)
        self.ss = np.ascontiguousarray(suffix_start, dtype=np.int64)
        self.sl = np.ascontiguousarray(suffix_len, dtype=np.int32)
        self.nl = np.ascontiguousarray(new_len, dtype=np.int32)
        self.qs = np.ascontiguousarray(q_start, dtype=np.int64)
        S = P * G
        if self.ps.shape != (P,) or self.pl.shape != (P,) or \
                any(x.shape != (S,) for x in (self.ss, self.sl, self.nl, self.qs)):
            raise ValueError("length arrays must be [P] (prefix) and [P*G] (candidates)")
        if kv_layout not in KV_LAYOUTS:
            raise ValueError(f"kv_layout must be one of {sorted(KV_LAYOUTS)}")
        self.shape = DecodeShape(P, G, Hq, Hkv, D, float(np.float32(scale)), 0, KV_LAYOUTS[kv_layout])
        self.lens = ExtendLens(self.ps.ctypes.data, self.pl.ctypes.data, self.ss.ctypes.data,
                               self.sl.ctypes.data, self.nl.ctypes.data, self.qs.ctypes.data,
                               int(prefix_rows), int(suffix_rows), int(q_rows))


def extend_attn_workspace_size(P, G, Hq, Hkv, D, prefix_start, prefix_len, suffix_start, suffix_len,
                               new_len, q_start, prefix_rows, suffix_rows, q_rows, scale=None,
                               kv_layout: str = "token") -> int:
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    a = _ExtendArgs(P, G, Hq, Hkv, D, scale, prefix_start, prefix_len, suffix_start, suffix_len,
                    new_len, q_start, prefix_rows, suffix_rows, q_rows, kv_layout)
    n = ctypes.c_size_t(0)
    _check(_lib.rl_extend_attn_workspace_size(ctypes.byref(a.shape), ctypes.byref(a.lens), ctypes.byref(n)),
           "rl_extend_attn_workspace_size")
    return n.value


@_on_call_stream
def extend_attn(q: torch.Tensor, k_prefix: torch.Tensor, v_prefix: torch.Tensor,
                k_suffix: torch.Tensor, v_suffix: torch.Tensor,
                prefix_start, prefix_len, suffix_start, suffix_len, new_len, q_start, group_size: int,
                scale: Optional[float] = None, return_lse: bool = False,
                out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, stream=None, kv_layout: str = "token"):
    """Causal extend (prefill) attention of each candidate's new tokens.

    The last new_len[s] tokens of candidate s's suffix are new; new token i
    (query row q_start[s] + i of q) attends to the prompt's prefix and to the
    suffix up to and including itself.  q [Q, Hq, D] bf16; KV tensors as for
    decode_attn; length arrays on the host.  Returns out [Q, Hq, D] bf16 (and
    lse [Q, Hq] fp32); rows of no candidate are left as allocated.
    """
    for t, n in ((q, "q"), (k_prefix, "k_prefix"), (v_prefix, "v_prefix"),
                 (k_suffix, "k_suffix"), (v_suffix, "v_suffix")):
        _bf16_dev(t, n)
    Q, Hq, D = q.shape
    G = int(group_size)
    S = len(suffix_len)
    if G <= 0 or S % G:
        raise ValueError("the number of candidates must be a positive multiple of group_size")
    P = S // G
    head_major = kv_layout == "head"
    hdim, rdim = (0, 1) if head_major else (1, 0)
    Hkv = k_suffix.shape[hdim]
    for t in (k_prefix, v_prefix, k_suffix, v_suffix):
        if t.dim() != 3 or t.shape[hdim] != Hkv or t.shape[2] != D:
            raise ValueError("KV tensors must be [rows, Hkv, D] (token) or [Hkv, rows, D] (head)")
    if k_prefix.shape != v_prefix.shape or k_suffix.shape != v_suffix.shape:
        raise ValueError("K and V shapes differ")
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    a = _ExtendArgs(P, G, Hq, Hkv, D, scale, prefix_start, prefix_len, suffix_start, suffix_len,
                    new_len, q_start, k_prefix.shape[rdim], k_suffix.shape[rdim], Q, kv_layout)
    if out is None:
        out = torch.empty((Q, Hq, D), dtype=torch.bfloat16, device=q.device)
    if return_lse and lse is None:
        lse = torch.empty((Q, Hq), dtype=torch.float32, device=q.device)
    _bf16_dev(out, "out")
    if out.shape != (Q, Hq, D):
        raise ValueError("out must be [Q, Hq, D]")
    if lse is not None:
        _on_device(lse, "lse")
        if lse.dtype != torch.float32 or lse.shape != (Q, Hq) or not lse.is_contiguous():
            raise ValueError("lse must be a contiguous fp32 [Q, Hq] tensor")
    need = ctypes.c_size_t(0)
    _check(_lib.rl_extend_attn_workspace_size(ctypes.byref(a.shape), ctypes.byref(a.lens), ctypes.byref(need)),
           "rl_extend_attn_workspace_size")
    if workspace is None:
        workspace = torch.empty(max(need.value, 1), dtype=torch.uint8, device=q.device)
    _on_device(workspace, "workspace")
    ptrs = DecodePtrs(q.data_ptr() if q.numel() else None, k_prefix.data_ptr() if k_prefix.numel() else None,
                      v_prefix.data_ptr() if v_prefix.numel() else None,
                      k_suffix.data_ptr() if k_suffix.numel() else None,
                      v_suffix.data_ptr() if v_suffix.numel() else None,
                      out.data_ptr() if out.numel() else None, lse.data_ptr() if lse is not None and lse.numel() else None)
    _check(_lib.rl_extend_attn(ctypes.byref(a.shape), ctypes.byref(a.lens), ctypes.byref(ptrs),
                               ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                               _stream_handle(stream)), "rl_extend_attn")
    return (out, lse) if return_lse else out


def token_logprob_workspace_size(rows: int, hidden: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.rl_token_logprob_workspace_size(rows, hidden, vocab, ctypes.byref(n)),
           "rl_token_logprob_workspace_size")
    return n.value


@_on_call_stream
def token_logprob(hidden: torch.Tensor, w_lm: torch.Tensor, target: torch.Tensor,
                  inv_temperature: float = 1.0, logprob: Optional[torch.Tensor] = None,
                  lse: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                  stream=None):
    """Log-prob of target[r] under softmax(inv_temperature * hidden[r] @ w_lm^T).

    hidden [R, H] bf16, w_lm [V, H] bf16, target [R] int32 (device; -1 = masked).
    Returns (logprob [R] fp32, lse [R] fp32).
    """
    _bf16_dev(hidden, "hidden")
    _bf16_dev(w_lm, "w_lm")
    _on_device(target, "target")
    if target.dtype != torch.int32 or not target.is_contiguous():
        raise TypeError("target must be a contiguous int32 tensor")
    R, H = hidden.shape
    V, H2 = w_lm.shape
    if H2 != H or target.shape != (R,):
        raise ValueError("shapes: hidden [R, H], w_lm [V, H], target [R]")
    if logprob is None:
        logprob = torch.empty(R, dtype=torch.float32, device=hidden.device)
    if lse is None:
        lse = torch.empty(R, dtype=torch.float32, device=hidden.device)
    for t, n in ((logprob, "logprob"), (lse, "lse")):
        _on_device(t, n)
        if t.dtype != torch.float32 or t.shape != (R,) or not t.is_contiguous():
            raise ValueError(f"{n} must be a contiguous fp32 [R] tensor")
    need = token_logprob_workspace_size(R, H, V)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=hidden.device)
    _on_device(workspace, "workspace")
    _check(_lib.rl_token_logprob(R, H, V, _ptr(hidden), _ptr(w_lm), _ptr(target),
                                 float(inv_temperature), _ptr(logprob), _ptr(lse),
                                 ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                 _stream_handle(stream)), "rl_token_logprob")
    return logprob, lse


NOALLOC_SCRATCH_BYTES = 128 << 20


@_on_call_stream
def token_logprob_noalloc(hidden: torch.Tensor, w_lm: torch.Tensor, target: torch.Tensor,
                          logprob: torch.Tensor, lse: Optional[torch.Tensor] = None,
                          inv_temperature: float = 1.0, stream=None):
    """token_logprob through rl_token_logprob_noalloc: no workspace, and
    nothing allocated here either (the caller passes the outputs).  Its
    scratch is one static device array per GPU, so calls that overlap on a GPU
    race; sizes whose workspace exceeds NOALLOC_SCRATCH_BYTES raise."""
    _bf16_dev(hidden, "hidden")
    _bf16_dev(w_lm, "w_lm")
    _on_device(target, "target")
    if target.dtype != torch.int32 or not target.is_contiguous():
        raise TypeError("target must be a contiguous int32 tensor")
    R, H = hidden.shape
    V, H2 = w_lm.shape
    if H2 != H or target.shape != (R,):
        raise ValueError("shapes: hidden [R, H], w_lm [V, H], target [R]")
    for t, n in ((logprob, "logprob"), (lse, "lse")):
        if t is None and n == "lse":
            continue
        _on_device(t, n)
        if t.dtype != torch.float32 or t.shape != (R,) or not t.is_contiguous():
            raise ValueError(f"{n} must be a contiguous fp32 [R] tensor")
    _check(_lib.rl_token_logprob_noalloc(R, H, V, _ptr(hidden), _ptr(w_lm), _ptr(target), float(inv_temperature),
                                         _ptr(logprob), _ptr(lse) if lse is not None else None,
                                         _stream_handle(stream)), "rl_token_logprob_noalloc")
    return logprob, lse


def logprob_bounds(op: int, rows: int, hidden: int, vocab: int, every_stage: bool = False,
                   shrink_region: int = -1) -> BoundsReport:
    """Host replay of the global accesses of rl_token_logprob (op 0),
    rl_token_logprob_backward (op 1) or rl_sample_top_p (op 2) at these
    sizes (no device access)."""
    rep = BoundsReport()
    _check(_lib.rl_debug_logprob_bounds(op, rows, hidden, vocab, int(bool(every_stage)), shrink_region,
                                        ctypes.byref(rep)), "rl_debug_logprob_bounds")
    return rep


def extend_bounds(P, G, Hq, Hkv, D, prefix_start, prefix_len, suffix_start, suffix_len, new_len, q_start,
                  prefix_rows, suffix_rows, q_rows, kv_layout: str = "token", every_stage: bool = False,
                  shrink_region: int = -1) -> BoundsReport:
    """Host replay of the global accesses of rl_extend_attn for these lengths
    (no device access)."""
    a = _ExtendArgs(P, G, Hq, Hkv, D, 1.0 / math.sqrt(D), prefix_start, prefix_len, suffix_start, suffix_len,
                    new_len, q_start, prefix_rows, suffix_rows, q_rows, kv_layout)
    rep = BoundsReport()
    _check(_lib.rl_debug_extend_bounds(ctypes.byref(a.shape), ctypes.byref(a.lens), int(bool(every_stage)),
                                       shrink_region, ctypes.byref(rep)), "rl_debug_extend_bounds")
    return rep


TIMELINE_WORDS = 8


def logprob_timeline_records(rows: int, hidden: int, vocab: int) -> int:
    """Number of records rl_debug_logprob_timeline writes at these sizes."""
    n = ctypes.c_int64(0)
    _check(_lib.rl_debug_logprob_timeline(rows, hidden, vocab, None, None, None, 1.0, None, None, None, 0, None, 0,
                                          ctypes.byref(n), None), "rl_debug_logprob_timeline")
    return n.value


@_on_call_stream
def token_logprob_timeline(hidden: torch.Tensor, w_lm: torch.Tensor, target: torch.Tensor,
                           inv_temperature: float = 1.0, stream=None):
    """token_logprob through rl_debug_logprob_timeline: returns (logprob, lse,
    records), records an int64 [n, TIMELINE_WORDS] device tensor holding the
    per-wave timeline of the tile launches (word layout in rl_kernels.h)."""
    _bf16_dev(hidden, "hidden")
    _bf16_dev(w_lm, "w_lm")
    _on_device(target, "target")
    if target.dtype != torch.int32 or not target.is_contiguous():
        raise TypeError("target must be a contiguous int32 tensor")
    R, H = hidden.shape
    V, H2 = w_lm.shape
    if H2 != H or target.shape != (R,):
        raise ValueError("shapes: hidden [R, H], w_lm [V, H], target [R]")
    logprob = torch.empty(R, dtype=torch.float32, device=hidden.device)
    lse = torch.empty(R, dtype=torch.float32, device=hidden.device)
    need = token_logprob_workspace_size(R, H, V)
    workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=hidden.device)
    cap = logprob_timeline_records(R, H, V)
    records = torch.zeros((max(cap, 1), TIMELINE_WORDS), dtype=torch.int64, device=hidden.device)
    n = ctypes.c_int64(0)
    _check(_lib.rl_debug_logprob_timeline(R, H, V, _ptr(hidden), _ptr(w_lm), _ptr(target), float(inv_temperature),
                                          _ptr(logprob), _ptr(lse), ctypes.c_void_p(workspace.data_ptr()),
                                          workspace.numel(), ctypes.c_void_p(records.data_ptr()), cap,
                                          ctypes.byref(n), _stream_handle(stream)), "rl_debug_logprob_timeline")
    return logprob, lse, records[:n.value]


def token_logprob_backward_workspace_size(rows: int, hidden: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.rl_token_logprob_backward_workspace_size(rows, hidden, vocab, ctypes.byref(n)),
           "rl_token_logprob_backward_workspace_size")
    return n.value


@_on_call_stream
def token_logprob_backward(hidden: torch.Tensor, w_lm: torch.Tensor, target: torch.Tensor,
                           lse: torch.Tensor, grad_logprob: torch.Tensor, inv_temperature: float = 1.0,
                           grad_hidden: Optional[torch.Tensor] = None,
                           workspace: Optional[torch.Tensor] = None, stream=None):
    """d(sum_r grad_logprob[r] * logprob[r]) / d hidden, fp32 [R, H].

    lse is the forward's lse for the same inputs (token_logprob's second output).
    """
    _bf16_dev(hidden, "hidden")
    _bf16_dev(w_lm, "w_lm")
    _on_device(target, "target")
    if target.dtype != torch.int32 or not target.is_contiguous():
        raise TypeError("target must be a contiguous int32 tensor")
    R, H = hidden.shape
    V, H2 = w_lm.shape
    if H2 != H or target.shape != (R,):
        raise ValueError("shapes: hidden [R, H], w_lm [V, H], target [R]")
    _f32_dev(lse, "lse", (R,))
    _f32_dev(grad_logprob, "grad_logprob", (R,))
    if grad_hidden is None:
        grad_hidden = torch.empty(R, H, dtype=torch.float32, device=hidden.device)
    _f32_dev(grad_hidden, "grad_hidden", (R, H))
    need = token_logprob_backward_workspace_size(R, H, V)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=hidden.device)
    _on_device(workspace, "workspace")
    _check(_lib.rl_token_logprob_backward(R, H, V, _ptr(hidden), _ptr(w_lm), _ptr(target),
                                          float(inv_temperature), _ptr(lse), _ptr(grad_logprob),
                                          _ptr(grad_hidden), ctypes.c_void_p(workspace.data_ptr()),
                                          workspace.numel(), _stream_handle(stream)),
           "rl_token_logprob_backward")
    return grad_hidden


def sample_top_p_workspace_size(rows: int, hidden: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.rl_sample_top_p_workspace_size(rows, hidden, vocab, ctypes.byref(n)),
           "rl_sample_top_p_workspace_size")
    return n.value


@_on_call_stream
def sample_top_p(hidden: torch.Tensor, w_lm: torch.Tensor, inv_temperature: torch.Tensor, top_p: float,
                 uniform: torch.Tensor, token: Optional[torch.Tensor] = None,
                 logprob: Optional[torch.Tensor] = None, want_logprob: bool = True,
                 workspace: Optional[torch.Tensor] = None, stream=None):
    """Nucleus sampling of one token per row at a per-row temperature.

    hidden [R, H] bf16, w_lm [V, H] bf16, inv_temperature [R] fp32 (1/T per row),
    uniform [R] fp32 draws in [0, 1).  Returns (token int32 [R], logprob fp32 [R] or None).
    """
    _bf16_dev(hidden, "hidden")
    _bf16_dev(w_lm, "w_lm")
    R, H = hidden.shape
    V, H2 = w_lm.shape
    if H2 != H:
        raise ValueError("shapes: hidden [R, H], w_lm [V, H]")
    _f32_dev(inv_temperature, "inv_temperature", (R,))
    _f32_dev(uniform, "uniform", (R,))
    if token is None:
        token = torch.empty(R, dtype=torch.int32, device=hidden.device)
    _on_device(token, "token")
    if token.dtype != torch.int32 or token.shape != (R,) or not token.is_contiguous():
        raise ValueError("token must be a contiguous int32 [R] tensor")
    if logprob is None and want_logprob:
        logprob = torch.empty(R, dtype=torch.float32, device=hidden.device)
    if logprob is not None:
        _f32_dev(logprob, "logprob", (R,))
    need = sample_top_p_workspace_size(R, H, V)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=hidden.device)
    _on_device(workspace, "workspace")
    _check(_lib.rl_sample_top_p(R, H, V, _ptr(hidden), _ptr(w_lm), _ptr(inv_temperature), float(top_p),
                                _ptr(uniform), _ptr(token), _ptr(logprob),
                                ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                _stream_handle(stream)), "rl_sample_top_p")
    return token, logprob


def _f32_dev(t: torch.Tensor, name: str, shape) -> torch.Tensor:
    _on_device(t, name)
    if t.dtype != torch.float32 or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be a contiguous fp32 device tensor of shape {tuple(shape)}")
    return t


@_on_call_stream
def grpo_advantage(reward: torch.Tensor, group_size: int, adv: Optional[torch.Tensor] = None, stream=None):
    """Group-relative advantages (r - mean) / std over each group of group_size rewards.

    reward: fp32 [P*G] device tensor.  Returns adv fp32 [P*G].
    """
    G = int(group_size)
    n = reward.numel()
    if G <= 0 or n % G:
        raise ValueError("reward length must be a positive multiple of group_size")
    _f32_dev(reward, "reward", (n,))
    if adv is None:
        adv = torch.empty_like(reward)
    _f32_dev(adv, "adv", (n,))
    _check(_lib.rl_grpo_advantage(n // G, G, _ptr(reward), _ptr(adv), _stream_handle(stream)),
           "rl_grpo_advantage")
    return adv


def grpo_surrogate_workspace_size(rows: int, num_prompts: int, group_size: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.rl_grpo_surrogate_workspace_size(rows, num_prompts, group_size, ctypes.byref(n)),
           "rl_grpo_surrogate_workspace_size")
    return n.value


@_on_call_stream
def grpo_surrogate(logp_new: torch.Tensor, logp_old: torch.Tensor, seq: torch.Tensor, adv: torch.Tensor,
                   group_size: int, eps: float = 0.2, loss: Optional[torch.Tensor] = None,
                   grad: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None, stream=None):
    """Clipped GRPO surrogate loss (beta = 0) and its gradient with respect to logp_new.

    logp_new, logp_old: fp32 [R]; seq: int32 [R] (candidate of each row, -1 = none);
    adv: fp32 [P*G].  Returns (loss fp32 [1], grad fp32 [R]).
    """
    G = int(group_size)
    R = logp_new.numel()
    S = adv.numel()
    if G <= 0 or S % G:
        raise ValueError("adv length must be a positive multiple of group_size")
    _f32_dev(logp_new, "logp_new", (R,))
    _f32_dev(logp_old, "logp_old", (R,))
    _f32_dev(adv, "adv", (S,))
    _on_device(seq, "seq")
    if seq.dtype != torch.int32 or not seq.is_contiguous() or tuple(seq.shape) != (R,):
        raise ValueError("seq must be a contiguous int32 device tensor of shape (R,)")
    dev = logp_new.device
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=dev)
    if grad is None:
        grad = torch.empty(R, dtype=torch.float32, device=dev)
    _f32_dev(loss, "loss", (1,))
    _f32_dev(grad, "grad", (R,))
    need = grpo_surrogate_workspace_size(R, S // G, G)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    _on_device(workspace, "workspace")
    _check(_lib.rl_grpo_surrogate(R, S // G, G, _ptr(logp_new), _ptr(logp_old), _ptr(seq), _ptr(adv),
                                  float(eps), _ptr(loss), _ptr(grad), ctypes.c_void_p(workspace.data_ptr()),
                                  workspace.numel(), _stream_handle(stream)), "rl_grpo_surrogate")
    return loss, grad
