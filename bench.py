#!/usr/bin/env python3
"""Throughput of the rollout hot path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input that is
already resident in HBM: prefix-shared decode attention for all candidates of
the batch, then the fused lm-head token log-prob of their rows.  The default
(headline) workload is the 32B-class single-layer decode step, the largest
configuration with both halves of the path: 16 prompts x G=16, 64 query / 8
kv heads, head dim 128, shared prefix 2048, suffix lengths uniform in [512,
8192]; lm-head 256 rows x hidden 5120 x vocab 151936.  `value` is its decode
attention's effective KV bandwidth (algorithmic bytes, the prefix counted once
per prompt, over the measured decode time); `roofline` is the entry of the
operation that takes the most time, `roofline_other` the other one's.

The same run then measures the other configurations (--also, by default the
8B-class step, the multi-turn long context and the 262144-row policy pass),
each reported under "configs" with its own roofline entries, host time per
call and CPU baseline.  They are not part of the headline's timed steps.

Before every timed operation a 1 GiB buffer is read (outside the events), so
no operation finds its inputs in the 256 MB MALL or the L2 from the previous
one.  It is read, not written: a written buffer leaves the MALL full of
dirty lines, and their write-back would land inside the next timed
operation.  Per-operation durations are the medians of HIP events recorded on
the stream the kernels run on (created with a device-scope release, so
recording one does not write back the L2 to system memory and the interval
matches the kernels' own durations).  host_us is the wall time of the host
side of one call with the GPU idle (the binding's marshalling, the library's
planning and the launches), the median of a separate loop.

After the headline's steps, further operations at its shape are timed in
loops of their own and reported under "extra_ops": the KV append of one
token per candidate, the extend (prefill) of a refinement turn with every
suffix token new, the backward of the lm-head log-prob for the same rows, the
GRPO advantages and clipped surrogate over the policy pass's 262144 rows, and
the nucleus sampling head over the same rows.

Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2516.6  # MI355X dense bf16 MFMA (256 CUs x 4096 flop/clk x 2.4 GHz)

WORKLOADS = {
    # name: (decode config or None, logprob config or None, description)
    "8b": ("8b", "8b", "8B-class decode step: 64 prompts x G=8, 32/8 heads, D=128, prefix 1024, "
                       "suffix U[256,2048]; lm-head 512 x 4096 x 151936"),
    "32b": ("32b", "32b", "32B-class decode step: 16 prompts x G=16, 64/8 heads, D=128, prefix 2048, "
                          "suffix U[512,8192]; lm-head 256 x 5120 x 151936"),
    "longctx": ("longctx", None, "multi-turn long context: 4 prompts x G=8, 64/8 heads, D=128, "
                                 "prefix 24576, suffix geometric mean 1024 cap 4096"),
    "policy": (None, "policy", "policy-update log-prob pass: 262144 rows x 5120 x 151936"),
}


class HipEvents:
    """hipEventCreateWithFlags / Record / ElapsedTime through the HIP runtime the
    process already uses, with hipEventReleaseToDevice: a timing event that only
    needs device-scope ordering (torch.cuda.Event always fences at system scope)."""
    RELEASE_TO_DEVICE = 0x40000000

    def __init__(self, runtime_path: str):
        import ctypes
        self.ct = ctypes
        self.lib = ctypes.CDLL(runtime_path)
        self.lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        ev = self.ct.c_void_p()
        st = self.lib.hipEventCreateWithFlags(self.ct.byref(ev), self.RELEASE_TO_DEVICE)
        if st != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({st})")
        return ev

    def record(self, ev, stream_handle: int):
        st = self.lib.hipEventRecord(ev, self.ct.c_void_p(stream_handle))
        if st != 0:
            raise RuntimeError(f"hipEventRecord failed ({st})")

    def elapsed_ms(self, a, b) -> float:
        ms = self.ct.c_float()
        st = self.lib.hipEventElapsedTime(self.ct.byref(ms), a, b)
        if st != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({st})")
        return ms.value

    def destroy(self, ev):
        self.lib.hipEventDestroy(ev)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


CSRC = os.path.join(ROOT, "paper_2607_20908_amd", "csrc")
KERNEL_SOURCES = {"decode": "decode_attn.hip", "lmhead": "token_logprob.hip"}


def _local_sources(name: str, seen=None) -> list:
    """The kernel source and every header of the package it includes, in a
    fixed order."""
    import re
    seen = [] if seen is None else seen
    if name in seen or not os.path.exists(os.path.join(CSRC, name)):
        return seen
    seen.append(name)
    with open(os.path.join(CSRC, name)) as f:
        for inc in re.findall(r'^#include "([^"]+)"', f.read(), re.M):
            _local_sources(inc, seen)
    return seen


def source_sha256(op: str) -> str:
    """sha256 of the op's kernel source followed by the package headers it
    includes (so a change in a shared header also retires old counters)."""
    import hashlib
    h = hashlib.sha256()
    for name in _local_sources(KERNEL_SOURCES[op]):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(op: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary of this
    op and workload, if that summary was taken on the current kernel source;
    otherwise None.  The summary holds lines `source_sha256: ...` and
    `hbm_bytes_per_launch: ...` (FETCH_SIZE + WRITE_SIZE, calibrated)."""
    path = os.path.join(ROOT, "profiles", f"{op}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                fields[k.strip().strip("-* `")] = v.strip().strip("`")
    if fields.get("source_sha256") != source_sha256(op):
        return None
    try:
        return int(float(fields["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def decode_bytes(x) -> int:
    """Algorithmic HBM bytes of one decode-attention call: K and V of every
    prefix token once per prompt and of every suffix token once, q read, out
    written (bf16), lse written (fp32)."""
    c = x.cfg
    S = c.num_seqs
    kv = 2 * 2 * c.head_dim * c.num_kv_heads * (int(x.prefix_len.sum()) + int(x.suffix_len.sum()))
    return kv + 2 * (2 * S * c.num_q_heads * c.head_dim) + 4 * S * c.num_q_heads


def lmhead_flops(cfg) -> int:
    return 2 * cfg.rows * cfg.hidden * cfg.vocab


def lmhead_bytes(cfg) -> int:
    """Algorithmic HBM bytes of one lm-head pass: W and the hidden rows read
    once, target read, log-prob and lse written."""
    return 2 * cfg.vocab * cfg.hidden + 2 * cfg.rows * cfg.hidden + 4 * cfg.rows + 8 * cfg.rows


def grpo_bytes(gx) -> int:
    """Algorithmic HBM bytes of the GRPO advantages and surrogate: rewards read
    and advantages written; per row logp_new, logp_old and seq read and grad
    written; the loss written."""
    S = gx.reward.numel()
    R = gx.seq.numel()
    return 8 * S + 16 * R + 4


def extend_flops(xe) -> int:
    """Algorithmic flops of one extend call: 2 D for the score and 2 D for the
    value sum of every (new token, query head, visible token)."""
    c = xe.dec.cfg
    vis = 0
    for s in range(c.num_seqs):
        n = int(xe.new_len[s])
        base = int(xe.dec.prefix_len[s // c.group_size]) + int(xe.dec.suffix_len[s]) - n
        vis += n * base + n * (n + 1) // 2
    return 4 * c.head_dim * c.num_q_heads * vis


def cpu_baseline_decode(x, budget_s: float):
    """The fp64 oracle on the host over the workload's prompts (all their
    candidates), prompt by prompt, cycling through the batch until the time
    budget is spent."""
    import oracle
    import workloads as W
    c = x.cfg
    G = c.group_size
    q = W.bf16_bits(x.q)
    kp, vp = W.bf16_bits(x.token_major(x.k_prefix)), W.bf16_bits(x.token_major(x.v_prefix))
    ks, vs = W.bf16_bits(x.token_major(x.k_suffix)), W.bf16_bits(x.token_major(x.v_suffix))
    total_bytes, total_s, n = 0, 0.0, 0
    while total_s < budget_s and n < 64 * c.num_prompts:
        p = n % c.num_prompts
        a, lp = int(x.prefix_start[p]), int(x.prefix_len[p])
        sl = slice(p * G, (p + 1) * G)
        ls = x.suffix_len[sl]
        b0 = int(x.suffix_start[p * G])
        rows_s = int(ls.sum())
        args = (q[sl], kp[a:a + lp], vp[a:a + lp], ks[b0:b0 + rows_s], vs[b0:b0 + rows_s],
                np.array([0]), np.array([lp]), x.suffix_start[sl] - b0, ls, G, x.scale)
        t0 = time.perf_counter()
        oracle.decode_attn(*args)
        total_s += time.perf_counter() - t0
        total_bytes += (2 * 2 * c.head_dim * c.num_kv_heads * (lp + rows_s)
                        + 2 * 2 * G * c.num_q_heads * c.head_dim + 4 * G * c.num_q_heads)
        n += 1
    # the oracle spreads a call over (candidate, query head) pairs
    cores = min(oracle.num_threads(), G * c.num_q_heads)
    return {"value": round(total_bytes / total_s / 1e9, 3), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "seconds": round(total_s, 3),
            "sample": f"decode attention of {n} prompt groups ({n // c.num_prompts} full passes over the "
                      f"{c.num_prompts} prompts + {n % c.num_prompts}), {G} candidates each, fp64 CPU oracle, "
                      f"{total_bytes / 1e9:.2f} GB of algorithmic KV bytes"}


def subsample_rows(R: int, n: int, seed: int = 0) -> np.ndarray:
    """n distinct rows of R, seeded, rows 0 and R - 1 included, ascending."""
    if n >= R:
        return np.arange(R)
    rng = np.random.Generator(np.random.PCG64(seed))
    mid = rng.choice(np.arange(1, R - 1), size=n - 2, replace=False)
    return np.sort(np.concatenate([[0, R - 1], mid]))


def cpu_baseline_logprob(y, budget_s: float, fixed_rows: int = 0):
    """The fp64 oracle on the host.  The oracle spreads a call over its rows,
    so each call takes as many rows as it has threads.  With fixed_rows, a
    seeded subsample of that many rows (rows 0 and R - 1 included) runs to the
    end and the full pass's time is extrapolated from it; otherwise the first
    rows run until the time budget is spent."""
    import oracle
    import workloads as W
    c = y.cfg
    w = W.bf16_bits(y.w_lm)
    threads = oracle.num_threads()
    rows = subsample_rows(c.rows, fixed_rows) if fixed_rows else np.arange(c.rows)
    total_s, n = 0.0, 0
    while n < len(rows) and (fixed_rows or total_s < budget_s):
        idx = rows[n:n + threads]
        h = W.bf16_bits(y.hidden[torch.from_numpy(idx).to(y.hidden.device)])
        t0 = time.perf_counter()
        oracle.token_logprob(h, w, y.target[torch.from_numpy(idx).to(y.target.device)].cpu().numpy(),
                             y.inv_temperature)
        total_s += time.perf_counter() - t0
        n += len(idx)
    flops = 2 * n * c.hidden * c.vocab
    res = {"value": round(flops / total_s / 1e12, 5), "unit": "TFLOP/s", "cores": min(threads, n),
           "kind": "oracle", "seconds": round(total_s, 3)}
    if fixed_rows:
        res["sample"] = (f"token log-prob of a seeded subsample of {n} of {c.rows} rows (rows 0 and "
                         f"{c.rows - 1} included; full vocabulary), fp64 CPU oracle, {threads} rows per call")
        res["rows_per_s"] = round(n / total_s, 3)
        res["extrapolated_full_pass_s"] = round(c.rows * total_s / n, 1)
    else:
        res["sample"] = (f"token log-prob of the first {n} of {c.rows} rows (full vocabulary), fp64 CPU "
                         f"oracle, {threads} rows per call")
    return res


class Timer:
    """Times a list of operations on one stream with HIP events, medians over
    `steps` repetitions after `warmup`, each operation behind an eviction
    write (outside its events)."""

    def __init__(self, hip, stream, evict):
        self.hip, self.sh, self.evict = hip, stream.cuda_stream, evict

    def run(self, ops, steps: int, warmup: int):
        for _ in range(warmup):
            for _, f in ops:
                self.evict()
                f()
        torch.cuda.synchronize()
        hip, sh = self.hip, self.sh
        ev = [[(hip.create(), hip.create()) for _ in ops] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(steps):
            for j, (name, f) in enumerate(ops):
                self.evict()
                hip.record(ev[k][j][0], sh)
                f()
                hip.record(ev[k][j][1], sh)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = {name: np.array([hip.elapsed_ms(*ev[k][j]) for k in range(steps)]) for j, (name, _) in enumerate(ops)}
        for pair in (p for row in ev for p in row):
            for e in pair:
                hip.destroy(e)
        # the host side of one call with the GPU idle: marshalling, planning
        # and the launches (in the loop above the host runs ahead of the GPU)
        host = {name: [] for name, _ in ops}
        for _ in range(min(steps, 10)):
            for name, f in ops:
                torch.cuda.synchronize()
                h0 = time.perf_counter()
                f()
                host[name].append(time.perf_counter() - h0)
        torch.cuda.synchronize()
        return {"ms": {n: float(np.median(v)) for n, v in ms.items()},
                "p10_p90": {n: [round(float(np.percentile(v, 10)), 4), round(float(np.percentile(v, 90)), 4)]
                            for n, v in ms.items()},
                "host_us": {n: round(float(np.median(v)) * 1e6, 1) for n, v in host.items()},
                "wall_s": wall}


def decode_setup(rk, x, kv_layout, dev):
    c = x.cfg
    out = torch.empty((c.num_seqs, c.num_q_heads, c.head_dim), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((c.num_seqs, c.num_q_heads), dtype=torch.float32, device=dev)
    rdim = 1 if kv_layout == "head" else 0
    need = rk.decode_attn_workspace_size(c.num_prompts, c.group_size, c.num_q_heads, c.num_kv_heads,
                                         c.head_dim, x.prefix_start, x.prefix_len, x.suffix_start,
                                         x.suffix_len, x.k_prefix.shape[rdim], x.k_suffix.shape[rdim],
                                         x.scale, kv_layout=kv_layout)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)

    def run():
        rk.decode_attn(x.q, x.k_prefix, x.v_prefix, x.k_suffix, x.v_suffix, x.prefix_start,
                       x.prefix_len, x.suffix_start, x.suffix_len, c.group_size, scale=x.scale,
                       out=out, lse=lse, workspace=ws, return_lse=True, kv_layout=kv_layout)
    return run


def logprob_setup(rk, y, dev):
    cl = y.cfg
    lp = torch.empty(cl.rows, dtype=torch.float32, device=dev)
    lse = torch.empty(cl.rows, dtype=torch.float32, device=dev)
    ws = torch.empty(rk.token_logprob_workspace_size(cl.rows, cl.hidden, cl.vocab), dtype=torch.uint8, device=dev)

    def run():
        rk.token_logprob(y.hidden, y.w_lm, y.target, y.inv_temperature, logprob=lp, lse=lse, workspace=ws)
    return run, lse


def decode_entry(x, ms, workload):
    nbytes = decode_bytes(x)
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"kernel": "decode attention (work-list fetch + split + combine kernels)", "bound": "hbm",
            "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic("decode", workload), "algorithmic_bytes": nbytes}


def lmhead_entry(cfg, ms, workload):
    """The bound is the resource whose peak allows the longer time: MFMA at
    the 8B-class and policy shapes, HBM (the weights) at 256 rows."""
    fl = lmhead_flops(cfg)
    nb = lmhead_bytes(cfg)
    tf = fl / (ms * 1e-3) / 1e12
    e = {"kernel": "lm-head log-prob (tile + combine kernels)"}
    if nb / (HBM_PEAK_GBS * 1e9) > fl / (MFMA_BF16_PEAK_TFLOPS * 1e12):
        gbs = nb / (ms * 1e-3) / 1e9
        e.update({"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                  "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic("lmhead", workload),
                  "algorithmic_bytes": nb, "tflops": round(tf, 1),
                  "mfma_frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)})
    else:
        e.update({"bound": "mfma", "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                  "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": measured_traffic("lmhead", workload),
                  "algorithmic_flops": fl})
    return e


def measure_workload(rk, W, name, args, timer, dev, steps, warmup, cpu_budget, keep=False):
    """Times one workload's operations and builds its report; with keep, also
    returns its inputs for the extra operations."""
    dname, lname, desc = WORKLOADS[name]
    x = W.make_decode_inputs(W.DECODE_CONFIGS[dname], dev, kv_layout=args.kv_layout) if dname else None
    y = W.make_logprob_inputs(W.LOGPROB_CONFIGS[lname], dev) if lname else None
    ops, lse_l = [], None
    if x is not None:
        ops.append(("decode", decode_setup(rk, x, args.kv_layout, dev)))
    if y is not None:
        run_l, lse_l = logprob_setup(rk, y, dev)
        ops.append(("lmhead", run_l))
    log(f"bench: workload {name}: warmup {warmup}, timing {steps} steps")
    t = timer.run(ops, steps, warmup)
    log(f"bench: {name}: per op {t['ms']} ms, host {t['host_us']} us")
    rep = {"workload": desc, "steps": steps, "ms_per_step": round(t["wall_s"] * 1e3 / steps, 4),
           "ops": {}}
    entries = []
    if x is not None:
        e = decode_entry(x, t["ms"]["decode"], name)
        rep["ops"]["decode"] = {"ms": round(t["ms"]["decode"], 4), "ms_p10_p90": t["p10_p90"]["decode"],
                                "host_us": t["host_us"]["decode"], "roofline": e}
        entries.append((t["ms"]["decode"], e))
    if y is not None:
        e = lmhead_entry(y.cfg, t["ms"]["lmhead"], name)
        rep["ops"]["lmhead"] = {"ms": round(t["ms"]["lmhead"], 4), "ms_p10_p90": t["p10_p90"]["lmhead"],
                                "host_us": t["host_us"]["lmhead"], "roofline": e}
        entries.append((t["ms"]["lmhead"], e))
    entries.sort(key=lambda p: -p[0])
    rep["roofline"] = entries[0][1]
    if cpu_budget > 0:
        log(f"bench: {name}: cpu baseline (fp64 oracle)")
        if x is not None:
            rep["ops"]["decode"]["cpu_baseline"] = cpu_baseline_decode(x, cpu_budget)
        if y is not None:
            fixed = 1024 if y.cfg.rows > 65536 else 0
            rep["ops"]["lmhead"]["cpu_baseline"] = cpu_baseline_logprob(y, cpu_budget, fixed_rows=fixed)
        rep["cpu_baseline"] = rep["ops"]["decode" if x is not None else "lmhead"]["cpu_baseline"]
    if keep:
        return rep, t, (x, y, ops, lse_l)
    del x, y, ops
    torch.cuda.empty_cache()
    return rep, t, None


def extra_ops(rk, W, args, x, y, lse2, ops, hip, sh, dev):
    """The operations timed after the headline's steps at its shape."""
    update = None
    if x is not None and not args.no_update:
        # the decode loop's cache update: one new token per candidate appended
        # in place after its suffix (a cache with 16 free rows per candidate)
        c = x.cfg
        S = c.num_seqs
        kn = torch.randn((S, c.num_kv_heads, c.head_dim), device=dev).to(torch.bfloat16)
        vn = torch.randn_like(kn)
        cshape = (c.num_kv_heads, S * 16, c.head_dim) if args.kv_layout == "head" else (S * 16, c.num_kv_heads,
                                                                                       c.head_dim)
        kc = torch.zeros(cshape, dtype=torch.bfloat16, device=dev)
        vc = torch.zeros_like(kc)
        a_ss, a_sl = np.arange(S, dtype=np.int64) * 16, np.zeros(S, np.int32)
        a_ns, a_nl = np.arange(S, dtype=np.int64), np.ones(S, np.int32)
        ws_a = torch.empty(max(256, 16 * S + 256), dtype=torch.uint8, device=dev)
        run_append = lambda: rk.kv_append(kn, vn, kc, vc, a_ss, a_sl, a_ns, a_nl, c.group_size,
                                          kv_layout=args.kv_layout, workspace=ws_a)
        for _ in range(3):
            run_append()
        torch.cuda.synchronize()
        # each timed append follows a decode call, as in a rollout loop: the
        # host enqueues the append while the GPU still runs the decode, so the
        # events bracket the append's GPU time and not the host's argument
        # marshalling in front of an idle GPU
        aev = [(hip.create(), hip.create()) for _ in range(args.steps)]
        for e0, e1 in aev:
            ops[0][1]()
            hip.record(e0, sh)
            run_append()
            hip.record(e1, sh)
        torch.cuda.synchronize()
        a_ms = float(np.mean([hip.elapsed_ms(e0, e1) for e0, e1 in aev]))
        for pair in aev:
            for e in pair:
                hip.destroy(e)
        nb_a = 2 * 2 * (2 * S * c.num_kv_heads * c.head_dim)      # K and V, read and written
        update = {"kv_append": {"kernel": "KV append, one token per candidate (fetch + copy kernels), timed "
                                          "behind a decode call",
                                "us": round(a_ms * 1e3, 2), "bound": "hbm",
                                "achieved": round(nb_a / (a_ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                                "unit": "GB/s", "algorithmic_bytes": nb_a}}
        del kc, vc
    if x is not None and not args.no_extend:
        c = x.cfg
        # a refinement turn's extend at the same shape: every candidate's whole
        # suffix is new and is read causally against the shared prefix
        xe = W.make_extend_inputs(c, dev, kv_layout=args.kv_layout)
        de = xe.dec
        e_out = torch.empty(xe.q.shape, dtype=torch.bfloat16, device=dev)
        e_lse = torch.empty(xe.q.shape[:2], dtype=torch.float32, device=dev)
        rdim = 1 if args.kv_layout == "head" else 0
        ws_e = torch.empty(max(256, rk.extend_attn_workspace_size(
            c.num_prompts, c.group_size, c.num_q_heads, c.num_kv_heads, c.head_dim, de.prefix_start,
            de.prefix_len, de.suffix_start, de.suffix_len, xe.new_len, xe.q_start, de.k_prefix.shape[rdim],
            de.k_suffix.shape[rdim], xe.q.shape[0], de.scale, kv_layout=args.kv_layout)),
            dtype=torch.uint8, device=dev)
        run_extend = lambda: rk.extend_attn(xe.q, de.k_prefix, de.v_prefix, de.k_suffix, de.v_suffix,
                                            de.prefix_start, de.prefix_len, de.suffix_start, de.suffix_len,
                                            xe.new_len, xe.q_start, c.group_size, scale=de.scale, out=e_out,
                                            lse=e_lse, workspace=ws_e, return_lse=True, kv_layout=args.kv_layout)
        run_extend()
        torch.cuda.synchronize()
        esteps = max(1, min(args.steps, 5))
        eev = [(hip.create(), hip.create()) for _ in range(esteps)]
        for e0, e1 in eev:
            hip.record(e0, sh)
            run_extend()
            hip.record(e1, sh)
        torch.cuda.synchronize()
        e_ms = float(np.mean([hip.elapsed_ms(e0, e1) for e0, e1 in eev]))
        for pair in eev:
            for e in pair:
                hip.destroy(e)
        fl_e = extend_flops(xe)
        tf_e = fl_e / (e_ms * 1e-3) / 1e12
        log(f"bench: extend {e_ms:.3f} ms, {tf_e:.1f} TFLOP/s")
        update = dict(update or {})
        update["extend"] = {"kernel": "extend (prefill) attention of a refinement turn, every suffix token new "
                                      f"({int(xe.new_len.sum())} tokens)", "ms": round(e_ms, 4), "steps": esteps,
                            "bound": "mfma", "achieved": round(tf_e, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                            "unit": "TFLOP/s", "frac": round(tf_e / MFMA_BF16_PEAK_TFLOPS, 4),
                            "algorithmic_flops": fl_e}
        del xe, de, e_out, e_lse, ws_e
    if y is not None and not args.no_update:
        cl = y.cfg
        g_b = torch.from_numpy(np.random.Generator(np.random.PCG64(5)).standard_normal(cl.rows)
                               .astype(np.float32)).to(dev)
        dh = torch.empty((cl.rows, cl.hidden), dtype=torch.float32, device=dev)
        ws_b = torch.empty(max(1, rk.token_logprob_backward_workspace_size(cl.rows, cl.hidden, cl.vocab)),
                           dtype=torch.uint8, device=dev)
        gx = W.make_grpo_inputs(W.GRPO_CONFIGS["policy"], dev)
        G = gx.cfg.group_size
        adv = rk.grpo_advantage(gx.reward, G)
        gl = torch.empty(1, dtype=torch.float32, device=dev)
        gg = torch.empty_like(gx.logp_new)
        ws_g = torch.empty(rk.grpo_surrogate_workspace_size(gx.seq.numel(), adv.numel() // G, G),
                           dtype=torch.uint8, device=dev)
        uops = [("backward", lambda: rk.token_logprob_backward(y.hidden, y.w_lm, y.target, lse2, g_b,
                                                               y.inv_temperature, grad_hidden=dh,
                                                               workspace=ws_b)),
                ("grpo", lambda: (rk.grpo_advantage(gx.reward, G, adv=adv),
                                  rk.grpo_surrogate(gx.logp_new, gx.logp_old, gx.seq, adv, G, gx.eps,
                                                    loss=gl, grad=gg, workspace=ws_g)))]
        sx = None
        if cl.rows <= 65536:
            # the sampling head at the decode step's shape: rows alternate
            # between the two temperatures, nucleus p = 0.9
            sx = W.make_sample_inputs(cl, dev)
            s_tok = torch.empty(cl.rows, dtype=torch.int32, device=dev)
            s_lp = torch.empty(cl.rows, dtype=torch.float32, device=dev)
            ws_s = torch.empty(rk.sample_top_p_workspace_size(cl.rows, cl.hidden, cl.vocab), dtype=torch.uint8,
                               device=dev)
            uops.append(("sample", lambda: rk.sample_top_p(sx.hidden, sx.w_lm, sx.inv_temperature, sx.top_p,
                                                           sx.uniform, token=s_tok, logprob=s_lp,
                                                           workspace=ws_s)))
        usteps = max(1, min(args.steps, 3 if cl.rows > 65536 else args.steps))
        for _, f in uops:
            f()
        torch.cuda.synchronize()
        uev = [[(hip.create(), hip.create()) for _ in uops] for _ in range(usteps)]
        for k in range(usteps):
            for j, (_, f) in enumerate(uops):
                hip.record(uev[k][j][0], sh)
                f()
                hip.record(uev[k][j][1], sh)
        torch.cuda.synchronize()
        u_ms = {name: float(np.mean([hip.elapsed_ms(*uev[k][j]) for k in range(usteps)]))
                for j, (name, _) in enumerate(uops)}
        for pair in (p for row in uev for p in row):
            for e in pair:
                hip.destroy(e)
        log(f"bench: policy update per op {u_ms}")
        fl_b = 4 * cl.rows * cl.hidden * cl.vocab
        tf_b = fl_b / (u_ms["backward"] * 1e-3) / 1e12
        nb_g = grpo_bytes(gx)
        update = dict(update or {})
        update.update({"steps": usteps,
                       "lmhead_backward": {"kernel": "log-prob backward (probability tile + vocab GEMM + finish "
                                                     "kernels, per 16384-row chunk)",
                                           "ms": round(u_ms["backward"], 4), "bound": "mfma",
                                           "achieved": round(tf_b, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                                           "unit": "TFLOP/s", "frac": round(tf_b / MFMA_BF16_PEAK_TFLOPS, 4),
                                           "algorithmic_flops": fl_b},
                       "grpo": {"kernel": "GRPO advantages + clipped surrogate, 4 x G=16 sequences x 4096 rows",
                                "us": round(u_ms["grpo"] * 1e3, 2), "bound": "hbm",
                                "achieved": round(nb_g / (u_ms["grpo"] * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                                "unit": "GB/s", "algorithmic_bytes": nb_g}})
        if sx is not None:
            fl_s = lmhead_flops(cl)
            tf_s = fl_s / (u_ms["sample"] * 1e-3) / 1e12
            update["sampling_head"] = {
                "kernel": "nucleus sampling head (logits tile + per-row selection kernels), T in {0.2, 0.7}, "
                          "top-p 0.9", "ms": round(u_ms["sample"], 4), "bound": "mfma",
                "achieved": round(tf_s, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf_s / MFMA_BF16_PEAK_TFLOPS, 4), "algorithmic_flops": fl_s}
    return update


TIMELINE_KINDS = {0: "whole tiles", 1: "narrow tiles", 2: "tail parts"}


def provenance(op: str) -> str:
    """The command line that wrote a summary (as run from the repository
    root) and the sha256 of the kernel sources it measured."""
    argv = " ".join(["python3", "bench.py"] + [a if a else "''" for a in sys.argv[1:]])
    return (f"\nCommand (on the MI355X box, from the repository root): `{argv}`\n\n"
            f"Kernel sources: {op} sha256 {source_sha256(op)}\n")


def timeline_report(rk, y, evict, desc: str) -> str:
    """The tile launches of one lm-head call, one record per wave from
    rl_debug_logprob_timeline (after the same cache eviction as the timed
    operations), summarised as markdown."""
    plain = lambda: rk.token_logprob(y.hidden, y.w_lm, y.target, y.inv_temperature)
    stamped = lambda: rk.token_logprob_timeline(y.hidden, y.w_lm, y.target, y.inv_temperature)
    for _ in range(2):
        plain()
        stamped()
    # both entry points alternately, each call after the eviction, by events
    ms = {"plain": [], "stamped": []}
    for _ in range(5):
        for name, f in (("plain", plain), ("stamped", stamped)):
            evict()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            out = f()
            e1.record()
            torch.cuda.synchronize()
            ms[name].append(e0.elapsed_time(e1))
    lp, lse, rec = out                      # the last stamped call's
    ref_lp, ref_lse = plain()
    same = bool(torch.equal(lp, ref_lp) and torch.equal(lse, ref_lse))
    return timeline_markdown(rec.cpu().numpy(), same, 2 * y.cfg.vocab * y.cfg.hidden, desc,
                             float(np.median(ms["plain"])), float(np.median(ms["stamped"])))


def timeline_markdown(r: np.ndarray, same: bool, wbytes: int, desc: str, plain_ms: float = None,
                      stamped_ms: float = None) -> str:
    """Markdown summary of timeline records (int64 [n, 8], one per wave, the
    waves of a workgroup consecutive; word layout in rl_kernels.h); plain_ms
    and stamped_ms are the whole call's event times without and with the
    stamps."""
    hw = r[:, 0] & 0xFFFFFFFF
    wpg = int(((r[:, 0] >> 48) & 0xFF).max()) + 1    # waves per workgroup
    xcc = (r[:, 0] >> 32) & 0xFF
    kind = (r[:, 0] >> 40) & 0xFF
    t_start, t_loop0, t_loop1, t_end = (r[:, i] for i in range(1, 5))
    wait, cyc, nks = r[:, 5], r[:, 6], (r[:, 7] >> 32) & 0xFFFF
    samples = np.maximum((r[:, 7] >> 48) & 0xFFFF, 1)
    wait = wait / samples * nks          # the sampled stages' mean wait, over all stages
    # HW_ID: CU id bits 11:8, shader array bit 12, shader engine bits 15:13
    cu = xcc * 256 + ((hw >> 13) & 7) * 32 + ((hw >> 12) & 1) * 16 + ((hw >> 8) & 0xF)
    t0 = int(t_start.min())
    us = lambda t: (t - t0) * 0.01        # 100 MHz wall clock
    q = lambda v: "/".join(f"{np.percentile(v, p):.1f}" for p in (10, 50, 90))
    out = [f"# lm-head tile timeline: {desc}", "",
           "One call of rl_debug_logprob_timeline (the tile launches of rl_token_logprob with per-wave "
           "timestamps; the log-prob and lse it returned are "
           f"{'bit-identical to' if same else 'NOT identical to'} rl_token_logprob's), after a 1 GiB read that "
           "empties the caches.  Wall clock: s_memrealtime (100 MHz); cycles: s_memtime (its rate is not the shader "
           "clock's: compare the MFMA-busy counters).  Per workgroup the "
           f"earliest start and the latest end of its {wpg} waves; waits and cycles averaged over the waves.  The stage-end "
           "wait (loads of the next stage, then the barrier) is sampled in one stage of every 8.", "",
           "| launch | workgroups | stages | first start - last end (us) | tile us p10/p50/p90 | "
           "prologue us | loop us | epilogue us | ns per stage | stage-end wait share | s_memtime cycles per ns |",
           "|---|---:|---:|---|---|---|---|---|---:|---:|---:|"]
    per_kind = {}
    for k in sorted(set(kind.tolist())):
        m = kind == k
        n = int(m.sum()) // wpg
        g = lambda v: v[m].reshape(n, wpg)
        st, lo0, lo1, en = g(t_start).min(1), g(t_loop0).max(1), g(t_loop1).max(1), g(t_end).max(1)
        wt, cy, ns = g(wait).mean(1), g(cyc).mean(1), g(nks)[:, 0]
        wall_loop = (lo1 - lo0) * 10.0     # ns
        per_kind[k] = (st, en, g(cu)[:, 0], g(xcc)[:, 0])
        out.append(f"| {TIMELINE_KINDS.get(k, k)} | {n} | {int(np.median(ns))} | {us(st.min()):.1f} - {us(en.max()):.1f} "
                   f"| {q((en - st) * 0.01)} | {q((lo0 - st) * 0.01)} | {q((lo1 - lo0) * 0.01)} "
                   f"| {q((en - lo1) * 0.01)} | {np.median(wall_loop / ns):.0f} | {np.median(wt / cy):.3f} "
                   f"| {np.median(cy / wall_loop):.3f} |")
    out += ["", "Per CU (XCD, shader engine, CU): workgroups run one after another; the gap is the time from one "
            "workgroup's end to the next one's start on the same CU, the idle tail the time from a CU's last end "
            "to the launch's last end.", "",
            "| launch | CUs used | workgroups per CU | gap us p10/p50/p90 | idle tail us p10/p50/p90 | "
            "last end per XCD (us) |", "|---|---:|---|---|---|---|"]
    for k, (st, en, c, x) in per_kind.items():
        gaps, tails, counts = [], [], []
        for cid in np.unique(c):
            o = np.argsort(st[c == cid])
            s1, e1 = st[c == cid][o], en[c == cid][o]
            counts.append(len(o))
            gaps += ((s1[1:] - e1[:-1]) * 0.01).tolist()
            tails.append((en.max() - e1[-1]) * 0.01)
        xe = " ".join(f"{us(en[x == i].max()):.0f}" for i in range(8) if (x == i).any())
        hist = {v: counts.count(v) for v in sorted(set(counts))}
        out.append(f"| {TIMELINE_KINDS.get(k, k)} | {len(counts)} | "
                   f"{', '.join(f'{v}: {c_} CUs' for v, c_ in hist.items())} | {q(np.array(gaps)) if gaps else '-'} "
                   f"| {q(np.array(tails))} | {xe} |")
    span = us(t_end.max())
    out += ["", f"All tile launches: {span:.1f} us from the first start to the last end; the weights "
            f"({wbytes / 1e9:.3f} GB) over that span stream at {wbytes / (span * 1e-6) / 1e9:.0f} GB/s."]
    if plain_ms is not None:
        out += ["", f"Whole call by events (medians of 5, each after the eviction; both entry points "
                f"alternately): rl_token_logprob {plain_ms * 1e3:.1f} us, rl_debug_logprob_timeline "
                f"{stamped_ms * 1e3:.1f} us."]
    return "\n".join(out) + "\n"


def decode_timeline_report(rk, x, evict, kv_layout: str, desc: str) -> str:
    """The split kernel of one decode-attention call, one record per work item
    from rl_debug_decode_timeline (after the same cache eviction as the timed
    operations), summarised as markdown."""
    c = x.cfg
    args = (x.q, x.k_prefix, x.v_prefix, x.k_suffix, x.v_suffix, x.prefix_start, x.prefix_len, x.suffix_start,
            x.suffix_len, c.group_size)
    plain = lambda: rk.decode_attn(*args, scale=x.scale, return_lse=True, kv_layout=kv_layout)
    stamped = lambda: rk.decode_attn_timeline(*args, scale=x.scale, kv_layout=kv_layout)
    for _ in range(2):
        plain()
        stamped()
    ms = {"plain": [], "stamped": []}
    for _ in range(5):
        for name, f in (("plain", plain), ("stamped", stamped)):
            evict()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            res = f()
            e1.record()
            torch.cuda.synchronize()
            ms[name].append(e0.elapsed_time(e1))
    o, l, rec = res                         # the last stamped call's
    ro, rl = plain()
    same = bool(torch.equal(o.view(torch.int16), ro.view(torch.int16)) and torch.equal(l, rl))
    return decode_timeline_markdown(rec.cpu().numpy(), same, 4 * c.head_dim, decode_bytes(x), desc,
                                    float(np.median(ms["plain"])), float(np.median(ms["stamped"])))


def decode_timeline_markdown(r: np.ndarray, same: bool, token_bytes: int, alg_bytes: int, desc: str,
                             plain_ms: float = None, stamped_ms: float = None) -> str:
    """Markdown summary of decode timeline records (int64 [n, 8], one per work
    item; word layout in rl_kernels.h).  token_bytes: K and V bytes of one
    token at one kv head; alg_bytes: the call's algorithmic bytes."""
    hw = r[:, 0] & 0xFFFFFFFF
    xcc = (r[:, 0] >> 32) & 0xFF
    kind = (r[:, 0] >> 40) & 0xFF
    rows = (r[:, 0] >> 48) & 0xFFFF
    st, first, loop1, en = (r[:, i] for i in range(1, 5))
    ntok, tiles = r[:, 5] & 0xFFFFFFFF, r[:, 5] >> 32
    cu = xcc * 256 + ((hw >> 13) & 7) * 32 + ((hw >> 12) & 1) * 16 + ((hw >> 8) & 0xF)
    t0 = int(st.min())
    span = (int(en.max()) - t0) * 0.01
    q = lambda v: "/".join(f"{np.percentile(v, p):.1f}" for p in (10, 50, 90)) if len(v) else "-"
    out = [f"# Decode split kernel timeline: {desc}", "",
           "One call of rl_debug_decode_timeline (rl_decode_attn with the split kernel built to leave one "
           "record per work item; the output and lse it returned are "
           f"{'bit-identical to' if same else 'NOT identical to'} rl_decode_attn's), after a 1 GiB read that "
           "empties the caches.  Wall clock: s_memrealtime (100 MHz).  The work list runs in its planned order "
           "(longest items first).", "",
           "| items | query rows | count | KV tokens p10/p50/p90 | item us p10/p50/p90 | first tile us | "
           "ns per 64-token tile | partials us | KV GB |",
           "|---|---:|---:|---|---|---|---:|---|---:|"]
    for k, name in ((0, "prefix"), (1, "suffix")):
        m = kind == k
        if not m.any():
            continue
        for rr in np.unique(rows[m]):
            mm = m & (rows == rr)
            loop_ns = (loop1[mm] - first[mm]) * 10.0
            out.append(f"| {name} | {rr} | {int(mm.sum())} | {q(ntok[mm])} | {q((en[mm] - st[mm]) * 0.01)} | "
                       f"{q((first[mm] - st[mm]) * 0.01)} | {np.median(loop_ns / np.maximum(tiles[mm], 1)):.0f} | "
                       f"{q((en[mm] - loop1[mm]) * 0.01)} | {ntok[mm].sum() * token_bytes / 1e9:.3f} |")
    # occupancy: items resident per CU over the span
    ncu = len(np.unique(cu))
    busy = (en - st).sum() * 0.01
    events = np.concatenate([np.stack([st, np.ones_like(st)], 1), np.stack([en, -np.ones_like(en)], 1)])
    events = events[np.lexsort((events[:, 1], events[:, 0]))]
    resident = np.cumsum(events[:, 1])
    times = (events[:, 0] - t0) * 0.01
    # the last moment every CU still holds an item, from the per-CU last ends
    cu_last = np.array([en[cu == c].max() for c in np.unique(cu)])
    tails = (en.max() - cu_last) * 0.01
    peak = int(resident.max())
    out += ["", f"Span (first start to last end): {span:.1f} us over {ncu} CUs; the algorithmic "
            f"{alg_bytes / 1e9:.3f} GB over the span stream at {alg_bytes / (span * 1e-6) / 1e9:.0f} GB/s.  "
            f"Items resident at once: at most {peak} ({peak / ncu:.2f} per CU), on average "
            f"{busy / span / ncu:.2f} per CU.  The last item starts at {(st.max() - t0) * 0.01:.1f} us; "
            f"the CUs' idle tails (a CU's last end to the kernel's) are {q(tails)} us (p10/p50/p90).  "
            f"Last end per XCD (us): "
            + " ".join(f"{(en[xcc == i].max() - t0) * 0.01:.0f}" for i in range(8) if (xcc == i).any()) + "."]
    late = int(np.argmax(en))
    out += ["", f"The item that ends last: {'suffix' if kind[late] else 'prefix'}, {rows[late]} rows, "
            f"{ntok[late]} tokens, started at {(st[late] - t0) * 0.01:.1f} us and took "
            f"{(en[late] - st[late]) * 0.01:.1f} us."]
    if plain_ms is not None:
        out += ["", f"Whole call by events (medians of 5, each after the eviction; both entry points "
                f"alternately): rl_decode_attn {plain_ms * 1e3:.1f} us, rl_debug_decode_timeline "
                f"{stamped_ms * 1e3:.1f} us."]
    return "\n".join(out) + "\n"


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="32b", choices=sorted(WORKLOADS),
                    help="the headline workload (value, roofline, extra operations)")
    ap.add_argument("--also", default="8b,longctx,policy",
                    help="comma-separated workloads measured after the headline, reported under configs "
                         "('' for none)")
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="seconds of oracle time per headline operation for the CPU baseline (0 to skip); "
                         "the other workloads get half")
    ap.add_argument("--kv-layout", default="head", choices=["head", "token"],
                    help="KV cache layout: head-major [Hkv, rows, D] (default) or token-major [rows, Hkv, D]")
    ap.add_argument("--evict-mb", type=int, default=1024,
                    help="MiB read before every timed operation, outside its events (0: none)")
    ap.add_argument("--no-update", action="store_true",
                    help="skip the policy-update operations (log-prob backward, GRPO surrogate, sampling head), "
                         "which are timed after the step in a loop of their own")
    ap.add_argument("--no-extend", action="store_true",
                    help="skip the extend (prefill) of a refinement turn, timed after the step")
    ap.add_argument("--timeline", default="",
                    help="write a markdown summary of the headline lm-head's tile launches (per-wave timestamps "
                         "from rl_debug_logprob_timeline) to this file")
    ap.add_argument("--decode-timeline", default="",
                    help="write a markdown summary of the headline decode attention's split kernel (one record per "
                         "work item from rl_debug_decode_timeline) to this file")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one 1 GiB device copy before the steps (outside the timed region) so a "
                         "rocprofv3 --pmc run can scale FETCH_SIZE / WRITE_SIZE against known bytes")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library runs the hot path on a single MI355X "
              "and has no multi-GPU path; run it without --gpus or with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    also = [w for w in args.also.split(",") if w and w != args.workload]
    for w in also:
        if w not in WORKLOADS:
            sys.exit(f"unknown workload {w}")

    import paper_2607_20908_amd as rk
    import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    evict_buf = torch.zeros((max(1, args.evict_mb) << 20) // 4, dtype=torch.float32, device=dev) \
        if args.evict_mb else None

    def evict():
        if evict_buf is not None:
            torch.amax(evict_buf)             # a read of the whole buffer; the result is not used
    if args.copy_calibration:
        src = torch.ones(1 << 29, dtype=torch.bfloat16, device=dev)      # 1 GiB
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    runtimes = rk.hip_runtimes_mapped()
    if len(runtimes) != 1:
        raise RuntimeError(f"expected one HIP runtime in the process, found {runtimes}")
    hip = HipEvents(runtimes[0])
    timer = Timer(hip, stream, evict)

    head, t, (x, y, ops, lse2) = measure_workload(rk, W, args.workload, args, timer, dev, args.steps, args.warmup,
                                                  args.cpu_budget, keep=True)
    if args.decode_timeline and x is not None:
        with open(args.decode_timeline, "w") as f:
            f.write(decode_timeline_report(rk, x, evict, args.kv_layout, head["workload"]))
            f.write(provenance("decode"))
        log(f"bench: decode timeline written to {args.decode_timeline}")
    if args.timeline and y is not None:
        with open(args.timeline, "w") as f:
            f.write(timeline_report(rk, y, evict, head["workload"]))
            f.write(provenance("lmhead"))
        log(f"bench: tile timeline written to {args.timeline}")
    update = extra_ops(rk, W, args, x, y, lse2, ops, hip, stream.cuda_stream, dev)
    del x, y, ops, lse2
    torch.cuda.empty_cache()
    configs = {args.workload: head}
    for w in also:
        steps = min(args.steps, 5) if w == "policy" else args.steps
        rep, _, _ = measure_workload(rk, W, w, args, timer, dev, steps, min(args.warmup, 2) if w == "policy"
                                     else args.warmup, args.cpu_budget / 2)
        configs[w] = rep

    hops = head["ops"]
    both = "decode" in hops and "lmhead" in hops
    res = {"metric": "decode-attn effective KV GB/s (% HBM peak); lm-head logprob TFLOP/s (% MFMA)" if both else
           ("decode-attn effective KV GB/s (% HBM peak)" if "decode" in hops else "lm-head logprob TFLOP/s (% MFMA)"),
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": head["ms_per_step"], "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded, HBM-resident)",
           "config": {"workload": head["workload"], "kv_layout": args.kv_layout if "decode" in hops else None,
                      "evict_mib_between_ops": args.evict_mb}}
    if "decode" in hops:
        d = hops["decode"]
        res.update({"value": d["roofline"]["achieved"], "unit": "GB/s", "decode_ms": d["ms"],
                    "decode_ms_p10_p90": d["ms_p10_p90"], "decode_host_us": d["host_us"],
                    "decode_hbm_frac": d["roofline"]["frac"],
                    "decode_algorithmic_bytes": d["roofline"]["algorithmic_bytes"]})
    if "lmhead" in hops:
        l = hops["lmhead"]
        fl = lmhead_flops(W.LOGPROB_CONFIGS[WORKLOADS[args.workload][1]])
        tf = fl / (l["ms"] * 1e-3) / 1e12
        res.update({"lmhead_ms": l["ms"], "lmhead_ms_p10_p90": l["ms_p10_p90"], "lmhead_host_us": l["host_us"],
                    "lmhead_tflops": round(tf, 1), "lmhead_mfma_frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
                    "lmhead_flops": fl})
        if "decode" not in hops:
            res.update({"value": round(tf, 1), "unit": "TFLOP/s"})
    res["roofline"] = head["roofline"]
    other = [o["roofline"] for n, o in hops.items() if o["roofline"] is not head["roofline"]]
    if other:
        res["roofline_other"] = other[0]
    if "cpu_baseline" in head:
        res["cpu_baseline"] = head["cpu_baseline"]
        if both:
            res["cpu_baseline_lmhead"] = hops["lmhead"]["cpu_baseline"]
    if update is not None:
        res["extra_ops"] = update
    res["configs"] = configs
    order = ["metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
             "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"]
    line = {k: res[k] for k in order if k in res}
    line.update({k: v for k, v in res.items() if k not in line})
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
