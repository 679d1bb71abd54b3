#!/usr/bin/env python3
"""Throughput of the rollout hot path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input that is
already resident in HBM: prefix-shared decode attention for all candidates of
the batch, then the fused lm-head token log-prob of their rows.  The default
workload is the 8B-class single-layer decode step (64 prompts x G=8, 32 query
/ 8 kv heads, head dim 128, shared prefix 1024, suffix lengths uniform in
[256, 2048]; lm-head 512 rows x hidden 4096 x vocab 151936).

After the timed steps, further operations are timed in a loop of their own
(outside the step): the KV append of one token per candidate, the extend
(prefill) of a refinement turn at the same shape with every suffix token new,
the backward
of the lm-head log-prob for the same rows,
the GRPO advantages and clipped surrogate over the policy pass's 262144 rows,
and (at decode shapes) the nucleus sampling head over the same rows.  They
are reported under "extra_ops".

Prints ONE JSON line.  `value` is decode attention's effective KV bandwidth
(algorithmic bytes, the prefix counted once per prompt, over the measured
decode time); the lm-head's TFLOP/s are reported beside it.  Per-operation
durations come from HIP events recorded on the stream the kernels run on
(created with a device-scope release, so recording one does not write back the
L2 to system memory and the interval matches the kernels' own durations).
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


def source_sha256(op: str) -> str:
    import hashlib
    with open(os.path.join(CSRC, KERNEL_SOURCES[op]), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


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
    return {"value": round(total_bytes / total_s / 1e9, 3), "unit": "GB/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": round(total_s, 3),
            "sample": f"decode attention of {n} prompt groups ({n // c.num_prompts} full passes over the "
                      f"{c.num_prompts} prompts + {n % c.num_prompts}), {G} candidates each, fp64 CPU oracle, "
                      f"{total_bytes / 1e9:.2f} GB of algorithmic KV bytes"}


def cpu_baseline_logprob(y, budget_s: float):
    """The fp64 oracle on the host over the first rows of the workload, two rows
    at a time, until the time budget is spent."""
    import oracle
    import workloads as W
    c = y.cfg
    w = W.bf16_bits(y.w_lm)
    total_s, n = 0.0, 0
    rows_per = 2
    while n < c.rows and total_s < budget_s:
        idx = slice(n, min(c.rows, n + rows_per))
        t0 = time.perf_counter()
        oracle.token_logprob(W.bf16_bits(y.hidden[idx]), w, y.target[idx].cpu().numpy(), y.inv_temperature)
        total_s += time.perf_counter() - t0
        n = idx.stop
    flops = 2 * n * c.hidden * c.vocab
    return {"value": round(flops / total_s / 1e12, 5), "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": round(total_s, 3),
            "sample": f"token log-prob of the first {n} of {c.rows} rows (full vocabulary), fp64 CPU oracle"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="8b", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="seconds of oracle time per operation for the CPU baseline (0 to skip)")
    ap.add_argument("--kv-layout", default="head", choices=["head", "token"],
                    help="KV cache layout: head-major [Hkv, rows, D] (default) or token-major [rows, Hkv, D]")
    ap.add_argument("--no-update", action="store_true",
                    help="skip the policy-update operations (log-prob backward, GRPO surrogate), which "
                         "are timed after the step in a loop of their own")
    ap.add_argument("--no-extend", action="store_true",
                    help="skip the extend (prefill) of a refinement turn, timed after the step")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one 1 GiB device copy before the steps (outside the timed region) so a "
                         "rocprofv3 --pmc run can scale FETCH_SIZE / WRITE_SIZE against known bytes")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library runs the hot path on a single MI355X "
              "and has no multi-GPU path; run it without --gpus or with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import paper_2607_20908_amd as rk
    import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dname, lname, desc = WORKLOADS[args.workload]
    x = W.make_decode_inputs(W.DECODE_CONFIGS[dname], dev, kv_layout=args.kv_layout) if dname else None
    y = W.make_logprob_inputs(W.LOGPROB_CONFIGS[lname], dev) if lname else None

    ops = []
    if x is not None:
        c = x.cfg
        out = torch.empty((c.num_seqs, c.num_q_heads, c.head_dim), dtype=torch.bfloat16, device=dev)
        lse = torch.empty((c.num_seqs, c.num_q_heads), dtype=torch.float32, device=dev)
        rdim = 1 if args.kv_layout == "head" else 0
        need = rk.decode_attn_workspace_size(c.num_prompts, c.group_size, c.num_q_heads, c.num_kv_heads,
                                             c.head_dim, x.prefix_start, x.prefix_len, x.suffix_start,
                                             x.suffix_len, x.k_prefix.shape[rdim], x.k_suffix.shape[rdim],
                                             x.scale, kv_layout=args.kv_layout)
        ws_d = torch.empty(need, dtype=torch.uint8, device=dev)

        def run_decode():
            rk.decode_attn(x.q, x.k_prefix, x.v_prefix, x.k_suffix, x.v_suffix, x.prefix_start,
                           x.prefix_len, x.suffix_start, x.suffix_len, c.group_size, scale=x.scale,
                           out=out, lse=lse, workspace=ws_d, return_lse=True, kv_layout=args.kv_layout)
        ops.append(("decode", run_decode))
    if y is not None:
        cl = y.cfg
        lp = torch.empty(cl.rows, dtype=torch.float32, device=dev)
        lse2 = torch.empty(cl.rows, dtype=torch.float32, device=dev)
        ws_l = torch.empty(rk.token_logprob_workspace_size(cl.rows, cl.hidden, cl.vocab),
                           dtype=torch.uint8, device=dev)

        def run_logprob():
            rk.token_logprob(y.hidden, y.w_lm, y.target, y.inv_temperature, logprob=lp, lse=lse2,
                             workspace=ws_l)
        ops.append(("lmhead", run_logprob))

    stream = torch.cuda.current_stream()
    if args.copy_calibration:
        src = torch.ones(1 << 29, dtype=torch.bfloat16, device=dev)      # 1 GiB
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    log(f"bench: workload {args.workload}: warmup {args.warmup}")
    for _ in range(args.warmup):
        for _, f in ops:
            f()
    torch.cuda.synchronize()
    runtimes = rk.hip_runtimes_mapped()
    if len(runtimes) != 1:
        raise RuntimeError(f"expected one HIP runtime in the process, found {runtimes}")
    hip = HipEvents(runtimes[0])
    sh = stream.cuda_stream
    ev = [[(hip.create(), hip.create()) for _ in ops] for _ in range(args.steps)]
    log(f"bench: timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        for j, (_, f) in enumerate(ops):
            hip.record(ev[k][j][0], sh)
            f()
            hip.record(ev[k][j][1], sh)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # per-operation duration: the median over the timed steps (p10 and p90
    # reported beside it).  The first step's interval also holds the host's
    # planning of that call, since the GPU has drained before the timed region.
    op_all = {name: np.array([hip.elapsed_ms(*ev[k][j]) for k in range(args.steps)])
              for j, (name, _) in enumerate(ops)}
    op_ms = {name: float(np.median(v)) for name, v in op_all.items()}
    op_pct = {name: [round(float(np.percentile(v, 10)), 4), round(float(np.percentile(v, 90)), 4)]
              for name, v in op_all.items()}
    for pair in (p for row in ev for p in row):
        for e in pair:
            hip.destroy(e)
    ms_per_step = wall * 1e3 / args.steps
    log(f"bench: {ms_per_step:.3f} ms/step; per op {op_ms}")

    # ---- policy-update operations, timed on their own after the step: the
    # backward of the lm-head log-prob for the same rows (incoming gradient
    # seeded N(0, 1), lse from the forward above) and the GRPO surrogate over
    # the policy pass's 262144 rows
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

    res = {"n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded, HBM-resident)",
           "config": {"workload": desc, "kv_layout": args.kv_layout if x is not None else None}}
    rooflines = []
    if x is not None:
        nbytes = decode_bytes(x)
        gbs = nbytes / (op_ms["decode"] * 1e-3) / 1e9
        res.update({"metric": "decode-attn effective KV GB/s (% HBM peak)", "value": round(gbs, 1),
                    "unit": "GB/s", "decode_ms": round(op_ms["decode"], 4),
                    "decode_ms_p10_p90": op_pct["decode"],
                    "decode_hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
                    "decode_algorithmic_bytes": nbytes})
        rooflines.append((op_ms["decode"], {"kernel": "decode attention (split + combine kernels)",
                                            "bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                                            "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                                            "traffic": measured_traffic("decode", args.workload),
                                            "algorithmic_bytes": nbytes}))
    if y is not None:
        fl = lmhead_flops(y.cfg)
        tf = fl / (op_ms["lmhead"] * 1e-3) / 1e12
        res.update({"lmhead_ms": round(op_ms["lmhead"], 4), "lmhead_ms_p10_p90": op_pct["lmhead"],
                    "lmhead_tflops": round(tf, 1),
                    "lmhead_mfma_frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4), "lmhead_flops": fl})
        if x is None:
            res.update({"metric": "lm-head logprob TFLOP/s (% MFMA)", "value": round(tf, 1),
                        "unit": "TFLOP/s"})
        # the bound is the resource whose peak allows the longer time: MFMA
        # at the 8B-class and policy shapes, HBM (the weights) at 256 rows
        nb = lmhead_bytes(y.cfg)
        if nb / (HBM_PEAK_GBS * 1e9) > fl / (MFMA_BF16_PEAK_TFLOPS * 1e12):
            gbs_l = nb / (op_ms["lmhead"] * 1e-3) / 1e9
            entry = {"kernel": "lm-head log-prob (tile + combine kernels)", "bound": "hbm",
                     "achieved": round(gbs_l, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs_l / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic("lmhead", args.workload), "algorithmic_bytes": nb}
        else:
            entry = {"kernel": "lm-head log-prob (tile + combine kernels)", "bound": "mfma",
                     "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic("lmhead", args.workload), "algorithmic_flops": fl}
        rooflines.append((op_ms["lmhead"], entry))
    res["metric"] = "decode-attn effective KV GB/s (% HBM peak); lm-head logprob TFLOP/s (% MFMA)" \
        if (x is not None and y is not None) else res["metric"]
    rooflines.sort(key=lambda t: -t[0])
    res["roofline"] = rooflines[0][1]            # the operation that takes the most time
    if len(rooflines) > 1:
        res["roofline_other"] = rooflines[1][1]
    if update is not None:
        res["extra_ops"] = update
    if args.cpu_budget > 0:
        log("bench: cpu baseline (fp64 oracle)")
        if x is not None:
            res["cpu_baseline"] = cpu_baseline_decode(x, args.cpu_budget)
            if y is not None:
                res["cpu_baseline_lmhead"] = cpu_baseline_logprob(y, args.cpu_budget)
        else:
            res["cpu_baseline"] = cpu_baseline_logprob(y, args.cpu_budget)
    order = ["metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
             "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"]
    line = {k: res[k] for k in order if k in res}
    line.update({k: v for k, v in res.items() if k not in line})
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
