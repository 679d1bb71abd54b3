"""Builds librlkern.so for gfx950 with hipcc.

Each source is compiled to an object under _build/ (in parallel), then linked
into paper_2607_20908_amd/librlkern.so.  Packed-fp32 VALU instructions are
disabled for all device code.

The sources that stage tiles with the inline-asm global->LDS loads are also
compiled to gfx950 assembly, which is checked for a hazard the compiler
cannot see inside the asm: on gfx9 a VMEM instruction that reads an SGPR
needs 5 wait states after a VALU instruction wrote it, and the loads' "saddr"
form reads its base address from SGPRs.  The build fails if any base SGPR may
have been written by the VALU fewer than 5 wait states before its load, or if
a base ends up in VGPRs.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "librlkern.so")
SOURCES = ["plan.cpp", "abi.cpp", "bounds.cpp", "decode_attn.hip", "extend_attn.hip", "kv_append.hip", "token_logprob.hip", "token_logprob_bwd.hip", "sample_top_p.hip", "grpo.hip", "noalloc.hip"]
ARCH = "gfx950"
# sources whose kernels stage tiles through the inline-asm global->LDS loads
STAGING_ASM = ["extend_attn.hip", "token_logprob.hip", "token_logprob_bwd.hip"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def common_flags() -> list[str]:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-unused-function", "-Werror=inline-asm",
            f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *common_flags(), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # the host pass does not know the packed-fp32 feature; drop that one warning
    noise = [l for l in r.stderr.splitlines() if l.strip() and "packed-fp32-ops" not in l]
    if noise:
        sys.stderr.write("\n".join(noise) + "\n")
    return obj


def _device_asm(src: str) -> str:
    out = os.path.join(BUILD, os.path.splitext(src)[0] + ".gfx950.s")
    cmd = [hipcc(), *common_flags(), "-S", "--cuda-device-only", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"assembling {src} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    with open(out) as f:
        return f.read()


def _sgprs(tok: str) -> set:
    """Scalar registers named by one operand (M0 as "m0")."""
    if tok == "m0":
        return {"m0"}
    m = re.match(r"s\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"s(\d+)$", tok)
    return {int(m.group(1))} if m else set()


# VALU instructions that also write an SGPR pair as their second operand (carry out)
_CARRY_OUT = ("v_mad_u64_u32", "v_mad_i64_i32", "v_add_co_u32", "v_sub_co_u32", "v_addc_co_u32", "v_subb_co_u32",
              "v_subrev_co_u32", "v_subbrev_co_u32", "v_div_scale")
# instructions after which execution never falls through to the next line
_NO_FALLTHROUGH = ("s_branch", "s_endpgm", "s_setpc_b64")
_WAIT_STATES = 5


def staging_hazards(asm: str) -> tuple[int, list]:
    """Checks every global_load_lds of a gfx950 assembly listing: returns the
    number of loads and a description of each that may read a base SGPR or M0
    fewer than 5 wait states after a VALU write of it (or takes a VGPR base).

    From each load the check walks back along every path that reaches it: at
    a label it continues into the fall-through predecessor and into every
    branch to that label, with the wait states counted so far.  On each path
    the first writer of a register decides; a path that starts at a kernel's
    entry within the window has no writer."""
    body = []
    for line in asm.splitlines():
        t = line.split(";")[0].strip()
        if t and (not t.startswith(".") or t.endswith(":")):   # instructions and labels, no directives
            body.append(t)
    branches = {}
    for k, ins in enumerate(body):
        parts = ins.split(None, 1)
        if parts[0].startswith(("s_branch", "s_cbranch")) and len(parts) > 1:
            branches.setdefault(parts[1].strip(), []).append(k)

    def walk(j, need, ws, ins, via, errs, seen):
        while j >= 0 and need and ws < _WAIT_STATES:
            prev = body[j]
            if prev.endswith(":"):
                key = (j, ws, frozenset(need))
                if key in seen:
                    return
                seen.add(key)
                preds = list(branches.get(prev[:-1], []))
                if j > 0 and (body[j - 1].endswith(":") or body[j - 1].split()[0] not in _NO_FALLTHROUGH):
                    preds.append(j - 1)
                for pj in preds:
                    walk(pj, set(need), ws, ins, via + [prev[:-1]], errs, seen)
                return
            parts = prev.split(None, 1)
            op = parts[0]
            pops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
            written = (_sgprs(pops[0]) if pops else set())
            if op.startswith(_CARRY_OUT) and len(pops) > 1:
                written |= _sgprs(pops[1])
            written &= need
            if written:
                if op.startswith("v_"):
                    path = f" (through {', '.join(via)})" if via else ""
                    errs.append(f"VALU write {ws} wait states before the load{path}: {prev} -> {ins}")
                need -= written
            ws += (int(pops[0]) + 1 if pops else 1) if op == "s_nop" else 1
            j -= 1

    loads, errs = 0, []
    for k, ins in enumerate(body):
        if not ins.startswith("global_load_lds"):
            continue
        loads += 1
        ops = [o.strip() for o in ins.split(None, 1)[1].split(",")]
        if len(ops) > 1 and ops[1].startswith("v"):
            errs.append(f"VGPR base: {ins}")
            continue
        need = {"m0"}
        for o in ops[1:]:
            need |= _sgprs(o)
        walk(k - 1, need, 0, ins, [], errs, set())
    return loads, errs


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES) + len(STAGING_ASM)) as ex:
        asm = {src: ex.submit(_device_asm, src) for src in STAGING_ASM}
        objs = list(ex.map(_compile, SOURCES))
        for src, fut in asm.items():
            loads, errs = staging_hazards(fut.result())
            if loads == 0 or errs:
                raise RuntimeError(f"{src}: {loads} staged loads; SGPR hazards:\n" + "\n".join(errs[:20]))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,--no-undefined", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
