"""bench.py's host-side pieces on the CPU: the algorithmic byte and flop
counts its rooflines divide by, the counter summaries it reads traffic from
(only while the kernel source is unchanged), the CPU-baseline sampler, and
the refusal of more than one GPU."""
import os
import subprocess
import sys
import types

import numpy as np
import pytest

import bench
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_decode_bytes_match_the_workload_sizes():
    # the 8B-class step: prefix 64 x 1024 tokens once, every suffix token once,
    # K and V of 8 kv heads x 128 dims in bf16, plus q, out (bf16) and lse (fp32)
    cfg = W.DECODE_CONFIGS["8b"]
    x = types.SimpleNamespace(cfg=cfg, prefix_len=np.full(64, 1024, np.int32),
                              suffix_len=W.suffix_lengths(cfg, seed=0))
    kv_tokens = 64 * 1024 + int(x.suffix_len.sum())
    expect = kv_tokens * 8 * 128 * 2 * 2 + 2 * 512 * 32 * 128 * 2 + 512 * 32 * 4
    assert bench.decode_bytes(x) == expect
    # the seeded suffix lengths of the bench workload (mean 1152 expected)
    assert expect == 2771460096


def test_lmhead_counts():
    cfg = W.LOGPROB_CONFIGS["8b"]
    assert bench.lmhead_flops(cfg) == 2 * 512 * 4096 * 151936 == 637265772544
    # W and the hidden rows once, target in, log-prob and lse out
    assert bench.lmhead_bytes(cfg) == 2 * 151936 * 4096 + 2 * 512 * 4096 + 4 * 512 + 8 * 512


def test_extend_flops_count_visible_pairs():
    # one candidate whose 3 new tokens see a prefix of 5 and 2 earlier suffix
    # tokens: visible pairs 7+1, 7+2, 7+3 = 27; 4 D Hq flops per pair
    cfg = W.DecodeConfig("t", 1, 1, 2, 1, 64, 5, "const", 5, 5)

    class Dec:
        pass

    class Ext:
        pass
    d = Dec()
    d.cfg = cfg
    d.prefix_len = np.array([5])
    d.suffix_len = np.array([5])
    e = Ext()
    e.dec = d
    e.new_len = np.array([3])
    assert bench.extend_flops(e) == 4 * 64 * 2 * 27


@pytest.mark.parametrize("op", ["decode", "lmhead"])
def test_traffic_read_only_for_the_current_source(op, tmp_path, monkeypatch):
    path = os.path.join(ROOT, "profiles", f"{op}_8b_traffic.md")
    assert os.path.exists(path), "the counter summary of the 8B-class step is committed"
    text = open(path).read()
    assert "hbm_bytes_per_launch:" in text and "source_sha256:" in text
    # a summary taken on another source is ignored
    fake = tmp_path / "profiles"
    fake.mkdir()
    (fake / f"{op}_8b_traffic.md").write_text(
        "\n".join(l if not l.startswith("- source_sha256:") else "- source_sha256: 0" for l in text.splitlines()))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic(op, "8b") is None
    # the same lines with the current hash are read back as an integer
    (fake / f"{op}_8b_traffic.md").write_text(
        "- source_sha256: " + bench.source_sha256(op) + "\n- hbm_bytes_per_launch: 1234\n")
    assert bench.measured_traffic(op, "8b") == 1234
    assert bench.measured_traffic(op, "32b") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in r.stderr and r.stdout == ""


def test_cpu_baseline_subsample_rows():
    r = bench.subsample_rows(262144, 1024, seed=0)
    assert len(r) == 1024 and len(np.unique(r)) == 1024
    assert r[0] == 0 and r[-1] == 262143 and np.all(np.diff(r) > 0)
    assert np.array_equal(r, bench.subsample_rows(262144, 1024, seed=0))
    # at least 64 distinct 256-row tiles, the last one included
    assert len(np.unique(r // 256)) >= 64 and (262143 // 256) in set(r // 256)
    assert np.array_equal(bench.subsample_rows(10, 50), np.arange(10))


def test_source_hash_covers_included_headers():
    names = bench._local_sources("token_logprob.hip")
    assert names[0] == "token_logprob.hip"
    assert {"lds_stage.h", "tile_index.h", "kernels.h"} <= set(names)
    assert "decode_attn.hip" in bench._local_sources("decode_attn.hip")


@pytest.mark.parametrize("waves", [4, 8])
def test_timeline_markdown_on_synthetic_records(waves):
    # 8 XCDs x 32 CUs, two rounds of whole tiles, then 100 tail parts; the
    # waves per workgroup come from the records' wave field
    cus = [(x, se, sh, c) for x in range(8) for se in range(4) for sh in range(2) for c in range(4)]
    recs, b = [], 0

    def word0(x, se, sh, c, w, kind):
        return (c << 8) | (sh << 12) | (se << 13) | (w << 4) | (x << 32) | (kind << 40) | (w << 48)

    for rnd in range(2):
        for (x, se, sh, c) in cus:
            st = rnd * 16000 + b % 7
            for w in range(waves):
                recs.append([word0(x, se, sh, c, w, 0), st, st + 300, st + 15500, st + 15800, 62500, 2000000,
                             b | (80 << 32) | (10 << 48)])
            b += 1
    for i, (x, se, sh, c) in enumerate(cus[:100]):
        st = 32000
        for w in range(waves):
            recs.append([word0(x, se, sh, c, w, 2), st, st + 300, st + 4000, st + 4100, 10000, 740000,
                         i | (20 << 32) | (2 << 48)])
    md = bench.timeline_markdown(np.array(recs, dtype=np.int64), True, 2 * 151936 * 5120, "synthetic")
    assert "bit-identical" in md and f"its {waves} waves" in md
    # first table: workgroups, stages, tile duration 158 us, loop 152 us, 1900 ns per stage,
    # wait share 0.25, 2e6 cycles over 152 us = 13.158 GHz
    whole = [l for l in md.splitlines() if l.startswith("| whole tiles | 512")][0].split("|")
    assert whole[3].strip() == "80" and whole[5].strip() == "158.0/158.0/158.0"
    assert whole[9].strip() == "1900" and whole[10].strip() == "0.250" and whole[11].strip() == "13.158"
    # per-CU table: 256 CUs with 2 tiles each, 100 CUs with one part
    per_cu = [l for l in md.splitlines() if l.startswith("| whole tiles | 256")]
    assert per_cu and "2: 256 CUs" in per_cu[0]
    assert any(l.startswith("| tail parts | 100 |") and "1: 100 CUs" in l for l in md.splitlines())
    assert "361.0 us from the first start" in md


def test_decode_timeline_markdown_on_synthetic_records():
    # 256 CUs; 256 prefix items (32 rows, 1024 tokens) then 512 suffix items (4 rows)
    recs = []
    for i in range(768):
        kind, rows, ntok = (0, 32, 1024) if i < 256 else (1, 4, 512)
        cu = i % 256
        x, rest = cu // 32, cu % 32
        se, sh, c = rest // 8, (rest // 4) % 2, rest % 4
        st = (i // 256) * 4000
        tiles = (ntok + 63) // 64
        recs.append([(c << 8) | (sh << 12) | (se << 13) | (x << 32) | (kind << 40) | (rows << 48), st, st + 300,
                     st + 300 + tiles * 200, st + 300 + tiles * 200 + 100, ntok | (tiles << 32), i, 0])
    md = bench.decode_timeline_markdown(np.array(recs, dtype=np.int64), True, 512, 10 ** 9, "synthetic")
    lines = md.splitlines()
    pre = [l for l in lines if l.startswith("| prefix | 32 | 256 |")][0].split("|")
    suf = [l for l in lines if l.startswith("| suffix | 4 | 512 |")][0].split("|")
    # prefix item: 16 tiles x 2 us + 3 us first tile + 1 us partials = 36 us; 2000 ns per tile
    assert pre[5].strip() == "36.0/36.0/36.0" and pre[7].strip() == "2000"
    assert suf[5].strip() == "20.0/20.0/20.0"
    assert "over 256 CUs" in md and "at most 256 (1.00 per CU)" in md
    assert "The item that ends last: suffix" in md


def test_provenance_names_command_and_sources(monkeypatch):
    """Summaries that bench.py writes itself record the command line and the
    sha256 of the kernel sources they measured."""
    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", "32b", "--also", "", "--timeline", "t.md"])
    p = bench.provenance("lmhead")
    assert "`python3 bench.py --workload 32b --also '' --timeline t.md`" in p
    assert bench.source_sha256("lmhead") in p
