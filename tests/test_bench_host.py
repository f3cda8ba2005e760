"""Host-side logic of bench.py (no GPU): the one-GPU guard, the CPU oracle
baseline's accounting, and the source hash that gates the traffic figure.

The baseline's FLOP count must be the metric's own (4 * head_dim * selected
pairs * Hq * batch per pass over the workload, pairs from the closed law of
the route, §3.1 Eq. 1), whichever sample of query blocks it timed.
"""

import os
import subprocess
import sys

import pytest

import bench
from oracle import bf1_oracle as orc
from paper_2608_20427_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_cpu_baseline_whole_passes_count_the_metric_flops():
    w = synth.WORKLOADS["tiny_n512"]
    rec = bench.cpu_baseline(w, max_seconds=30.0, min_seconds=0.2)
    assert rec["kind"] == "oracle" and rec["unit"] == "TFLOP/s"
    assert rec["cores"] >= 1 and rec["passes"] >= 1 and rec["seconds"] >= 0.2
    per_pass = 4 * w.d * orc.selected_pairs(w.n, w.b, w.L) * w.Hq * w.batch
    # whole passes only (the bound is far away), so the count is exact
    assert rec["gflop"] * 1e9 == pytest.approx(rec["passes"] * per_pass, rel=1e-12)
    assert rec["value"] == pytest.approx(rec["gflop"] * 1e9 / rec["seconds"] / 1e12, rel=1e-9)
    assert "whole workload" in rec["sample"]


def test_cpu_baseline_bounded_sample_counts_its_blocks():
    # a bound too short for one pass: the sample is a strided subset of query
    # blocks, heaviest first, and the count covers exactly those blocks
    w = synth.WORKLOADS["qwen_n4096"]
    rec = bench.cpu_baseline(w, max_seconds=1e-9)
    assert rec["passes"] == 0
    NB = orc.num_blocks(w.n, w.b)
    order = []
    for off in range(8):
        order.extend(range(NB - 1 - off, -1, -8))
    done = order[:16]                     # one chunk of 16 blocks runs before the bound is checked
    pairs = 0
    for j in done:
        r = min((j + 1) * w.b, w.n) - j * w.b
        earlier = sum(min((i + 1) * w.b, w.n) - i * w.b for i in orc.route(j, w.L) if i < j)
        pairs += r * earlier + r * (r + 1) // 2
    assert rec["gflop"] * 1e9 == pytest.approx(4 * w.d * pairs * w.Hq * w.batch, rel=1e-12)
    assert rec["sample"].startswith(f"16 of {NB} query blocks")


def test_kernel_source_hash_is_stable():
    h1 = bench.kernel_source_hash()
    assert h1 == bench.kernel_source_hash() and len(h1) == 64
    int(h1, 16)
    import json
    t = json.load(open(os.path.join(ROOT, "profiles", "bf1_fwd_traffic.json")))
    # the committed counter figure names the sources it was taken on; bench.py
    # reports it only while they match the tree
    assert len(t["kernel_source_sha256"]) == 64 and t["bytes_per_launch"] > 0


def test_profiles_index_lists_every_summary():
    # every committed profile summary is listed (with what it covers) in the index
    pdir = os.path.join(ROOT, "profiles")
    index = open(os.path.join(pdir, "README.md")).read()
    for name in sorted(os.listdir(pdir)):
        if name == "README.md":
            continue
        assert f"`{name}`" in index, name
