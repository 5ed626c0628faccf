"""bench.py's host-side logic, on the CPU: the single-GPU guard, the traffic summaries' source
check, the oracle baseline leg and the flop accounting (no GPU, no timing)."""
import hashlib
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_25683_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _summary(tmp_path, sha, hbm):
    (tmp_path / "profiles").mkdir(exist_ok=True)
    (tmp_path / "profiles" / "traffic_bwd_kv_cx.txt").write_text(
        f"# HBM traffic\nlaunches: 3\nhbm_bytes_per_launch: {hbm}\nkernel_source_sha256: {sha}\n")


def test_traffic_summary_is_used_only_for_the_current_sources(tmp_path, monkeypatch):
    h = hashlib.sha256()
    for f in bench.KERNEL_SRCS:
        h.update(open(f, "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.kernel_traffic("bwd_kv", "cx") is None           # no summary
    _summary(tmp_path, h.hexdigest(), "2.0548e+09")
    assert bench.kernel_traffic("bwd_kv", "cx") == 2.0548e9
    _summary(tmp_path, "0" * 64, "2.0548e+09")                      # taken with other sources
    assert bench.kernel_traffic("bwd_kv", "cx") is None


def test_traffic_hash_covers_the_kernels_and_the_planner():
    names = {os.path.basename(f) for f in bench.KERNEL_SRCS}
    assert {"psattn_fwd.hip", "psattn_bwd.hip", "psattn_device.h", "psattn_host.cpp", "psattn_plan.h"} <= names


def test_cpu_baseline_reports_the_oracle_sample():
    wl = W.custom([-1, 0, 0], [96, 40, 24], [1, 2], hq=4, hkv=2, d=64, dtype="bf16", seed=3,
                  block_policy=lambda L: W.blocks_fixed(L, 32))
    cb = bench.cpu_baseline(wl, 0.2)
    assert cb["kind"] == "oracle" and cb["unit"] == "tokens/s"
    assert cb["value"] > 0 and cb["cores"] >= 1 and cb["gflops_alg"] > 0
    assert cb["sample"].startswith("sample 0 (136 tokens)")
    assert "fp64" in cb["sample"]


def test_flop_accounting():
    # F_alg = 14 d per visible pair and head: forward 4 d, dK/dV 8 d, dQ 2 d; dQ executes 6 d
    assert sum(bench.FLOPS_PER_PAIR_PER_D.values()) == 14
    assert sum(bench.EXEC_FLOPS_PER_PAIR_PER_D.values()) == 18
    assert bench.PEAK_BF16_TFLOPS == 2500.0 and bench.PEAK_HBM_GBS == 8000.0
