"""Host logic of bench.py on the CPU: the one-GPU guard, the gating of the
committed profile figures by the kernel sources' hash, and the oracle's
CPU-baseline leg on the tiny fp32 workload (no GPU is touched)."""
import json
import os
import subprocess
import sys

import pytest

import bench
from paper_2609_39137_amd import synth
from paper_2609_39137_amd.profsum import router_source_hash

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=300, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = run_bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and "--gpus 2" in r.stderr
    assert r.stdout == ""


@pytest.mark.skipif(__import__("torch").cuda.is_available(), reason="checks the message of a machine without a GPU")
def test_no_gpu_means_no_measurement():
    r = run_bench("--steps", "1", "--warmup", "0", "--no-cpu-baseline")
    assert r.returncode == 1
    assert "needs a GPU" in r.stderr
    assert r.stdout == ""


def write_profiles(tmp_path, sha, variant=6):
    (tmp_path / "router_step_top10-of-768_hbm_traffic.json").write_text(json.dumps({
        "source_sha256": sha, "variant": variant,
        "kernels": {"router": {"hbm_bytes_per_launch": 123}, "select": {"hbm_bytes_per_launch": 456}}}))
    (tmp_path / "router_step_top10-of-768_kernel_stats.json").write_text(json.dumps({
        "source_sha256": sha, "kernels": {"router": {"avg_us": 53.704}}}))


def test_profile_figures_are_reported_only_for_the_sources_they_were_taken_with(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.load_traffic("top10-of-768", 6) is None  # absent
    assert bench.load_kernel_trace_us("top10-of-768") is None
    write_profiles(tmp_path, router_source_hash())
    assert bench.load_traffic("top10-of-768", 6) == 123
    assert bench.load_traffic("top10-of-768", 6, "select") == 456
    assert bench.load_traffic("top10-of-768", 6, "merge") is None
    assert bench.load_traffic("top10-of-768", 7) is None  # counted on another tiling
    assert bench.load_kernel_trace_us("top10-of-768") == 53.7
    write_profiles(tmp_path, "0" * 16)  # kernels changed since the counters were taken
    assert bench.load_traffic("top10-of-768", 6) is None
    assert bench.load_kernel_trace_us("top10-of-768") is None


def test_committed_profiles_carry_a_sources_hash():
    for wl in ("top10-of-768", "top5-of-768-mixture", "top3-of-768-drift", "large-d4096-top10"):
        with open(os.path.join(ROOT, "profiles", f"router_step_{wl}_kernel_stats.json")) as f:
            d = json.load(f)
        assert len(d["source_sha256"]) == 16 and d["kernels"]["router"]["avg_us"] > 0


def test_cpu_baseline_leg_times_the_oracle_on_a_bounded_sample():
    wl = synth.WORKLOADS["tiny-e64-k4"]
    W = synth.router_weight(wl)
    r = bench.cpu_baseline(wl, W, target_s=0.5)
    assert r["kind"] == "oracle" and r["unit"] == "routed tokens/s"
    assert r["value"] > 0 and r["single_thread_value"] > 0
    assert r["cores"] >= 1
    assert "oracle steps" in r["sample"] and wl.name in r["sample"]
