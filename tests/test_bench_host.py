"""Host-side parts of the benchmark (no GPU): the one-GPU refusal, the figures
derived from measured durations, the HBM-traffic record and its source hash,
and the CPU-oracle baseline on a short sample."""
import json
import os
import subprocess
import sys

import pytest

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_summarize_arithmetic():
    w = synth.WORKLOADS["14b-720p"]
    flops = 4.0 * w.chunk_tokens * 64800 * w.head_dim * w.heads   # one launch, 64800 visible keys
    m = dict(attn_flops=flops, attn_ms=11.5, attn_ms_std=0.1, pub_ms=0.075, pub_cold_ms=0.08,
             rope_ms=0.072, ms_total=20 * 470.0, step_ms_std=2.0, flops=20 * w.layers * flops,
             kv_tokens=64800, anchor_frames=3)
    s = bench.summarize(w, m, 20)
    tf = flops / 11.5e-3 / 1e12
    assert s["attention"]["tflops"] == pytest.approx(tf, abs=0.01)
    assert s["attention"]["pct_bf16_peak"] == pytest.approx(100 * tf / 2500.0, abs=0.01)
    # the 50 % target is half the peak's time for one chunk-stage's attention FLOPs
    assert s["ms_attn_target_at_50pct_peak"] == pytest.approx(w.layers * flops / 1.25e15 * 1e3, rel=1e-6)
    assert s["ms_attn_per_chunk_stage"] == pytest.approx(11.5 * w.layers)
    assert s["ms_attn_publish_per_chunk_stage"] == pytest.approx((11.5 + 0.075) * w.layers)
    # publish and RoPE move the chunk's two tensors in and out once (bf16)
    moved = 4.0 * w.chunk_tokens * w.heads * w.head_dim * 2
    assert s["kv_publish"]["gbs"] == pytest.approx(moved / 0.075e-3 / 1e9, abs=0.1)
    assert s["kv_publish_cold"]["pct_hbm_peak"] == pytest.approx(100 * moved / 0.08e-3 / 8e12, abs=0.01)
    assert s["rope3d"]["gbs"] == pytest.approx(moved / 0.072e-3 / 1e9, abs=0.1)
    assert s["tflops_step"] == pytest.approx(20 * w.layers * flops / 9.4 / 1e12, abs=0.01)
    assert s["ms_per_step"] == pytest.approx(470.0)


def test_traffic_record_follows_the_kernel_source(tmp_path, monkeypatch):
    path = os.path.join(ROOT, "profiles", "attn_bf16_14b-720p_hbm_traffic.md")
    rec = json.loads(open(path).read().split("```json", 1)[1].split("```", 1)[0])
    got, src = bench.measured_traffic("14b-720p")
    assert got == float(rec["hbm_bytes_per_launch"])
    assert src == os.path.join("profiles", "attn_bf16_14b-720p_hbm_traffic.md")
    assert rec["hbm_bytes_per_launch"] == rec["hbm_read_bytes_per_launch"] + rec["hbm_write_bytes_per_launch"]
    # another source: the record no longer applies
    other = tmp_path / "attn_bf16.hip"
    other.write_text(open(bench.ATTN_SOURCE).read() + "\n// changed\n")
    monkeypatch.setattr(bench, "ATTN_SOURCE", str(other))
    assert bench.measured_traffic("14b-720p") == (None, "kernel changed since the counters were taken")
    assert bench.measured_traffic("no-such-workload")[0] is None


def test_cpu_baseline_reports_the_oracle_and_the_host():
    w = synth.WORKLOADS["14b-720p"]
    b = bench.cpu_baseline(w, target_s=0.1)
    assert b["kind"] == "oracle" and b["unit"] == "TFLOP/s"
    assert b["value"] > 0 and b["cores"] >= 1 and b["threads_used"] == b["cores"]
    assert "1 head x 512 queries x 64800 keys x d 128" in b["sample"]
    assert "cpus_allowed" in b
