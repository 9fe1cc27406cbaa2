"""Host logic of bench.py (no GPU): the one-GPU contract and the stored
counter figures, which must read as null as soon as the kernel sources or
flags they were taken on change."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_every_counter_entry_names_existing_sources():
    for key, c in bench.COUNTERS.items():
        assert c["sources"], key
        for f in c["sources"]:
            assert os.path.isfile(os.path.join(ROOT, f)), (key, f)
        assert len(c["sha256_16"]) == 16


def test_stale_counters_read_as_null(monkeypatch, tmp_path):
    src = tmp_path / "kernel.hip"
    src.write_text("// version 1\n")
    rel = os.path.relpath(src, ROOT)
    entry = {"sources": [rel], "sha256_16": bench.sources_sha([rel]),
             "fetch_kib": 100.0, "write_kib": 50.0, "valu_per_wave_step": 64.0, "envs_per_wave": 64}
    monkeypatch.setitem(bench.COUNTERS, "probe", entry)
    assert bench.measured_traffic_bytes("probe") == pytest.approx(
        1024 * (100.0 * bench.READ_FACTOR + 50.0 * bench.WRITE_FACTOR))
    # 64 instructions per wave-step (of 64 environments) at 256 x 2.4e9
    # env-steps/s: one instruction per CU per cycle at the peak clock, half
    # the issue peak
    v = bench.valu_issue("probe", 256 * 2.4e9)
    assert v["per_cu_per_cycle"] == pytest.approx(1.0) and v["frac"] == pytest.approx(0.5)
    src.write_text("// version 2\n")
    assert bench.measured_traffic_bytes("probe") is None
    assert bench.valu_issue("probe", 1e9) is None


def test_peaks_and_algorithmic_figures():
    assert bench.HBM_PEAK_GBS == 8000.0
    assert bench.VALU_PEAK_TOPS == pytest.approx(78.6432)
    assert bench.STEP_BYTES_WITH_OUTPUTS == 20 + 20 + 16 + 4 + 1
    assert bench.STEP_BYTES_STREAM == 16 + 16 + 4 + 1
    assert bench.stream_bytes_per_env_step(0.045, 100) == pytest.approx(37 + 12 * 0.045 + 0.56)
    assert bench.STEP_BYTES_TRAJ_RESIDENT == 16 + 4 + 1
    assert bench.POLICY_FLOPS == 2 * (4 * 64 + 64 * 64 + 64 * 2)
    json.dumps(bench.COUNTERS)  # plain data
    assert bench.HEAD_N == 1 << 24 and bench.HEAD_T == 100
    for key, c in bench.COUNTERS.items():
        assert os.path.isfile(os.path.join(ROOT, c["profile"])), key
    # the two-environments-per-lane binary16 kernel counts 128 environments per wave
    assert bench.COUNTERS["resident_f16_1048576x1000"]["envs_per_wave"] == 128


def test_headline_line_shape():
    # the JSON line built from a headline measurement: the metric's fields,
    # the streaming workload in config, the roofline of the streaming kernel
    head = {"envs": 1 << 24, "steps_per_rollout": 100, "rollouts": 20, "wall_ms": 260.0,
            "event_ms": 255.0, "env_steps_per_s": (1 << 24) * 100 * 20 / 0.26,
            "ms_per_rollout": 13.0, "kernel_mean_us": 127.5, "termination_rate": 0.045}
    line = bench.headline_line(head, 20, 5)
    assert line["value"] == head["env_steps_per_s"] and line["unit"] == "env-steps/s"
    assert line["steps"] == 20 and line["warmup"] == 5 and line["n_gpus"] == 1
    assert line["ms_per_step"] == 13.0 and line["dtype"] == "f32"
    assert "16,777,216 envs x 100 steps" in line["config"]["workload"]
    r = line["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    bpe = 37 + 12 * 0.045 + 56 / 100
    assert r["bytes_per_env_step"] == pytest.approx(bpe)
    assert r["achieved"] == pytest.approx(bpe * (1 << 24) / 127.5e-6 / 1e9)
    assert r["frac"] == pytest.approx(r["achieved"] / 8000.0)
    assert r["launches_timed"] == 2000
    json.dumps(line)


def test_bad_step_counts_are_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "0"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "--steps" in r.stderr and r.stdout == ""
