"""bench.py's command-line contract: one JSON line with the fields the
benchmark report needs (GPU), and a clear refusal of multi-GPU runs (CPU)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


@pytest.mark.gpu
def test_json_line_fields():
    print("[case] bench.py tiny workload, 8 steps", flush=True)
    r = subprocess.run([sys.executable, BENCH, "--workload", "tiny", "--steps", "8",
                        "--warmup", "2", "--cpu-baseline", "0", "--peaks", "0",
                        "--calibrate-copy", "0", "--build-reps", "1"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, lines
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup",
                "ms_per_step", "higher_is_better", "scaling", "vs_baseline",
                "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 8 and d["warmup"] == 2
    assert d["value"] > 0 and d["ms_per_step"] > 0
    assert d["unit"] == "tokens/s" and d["higher_is_better"] is True
    assert "workload" in d["config"]
    rl = d["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in rl, key
    assert rl["bound"] == "hbm" and rl["unit"] == "GB/s" and rl["peak"] == 8000.0
    assert 0 < rl["frac"] < 1 and abs(rl["frac"] - rl["achieved"] / rl["peak"]) < 1e-3


@pytest.mark.gpu
def test_json_line_options():
    """--kv-host adds the host-link rate of the K/V gather; --n-features
    replaces the workload's feature count (and is named in config)."""
    print("[case] bench.py tiny workload, --kv-host 1 --n-features 1024", flush=True)
    r = subprocess.run([sys.executable, BENCH, "--workload", "tiny", "--steps", "4",
                        "--warmup", "1", "--cpu-baseline", "0", "--peaks", "0",
                        "--calibrate-copy", "0", "--build-reps", "1", "--build-warmup", "1",
                        "--kv-host", "1", "--n-features", "1024"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, lines
    d = json.loads(lines[0])
    assert d["config"]["kv"] == "pinned host memory"
    assert d["config"]["n_features"] == 1024 and d["config"]["n_features_override"]
    hl = d["host_link"]
    assert hl["unit"] == "GB/s" and hl["kv_bytes_per_step"] > 0
    assert 0 < hl["achieved"] and abs(hl["frac"] - hl["achieved"] / hl["peak"]) < 1e-3
    assert d["roofline"]["traffic"] is None        # no counter record for this run


def test_cpu_baseline_runs_the_oracle_in_a_pool():
    """The oracle's host timing: one process and a pool of one-thread
    workers over the affinity cores, both scaled to all heads (CPU)."""
    sys.path.insert(0, ROOT)
    import bench
    import workloads
    wl = workloads.WORKLOADS["llama2_16k"].scaled(name="cpu_pool", n_q_heads=4,
                                                  n_kv_heads=4, t0=700)
    inp = workloads.make_inputs(wl, "cpu", steps=3)
    r = bench.cpu_baseline(wl, inp, 0, 3, n_heads=2, min_s=0.2, max_s=5.0, workers=2)
    assert r["kind"] == "oracle" and r["unit"] == "tokens/s"
    assert r["cores"] == 2 and r["value"] > 0 and r["value_1_thread"] > 0
    assert r["cores_affinity"] >= 1 and r["blas_threads_per_process"] == 1
