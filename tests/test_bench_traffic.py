"""bench.py reports the committed counter traffic of its dominant kernel only
for a run with the record's kernel source, step range and call form (the
bytes a launch moves depend on all three)."""
import glob
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads  # noqa: E402


def _line(rec, **over):
    run = dict(rec["run"], **over)
    return {"steps": run["steps"], "warmup": run["warmup"],
            "config": {k: v for k, v in run.items() if k not in ("steps", "warmup")}}


def _records():
    out = []
    for p in sorted(glob.glob(os.path.join(ROOT, "profiles", "traffic_*.json"))):
        out.append(json.load(open(p)))
    return out


def test_records_are_for_the_default_runs():
    recs = _records()
    assert recs, "no committed traffic records"
    for rec in recs:
        wl = workloads.WORKLOADS[rec["workload"]]
        run = rec["run"]
        assert run["steps"] == wl.steps and run["warmup"] == 16, rec["workload"]
        assert run["schedule"] == "fixed" and run["selector"] == "radar"
        assert run["calls"] == "radar_append_decode"
        assert run["omega"] == ("bf16" if wl.dtype == "bf16" else "f32")


def test_traffic_only_for_the_same_run():
    for rec in _records():
        k, w = rec["kernel"], rec["workload"]
        t = bench.measured_traffic(k, w, _line(rec))
        src = os.path.join(ROOT, rec["source"])
        fresh = hashlib.sha256(open(src, "rb").read()).hexdigest() == rec["source_sha256"]
        if not fresh:
            assert t is None
            continue
        # the record rounds the KiB and the scales; the bytes agree to 1e-3
        assert abs(t - rec["traffic_bytes_per_launch"]) <= 1e-3 * rec["traffic_bytes_per_launch"]
        assert bench.measured_traffic(k, w, _line(rec, steps=rec["run"]["steps"] // 2)) is None
        assert bench.measured_traffic(k, w, _line(rec, warmup=0)) is None
        assert bench.measured_traffic(k, w, _line(rec, calls="radar_append + radar_decode")) is None
        assert bench.measured_traffic(k, w, _line(rec, schedule="sqrt")) is None
        assert bench.measured_traffic(k, w, _line(rec, omega="other")) is None
    assert bench.measured_traffic("k_decode_fused", "no_such_workload",
                                  {"steps": 1, "warmup": 0, "config": {}}) is None


def test_byte_model_with_sinks():
    """The sinks are attended on top of the same candidates and window:
    shifting the context by the sinks adds exactly their rows to the K/V
    bytes and leaves the summary bytes alone."""
    import numpy as np
    wl = workloads.WORKLOADS["mha_128k"]
    BH = wl.batch * wl.n_kv_heads
    U = np.full(BH, wl.top_k)
    for t in (wl.t0 + 1, wl.t0 + 255, wl.t0 + 256):
        base = bench.step_bytes(wl, t, U, 2)
        assert base == bench.step_bytes(wl, t, U, 2, n_sink=0)
        for s in (1, 64):
            sh = bench.step_bytes(wl, t + s, U, 2, n_sink=s)
            assert sh[2] - base[2] == BH * s * wl.head_dim * 2 * 2      # K/V gather
            assert sh[5] == base[5]                                      # summary rows
            assert sh[4] == base[4]                                      # row append
