"""bench.py reports the committed counter traffic of its dominant kernel only
for a run with the record's library sources and call form, as the record's
traffic-to-algorithmic ratio times the run's own algorithmic bytes per
launch (the step range scales both)."""
import glob
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads  # noqa: E402


def _line(run, **over):
    return {"config": dict(run, **over)}


def _records():
    return [json.load(open(p)) for p in
            sorted(glob.glob(os.path.join(ROOT, "profiles", "traffic_*.json")))]


def test_records_are_for_the_default_call_form():
    recs = _records()
    assert recs, "no committed traffic records"
    for rec in recs:
        wl = workloads.WORKLOADS[rec["workload"]]
        run = rec["run"]
        assert run["schedule"] == "fixed" and run["selector"] == "radar"
        assert run["calls"] == "radar_append_decode"
        assert run["omega"] == ("bf16" if wl.dtype == "bf16" else "f32")


def test_traffic_only_for_the_same_sources_and_call_form(tmp_path):
    run = {"decode_path": "fused", "schedule": "fixed", "calls": "radar_append_decode",
           "selector": "radar", "omega": "bf16"}
    rec = {"kernel": "k_decode_fused", "workload": "mha_128k",
           "sources_sha256": bench.source_sha256(), "traffic_ratio": 1.01, "run": run}
    (tmp_path / "traffic_k_decode_fused_mha_128k.json").write_text(json.dumps(rec))
    t = bench.measured_traffic("k_decode_fused", "mha_128k", _line(run), 1000,
                               profiles=str(tmp_path))
    assert t == (1010, 1.01)
    for over in ({"calls": "radar_append + radar_decode"}, {"schedule": "sqrt"},
                 {"omega": "f32"}, {"decode_path": "split"}, {"layers": 4},
                 {"kv": "pinned host memory"}):
        assert bench.measured_traffic("k_decode_fused", "mha_128k", _line(run, **over),
                                      1000, profiles=str(tmp_path)) is None, over
    rec["sources_sha256"] = "0" * 64
    (tmp_path / "traffic_k_decode_fused_mha_128k.json").write_text(json.dumps(rec))
    assert bench.measured_traffic("k_decode_fused", "mha_128k", _line(run), 1000,
                                  profiles=str(tmp_path)) is None
    assert bench.measured_traffic("k_decode_fused", "no_such_workload", _line(run),
                                  1000) is None


def test_committed_records_are_consistent():
    """A record's ratio is its traffic over its algorithmic bytes."""
    for rec in _records():
        if "traffic_ratio" not in rec:
            continue
        r = rec["traffic_bytes_per_launch"] / rec["algorithmic_bytes_per_launch"]
        assert abs(r - rec["traffic_ratio"]) < 1e-3, rec["workload"]


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
