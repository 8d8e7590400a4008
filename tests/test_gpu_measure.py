"""The measurement hooks: per-kernel event timing and the peak-rate
microkernels stay within what the hardware can do."""
import os
import sys

import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import _harness as H  # noqa: E402

import paper_2503_10571_amd as radar  # noqa: E402
import workloads  # noqa: E402

pytestmark = pytest.mark.gpu


def test_peak_rates_are_physical():
    print("[case] peak microkernels", flush=True)
    r = radar.peak_rates(iters=512)
    # dense bf16 matrix peak 2.5 PFLOP/s; exp2 on the vector ALUs at most
    # 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
    assert 100.0 < r["mfma_tflops"] < 2600.0, r
    assert 0.5 < r["exp_T_per_s"] < 40.0, r


def test_profile_hook_counts_launches():
    wl = workloads.WORKLOADS["tiny"]
    print("[case] profile hook", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=2)
    cfg = H.config_of(wl, wl.t0 + 2)
    summ = radar.new_summaries(cfg, "cuda")
    radar.profile_enable(True)
    try:
        radar.build_index(cfg, inp.K, inp.omega, wl.t0, summ)
        radar.decode(cfg, inp.q[0].contiguous(), inp.K, inp.V, inp.omega, summ,
                     wl.t0, wl.top_k)
        torch.cuda.synchronize()
        prof = radar.profile_read()
    finally:
        radar.profile_enable(False)
    assert prof["build"][1] == 1 and prof["build"][0] > 0
    path = radar.decode_path(cfg, wl.t0, wl.top_k)
    if path == radar.PATH_FUSED:
        assert prof["fused"][1] == 1
    else:
        assert prof["attend"][1] == 1 and prof["combine"][1] == 1
    assert radar.profile_read()["build"][1] == 0      # records released
