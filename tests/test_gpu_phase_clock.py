"""radar_set_phase_clock (a measurement hook): with the stamps on, the fused
kernel's results are bit-identical to a run without them, every workgroup
of the launch writes one row of stamps, and each row is non-decreasing (the
phases end in order). Covers the fused, select and scored paths."""
import os
import sys

import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import _harness as H  # noqa: E402

import paper_2503_10571_amd as radar  # noqa: E402
import workloads  # noqa: E402
from workloads import WORKLOADS  # noqa: E402

pytestmark = pytest.mark.gpu

CASES = [(radar.PATH_FUSED, WORKLOADS["llama2_16k"].scaled(name="clk_fused", n_q_heads=8,
                                                            n_kv_heads=8, t0=3000)),
         (radar.PATH_SELECT, WORKLOADS["gqa_64k"].scaled(name="clk_select", batch=2,
                                                         n_q_heads=8, n_kv_heads=2,
                                                         t0=5000)),
         (radar.PATH_SCORED, WORKLOADS["gqa_512k"].scaled(name="clk_scored", n_q_heads=8,
                                                          n_kv_heads=2, t0=20000))]


def _bits(x):
    return x.view(torch.int16 if x.element_size() == 2 else torch.int32)


@pytest.mark.parametrize("path,wl", CASES, ids=[c[1].name for c in CASES])
def test_phase_clock(path, wl):
    print(f"[case] phase clock {wl.name} path={path}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1)
    summ = radar.new_summaries(cfg, "cuda")
    radar.build_index(cfg, inp.K, inp.omega, wl.t0, summ)
    q = inp.q[0].contiguous()
    clocks = torch.full((4096, radar.CLOCK_STAMPS), -1, dtype=torch.int64, device="cuda")
    radar.set_decode_path(path)
    try:
        res = []
        for on in (False, True):
            radar.set_phase_clock(clocks if on else None)
            sel = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.int32,
                              device="cuda")
            out = radar.decode(cfg, q, inp.K, inp.V, inp.omega, summ, wl.t0, wl.top_k,
                               selected=sel)
            torch.cuda.synchronize()
            res.append((out.clone(), sel.clone()))
    finally:
        radar.set_phase_clock(None)
        radar.set_decode_path(radar.PATH_AUTO)
    assert torch.equal(_bits(res[0][0]), _bits(res[1][0]))
    assert torch.equal(res[0][1], res[1][1])
    c = clocks.cpu()
    written = c[:, 0] >= 0
    n = int(written.sum())
    # the launch's workgroups are rows 0 .. n-1: one per pair or R per pair
    assert n >= wl.batch * wl.n_kv_heads and n % (wl.batch * wl.n_kv_heads) == 0
    assert bool(written[:n].all()) and not bool(written[n:].any())
    rows = c[:n]
    assert bool((rows[:, 1:7] >= rows[:, :6]).all())
    assert bool((rows[:, 7] == rows[:, 0]).all())      # stamp 7 unused
    khz = radar.wall_clock_khz()
    assert khz > 0
    span_us = float((rows[:, 6].max() - rows[:, 0].min()) * 1e3 / khz)
    assert 0.0 < span_us < 1e5, span_us


def test_phase_clock_rejects_bad_buffer():
    with pytest.raises(ValueError):
        radar.set_phase_clock(torch.zeros(16, 4, dtype=torch.int64, device="cuda"))
    with pytest.raises(ValueError):
        radar.set_phase_clock(torch.zeros(16, 8, dtype=torch.int32, device="cuda"))
