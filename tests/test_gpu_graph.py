"""The decode calls under HIP graph capture. A run of steps (with a segment
close inside it, so a summary refresh is captured too) is captured once and
replayed three times, each replay from the same restored cache, summaries
and workspace state, with eager work and synchronisations in between; every
replay must give the eager run's outputs, selections, scores and summaries
bit for bit, on every decode path and both call forms. (The library records
no allocation, host synchronisation or memset node: capture would fail or
the replays would differ.)"""
import dataclasses
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

PATHS = pytest.mark.parametrize("path", [radar.PATH_SPLIT, radar.PATH_FUSED,
                                         radar.PATH_SELECT,
                                 radar.PATH_SCORED],
                                ids=["split", "fused", "select", "scored"])


def _bits(x):
    return x.view(torch.int16 if x.element_size() == 2 else torch.int32)


class _Run:
    """Static buffers for `steps` decode steps of one workload."""

    def __init__(self, wl, steps, merged):
        self.wl, self.steps, self.merged = wl, steps, merged
        self.inp = workloads.make_inputs(wl, "cuda", steps=steps)
        self.omega = self.inp.omega.to(torch.bfloat16)
        self.cfg = dataclasses.replace(H.config_of(wl, wl.t0 + steps),
                                       omega_dtype=torch.bfloat16)
        self.K, self.V = self.inp.K.clone(), self.inp.V.clone()
        self.summ = radar.new_summaries(self.cfg, "cuda")
        radar.build_index(self.cfg, self.K, self.omega, wl.t0, self.summ)
        self.K0, self.V0, self.summ0 = self.K.clone(), self.V.clone(), self.summ.clone()
        self.ws = radar.new_workspace(self.cfg, wl.top_k, "cuda")
        B, Hq, k, d = wl.batch, wl.n_q_heads, wl.top_k, wl.head_dim
        self.out = torch.empty(steps, B, Hq, d, dtype=self.inp.q.dtype, device="cuda")
        self.sel = torch.empty(steps, B, Hq, k, dtype=torch.int32, device="cuda")
        self.sc = torch.empty(steps, B, Hq, k, dtype=torch.float32, device="cuda")
        self.q = [self.inp.q[i].contiguous() for i in range(steps)]
        self.kn = [self.inp.k_new[i].contiguous() for i in range(steps)]
        self.vn = [self.inp.v_new[i].contiguous() for i in range(steps)]

    def restore(self):
        self.K.copy_(self.K0)
        self.V.copy_(self.V0)
        self.summ.copy_(self.summ0)
        self.ws.zero_()
        self.out.zero_()
        self.sel.zero_()
        self.sc.zero_()

    def steps_(self):
        cfg, wl = self.cfg, self.wl
        t = wl.t0
        for i in range(self.steps):
            if self.merged:
                t += 1
                radar.append_decode(cfg, self.q[i], self.K, self.V, self.kn[i], self.vn[i],
                                    self.omega, self.summ, t, wl.top_k, out=self.out[i],
                                    selected=self.sel[i], scores=self.sc[i], workspace=self.ws)
            else:
                radar.append(cfg, self.K, self.V, self.kn[i], self.vn[i], self.omega, t,
                             self.summ)
                t += 1
                radar.decode(cfg, self.q[i], self.K, self.V, self.omega, self.summ, t,
                             wl.top_k, out=self.out[i], selected=self.sel[i],
                             scores=self.sc[i], workspace=self.ws)

    def result(self):
        return [_bits(x).clone() for x in (self.out, self.sel, self.sc, self.summ, self.K)]


@PATHS
@pytest.mark.parametrize("merged", [False, True], ids=["separate", "merged"])
def test_graph_replays_equal_eager(merged, path):
    # G = 4, two sequences; a segment closes at t = 4352 (step 21 of 24)
    wl = WORKLOADS["gqa_64k"].scaled(name="graph_g4", batch=2, n_q_heads=8,
                                     n_kv_heads=2, t0=4331)
    print(f"[case] graph capture: {wl.name} path={path} merged={merged}", flush=True)
    r = _Run(wl, 24, merged)
    radar.set_decode_path(path)
    try:
        r.restore()
        r.steps_()
        torch.cuda.synchronize()
        eager = r.result()
        r.restore()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            r.steps_()
        for rep in range(3):
            r.restore()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            got = r.result()
            for a, b, what in zip(eager, got, ("out", "selected", "scores", "summaries", "K")):
                assert torch.equal(a, b), f"replay {rep}: {what}"
            # unrelated eager work between replays
            torch.randn(1 << 20, device="cuda").sum().item()
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
