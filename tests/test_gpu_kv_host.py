"""The K/V cache in pinned host memory mapped for the device (the offloading
idea of the paper's memory-efficient variant): the summaries, Omega and the
workspace stay on the GPU, so the selection reads them there, and the
attention gathers only the selected segments, the window and the sinks over
the host link; appends write their rows there. The kernels are the same, so
every output, selection, score, summary and cache row must equal the
device-resident run bit for bit, on every decode path and both call forms."""
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


def _pinned(x):
    t = torch.empty(x.shape, dtype=x.dtype, pin_memory=True)
    t.copy_(x)
    return t


def _episode(wl, cfg, omega, inp, K, V, steps, merged):
    summ = radar.new_summaries(cfg, "cuda")
    radar.build_index(cfg, K, omega, wl.t0, summ)
    ws = radar.new_workspace(cfg, wl.top_k, "cuda")
    outs, sels, scs = [], [], []
    t = wl.t0
    for i in range(steps):
        q = inp.q[i].contiguous()
        kn, vn = inp.k_new[i].contiguous(), inp.v_new[i].contiguous()
        out = torch.empty_like(q)
        sel = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.int32, device="cuda")
        sc = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.float32, device="cuda")
        if merged:
            t += 1
            radar.append_decode(cfg, q, K, V, kn, vn, omega, summ, t, wl.top_k, out=out,
                                selected=sel, scores=sc, workspace=ws)
        else:
            radar.append(cfg, K, V, kn, vn, omega, t, summ)
            t += 1
            radar.decode(cfg, q, K, V, omega, summ, t, wl.top_k, out=out, selected=sel,
                         scores=sc, workspace=ws)
        outs.append(out)
        sels.append(sel)
        scs.append(sc)
    torch.cuda.synchronize()
    return [summ, torch.stack(outs), torch.stack(sels), torch.stack(scs),
            K.cpu() if K.is_cuda else K.clone(), V.cpu() if V.is_cuda else V.clone()]


@PATHS
@pytest.mark.parametrize("merged", [False, True], ids=["separate", "merged"])
def test_host_cache_equals_device_cache(merged, path):
    # G = 4, two sequences; a segment closes at t = 4352 (step 21 of 24)
    wl = WORKLOADS["gqa_64k"].scaled(name="kvhost_g4", batch=2, n_q_heads=8,
                                     n_kv_heads=2, t0=4331)
    steps = 24
    print(f"[case] K/V in pinned host memory: {wl.name} path={path} merged={merged}",
          flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=steps)
    omega = inp.omega.to(torch.bfloat16)
    cfg = dataclasses.replace(H.config_of(wl, wl.t0 + steps), omega_dtype=torch.bfloat16)
    radar.set_decode_path(path)
    try:
        dev = _episode(wl, cfg, omega, inp, inp.K.clone(), inp.V.clone(), steps, merged)
        Kh, Vh = _pinned(inp.K), _pinned(inp.V)
        assert not Kh.is_cuda and Kh.is_pinned()
        host = _episode(wl, cfg, omega, inp, Kh, Vh, steps, merged)
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    for a, b, what in zip(dev, host, ("summaries", "outputs", "selected", "scores", "K", "V")):
        assert torch.equal(_bits(a.cpu()), _bits(b.cpu())), what


KVH_ORACLE = [
    # G = 4, bf16, two sequences; a segment closes at t = 4352 (step 20)
    WORKLOADS["gqa_64k"].scaled(name="kvhost_oracle_g4", batch=2, n_q_heads=8,
                                n_kv_heads=2, t0=4331),
    # one head per group, fp32 cache, d = 64; a segment closes at t = 1280
    WORKLOADS["tiny"].scaled(name="kvhost_oracle_f32", t0=1270),
]


@PATHS
@pytest.mark.parametrize("merged", [False, True], ids=["separate", "merged"])
@pytest.mark.parametrize("wl", KVH_ORACLE, ids=[w.name for w in KVH_ORACLE])
def test_host_cache_matches_oracle(wl, merged, path):
    """With K and V in pinned host memory, every step's selections, scores
    and outputs, and the summaries (built over the host link, and refreshed
    by the append that closes a segment) against the fp64 oracle."""
    steps = 24
    print(f"[case] K/V in pinned host memory vs oracle: {wl.name} path={path} "
          f"merged={merged}", flush=True)
    ep = H.Episode(wl, steps, path=path, merged=merged, kv_host=True,
                   omega_bf16=wl.dtype == "bf16")
    st = ep.run()
    assert not ep.K.is_cuda and ep.K.is_pinned()
    assert st.heads == steps * wl.batch * wl.n_q_heads


def test_binding_refuses_unpinned_host_cache():
    wl = WORKLOADS["tiny"].scaled(name="kvhost_refuse", t0=300, steps=1)
    cfg = H.config_of(wl, wl.t0 + 1)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    summ = radar.new_summaries(cfg, "cuda")
    with pytest.raises(ValueError):
        radar.build_index(cfg, inp.K.cpu(), inp.omega, wl.t0, summ)
    with pytest.raises(ValueError):
        radar.decode(cfg, inp.q[0].contiguous(), inp.K.cpu(), inp.V.cpu(), inp.omega,
                     summ, wl.t0, wl.top_k)


@pytest.mark.parametrize("schedule", ["fixed", "sqrt"])
def test_layer_with_host_cache(schedule):
    """RadarLayer over a cache in pinned host memory keeps its summaries and
    workspace on the GPU and steps exactly like the device-resident layer
    (with the sqrt schedule, a restructure falls inside the steps)."""
    wl = WORKLOADS["llama2_16k"].scaled(name="kvhost_layer", n_q_heads=4, n_kv_heads=4,
                                        t0=2020)
    steps = 30                                # 2025 = 45^2: a restructure at step 4
    print(f"[case] RadarLayer on a host cache: schedule={schedule}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=steps)
    omega = inp.omega.to(torch.bfloat16)
    cfg = dataclasses.replace(H.config_of(wl, wl.t0 + steps), omega_dtype=torch.bfloat16)
    layers = [radar.RadarLayer(cfg, omega, K=inp.K.clone(), V=inp.V.clone(), t=wl.t0,
                               top_k=wl.top_k, schedule=schedule),
              radar.RadarLayer(cfg, omega, K=_pinned(inp.K), V=_pinned(inp.V), t=wl.t0,
                               top_k=wl.top_k, schedule=schedule)]
    assert layers[1].summaries.is_cuda and layers[1].workspace.is_cuda
    assert not layers[1].K.is_cuda
    for i in range(steps):
        outs = [L.step(inp.q[i].contiguous(), inp.k_new[i].contiguous(),
                       inp.v_new[i].contiguous()) for L in layers]
        torch.cuda.synchronize()
        assert torch.equal(_bits(outs[0]), _bits(outs[1])), i
    assert torch.equal(_bits(layers[0].summaries), _bits(layers[1].summaries))
