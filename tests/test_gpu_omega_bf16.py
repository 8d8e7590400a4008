"""Omega passed as bf16 with a bf16 cache (radar_config.omega_dtype): the
projection rounds Omega to bf16 for such caches anyway, so every summary,
selection, score and output must equal, bit for bit, the run with the fp32
Omega that holds the same values; on every decode path and both call forms,
including segment closes inside the steps. Plus oracle parity of the bf16
Omega runs."""
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


def _workloads():
    return {
        # G = 1, d = 128, n = 256; a segment closes at t = 2176 (step 27)
        "g1": WORKLOADS["llama2_16k"].scaled(name="ob_g1", n_q_heads=4,
                                             n_kv_heads=4, t0=2149),
        # G = 4, n = 256, two sequences; a segment closes at t = 4352 (step 21)
        "g4": WORKLOADS["gqa_64k"].scaled(name="ob_g4", batch=2, n_q_heads=8,
                                          n_kv_heads=2, t0=4331),
        # d = 64, n = 512, G = 2
        "d64": WORKLOADS["gqa_512k"].scaled(name="ob_d64", n_q_heads=4,
                                            n_kv_heads=2, head_dim=64,
                                            seg_len=100, window=100, t0=4590),
    }


def _bits(x):
    return x.view(torch.int16 if x.element_size() == 2 else torch.int32)


def _episode(wl, cfg, omega, inp, steps, merged):
    K, V = inp.K.clone(), inp.V.clone()
    summ = radar.new_summaries(cfg, "cuda")
    radar.build_index(cfg, K, omega, wl.t0, summ)
    ws = radar.new_workspace(cfg, wl.top_k, "cuda")
    outs, sels, scs = [], [], []
    t = wl.t0
    for i in range(steps):
        q = inp.q[i].contiguous()
        kn, vn = inp.k_new[i].contiguous(), inp.v_new[i].contiguous()
        out = torch.empty_like(q)
        sel = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.int32,
                          device="cuda")
        sc = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.float32,
                         device="cuda")
        if merged:
            t += 1
            radar.append_decode(cfg, q, K, V, kn, vn, omega, summ, t, wl.top_k,
                                out=out, selected=sel, scores=sc, workspace=ws)
        else:
            radar.append(cfg, K, V, kn, vn, omega, t, summ)
            t += 1
            radar.decode(cfg, q, K, V, omega, summ, t, wl.top_k, out=out,
                         selected=sel, scores=sc, workspace=ws)
        outs.append(out)
        sels.append(sel)
        scs.append(sc)
    torch.cuda.synchronize()
    return summ, torch.stack(outs), torch.stack(sels), torch.stack(scs)


@PATHS
@pytest.mark.parametrize("merged", [False, True], ids=["separate", "merged"])
@pytest.mark.parametrize("name", ["g1", "g4", "d64"])
def test_bitwise_equal_to_fp32_omega(name, merged, path):
    wl = _workloads()[name]
    steps = 32
    print(f"[case] omega bf16 vs fp32: {wl.name} path={path} merged={merged}",
          flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=steps)
    cfg32 = H.config_of(wl, wl.t0 + steps)
    cfg16 = dataclasses.replace(cfg32, omega_dtype=torch.bfloat16)
    om16 = inp.omega.to(torch.bfloat16)
    assert torch.equal(om16.float(), inp.omega)
    radar.set_decode_path(path)
    try:
        a = _episode(wl, cfg32, inp.omega, inp, steps, merged)
        b = _episode(wl, cfg16, om16, inp, steps, merged)
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    for x, y, what in zip(a, b, ("summaries", "outputs", "selected", "scores")):
        assert torch.equal(_bits(x), _bits(y)), what


@PATHS
def test_oracle_parity_bf16_omega(path):
    wl = _workloads()["g4"]
    print(f"[case] omega bf16 oracle parity: {wl.name} path={path}", flush=True)
    st = H.Episode(wl, 24, path=path, omega_bf16=True).run()
    assert st.heads > 0


@PATHS
def test_oracle_parity_bf16_omega_with_options(path):
    """bf16 Omega together with attention sinks, per-head GQA masks and a
    ragged batch (each sequence at its own length, appending at its own
    position)."""
    wl = _workloads()["g4"].scaled(name="ob_opts", batch=3)
    print(f"[case] omega bf16 + sinks + per-head + ragged: {wl.name} path={path}",
          flush=True)
    st = H.Episode(wl, 24, path=path, omega_bf16=True, n_sink=3, per_head=True,
                   lens0=[wl.t0, 1200, 40]).run()
    assert st.heads > 0


def test_binding_refuses_mismatched_omega():
    wl = _workloads()["g1"]
    cfg = H.config_of(wl, wl.t0 + 1)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    summ = radar.new_summaries(cfg, "cuda")
    with pytest.raises(ValueError):           # bf16 tensor, fp32 config
        radar.build_index(cfg, inp.K, inp.omega.to(torch.bfloat16), wl.t0, summ)
    cfg16 = dataclasses.replace(cfg, omega_dtype=torch.bfloat16)
    with pytest.raises(ValueError):           # fp32 tensor, bf16 config
        radar.build_index(cfg16, inp.K, inp.omega, wl.t0, summ)
    f32 = dataclasses.replace(cfg16, dtype=torch.float32)
    K32 = inp.K.float()
    with pytest.raises(radar.RadarError):     # bf16 Omega with an fp32 cache
        radar.build_index(f32, K32, inp.omega.to(torch.bfloat16), wl.t0, summ)
