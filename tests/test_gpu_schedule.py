"""Algorithm 1's restructuring schedule on the GPU (segment length
sqrt(t) at every perfect square, buffer W = [c^2, t)) against the oracle at
every step, across several restructures, on both decode paths."""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import _harness as H  # noqa: E402

import paper_2503_10571_amd as radar  # noqa: E402
import workloads  # noqa: E402
from oracle import radar_oracle as orc  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("path", [radar.PATH_SPLIT, radar.PATH_FUSED,
                                 radar.PATH_SELECT,
                          radar.PATH_SCORED],
                         ids=["split", "fused", "select", "scored"])
@pytest.mark.parametrize("dtype,Hq,Hkv,d,k", [("bf16", 4, 2, 64, 3),
                                              ("f32", 2, 2, 128, 2)])
def test_sqrt_schedule_episode(path, dtype, Hq, Hkv, d, k):
    t0, steps, n = 90, 150, 128             # squares 100, 121, ..., 225 ahead
    wl = workloads.Workload("alg1", 1, Hq, Hkv, d, t0, 9, k, n, 0, dtype,
                            steps, "clustered", 0)
    print(f"[case] sqrt schedule {dtype} Hq{Hq}/{Hkv} d{d} k{k} path={path}",
          flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=steps)
    cfg = H.config_of(wl, t0 + steps)
    layer = radar.RadarLayer(cfg, inp.omega, K=inp.K.clone(), V=inp.V.clone(),
                             t=t0, top_k=k, schedule="sqrt")
    om = H.f64(inp.omega)
    G = Hq // Hkv
    keys = {g: H.f64(inp.keys_at(steps, 0, g)) for g in range(Hkv)}
    vals = {g: H.f64(inp.values_at(steps, 0, g)) for g in range(Hkv)}
    summ_cache = {}
    sel = torch.empty(1, Hq, k, dtype=torch.int32, device="cuda")
    sc = torch.empty(1, Hq, k, dtype=torch.float32, device="cuda")
    radar.set_decode_path(path)
    try:
        for i in range(steps):
            layer.append(inp.k_new[i].contiguous(), inp.v_new[i].contiguous())
            q = inp.q[i].contiguous()
            out = layer.decode(q, selected=sel, scores=sc)
            torch.cuda.synchronize()
            t = layer.t
            c, w = orc.sqrt_schedule(t)
            assert (layer.cfg.seg_len, layer.cfg.window) == (c, w)
            ws, n_cand = orc.window_split(t, c, w)
            assert n_cand == c and ws == c * c
            k_eff = min(k, n_cand)
            q64, o64 = H.f64(q), H.f64(out)
            s_np, sc_np = sel.cpu().numpy(), sc.cpu().numpy()
            for g in range(Hkv):
                if (g, c) not in summ_cache:
                    summ_cache[(g, c)] = orc.segment_summaries(keys[g], om, c)
                summ = summ_cache[(g, c)][:n_cand]
                union = set()
                for h in range(g * G, (g + 1) * G):
                    ora = orc.segment_scores(orc.random_features(q64[0, h], om),
                                             summ)
                    H.check_selection(s_np[0, h], ora, k_eff, n_cand)
                    picks = [int(x) for x in s_np[0, h, :k_eff]]
                    union.update(picks)
                    err = np.max(np.abs(sc_np[0, h, :k_eff] - ora[picks]) / ora[picks])
                    H.note_score_err(err)
                    assert err <= H.SCORE_TOL, (i, h, err)
                toks = orc.attended_tokens(sorted(union), c, ws, t)
                for h in range(g * G, (g + 1) * G):
                    ref = orc.attend(q64[0, h], keys[g], vals[g], toks)
                    e = H.rel_inf(o64[0, h], ref)
                    assert e <= H.OUT_TOL[dtype], (i, t, h, e)
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    assert layer.restructures == 6
    # the summaries of the last restructure (c = 15 at t = 225) equal the
    # oracle's for that segment length
    c = layer.cfg.seg_len
    got = layer.summaries.view(-1)[:Hkv * (cfg.capacity // c) * n].view(
        1, Hkv, cfg.capacity // c, n)
    for g in range(Hkv):
        ref = orc.segment_summaries(keys[g][:c * c], om, c)
        err = np.max(np.abs(H.f64(got[0, g, :c]) - ref) / ref)
        assert err <= H.SUMM_TOL
