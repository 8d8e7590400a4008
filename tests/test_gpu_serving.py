"""Serving options vs the fp64 oracle: attention sinks, per-head GQA
attention and ragged batches (per-sequence lengths on the device), on both
decode paths, plus the exact selector and attend_selected with the same
options.

Acceptance as in the core parity tests: selections equal as sets up to
swaps inside the 1e-5 tie band, selected scores within 2e-5, outputs within
2e-3 (fp32) / 1e-2 (bf16) of exact attention over the tokens the oracle's
layout assigns (sinks + the head's segments + window), summaries within
1e-4. A sequence whose length is invalid must come back with -1 ids, NaN
scores and NaN outputs.
"""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import _harness as H  # noqa: E402

import paper_2503_10571_amd as radar  # noqa: E402
import workloads  # noqa: E402
from workloads import Workload, WORKLOADS  # noqa: E402
from oracle import radar_oracle as orc  # noqa: E402

pytestmark = pytest.mark.gpu

PATHS = pytest.mark.parametrize("path", [radar.PATH_SPLIT, radar.PATH_FUSED,
                                 radar.PATH_SELECT,
                                 radar.PATH_SCORED],
                                ids=["split", "fused", "select", "scored"])


def _edge(name, **kw):
    base = dict(batch=1, n_q_heads=2, n_kv_heads=2, head_dim=128, t0=300,
                seg_len=16, top_k=3, n_features=128, window=32, dtype="bf16",
                steps=1, keys="clustered", planted=2)
    base.update(kw)
    return Workload(name, **base)


def _run(wl, steps, path, check_steps=None, **opt):
    print(f"[case] {wl.name} B{wl.batch} Hq{wl.n_q_heads}/{wl.n_kv_heads} "
          f"d{wl.head_dim} t0={wl.t0} c={wl.seg_len} k={wl.top_k} "
          f"w={wl.window} {wl.dtype} steps={steps} path={path} {opt}",
          flush=True)
    ep = H.Episode(wl, steps, path=path, **opt)
    st = ep.run(check_steps=check_steps)
    print(f"  heads={st.heads} out_err={st.max_out_err:.2e} "
          f"score_err={st.max_score_err:.2e} summ_err={st.max_summ_err:.2e} "
          f"band_swaps={st.band_swaps}", flush=True)
    assert st.heads > 0
    return ep


# --------------------------------------------------------------------------
# attention sinks
# --------------------------------------------------------------------------
SINKS = [
    # one sink token, as in the appendix visualisation
    (_edge("sink1", t0=500, seg_len=32, window=32, top_k=4), 1),
    # fewer sinks than a segment, window not aligned to them
    (_edge("sink5_c16", t0=300, seg_len=16, window=20), 5),
    # more sinks than a 64-token tile, several sink tiles
    (_edge("sink100_c48", t0=700, seg_len=48, window=48, top_k=4,
           dtype="f32", head_dim=64, n_features=64), 100),
    # the context starts inside the sinks and grows past them
    (_edge("sink_grow", t0=40, seg_len=16, window=16, top_k=2), 64),
    # grouped-query heads with sinks
    (_edge("sink_gqa4", n_q_heads=8, n_kv_heads=2, t0=2000, seg_len=64,
           window=64, top_k=4, n_features=256), 4),
]


@PATHS
@pytest.mark.parametrize("wl,n_sink", SINKS, ids=[w.name for w, _ in SINKS])
def test_sinks(wl, n_sink, path):
    _run(wl, 70, path, n_sink=n_sink)


# --------------------------------------------------------------------------
# per-head grouped-query attention
# --------------------------------------------------------------------------
PER_HEAD = [
    _edge("ph_g2", n_q_heads=4, n_kv_heads=2, t0=2000, seg_len=64, window=64,
          top_k=5),
    _edge("ph_g4_f32", n_q_heads=8, n_kv_heads=2, t0=1500, seg_len=48,
          window=50, top_k=3, dtype="f32", head_dim=64, n_features=256),
    _edge("ph_g8", n_q_heads=16, n_kv_heads=2, t0=3000, seg_len=128,
          window=128, top_k=4),
    WORKLOADS["gqa_64k"].scaled(name="ph_gqa_64k_s", batch=2, n_q_heads=8,
                                n_kv_heads=2, t0=12800),
]


@PATHS
@pytest.mark.parametrize("wl", PER_HEAD, ids=[w.name for w in PER_HEAD])
def test_per_head_gqa(wl, path):
    steps = 70 if wl.seg_len <= 64 else 8
    _run(wl, steps, path, per_head=True)


@PATHS
def test_per_head_widest_union(path):
    # eight heads, each selecting the largest k from the largest candidate
    # count (2048 one-token segments): the union and its eight-bit head masks
    # span the whole bitmap
    wl = _edge("ph_g8_k256", n_q_heads=8, n_kv_heads=1, t0=2055, seg_len=1,
               window=8, top_k=256, n_features=64, keys="clustered")
    _run(wl, 1, path, per_head=True)


# --------------------------------------------------------------------------
# ragged batches
# --------------------------------------------------------------------------
RAGGED = [
    (_edge("rag_mha", batch=4, t0=1200, seg_len=48, window=50, top_k=4,
           n_features=256), [1200, 1123, 97, 3], 0),
    (_edge("rag_gqa_sink", batch=3, n_q_heads=8, n_kv_heads=2, t0=2000,
           seg_len=64, window=64, top_k=3), [1999, 640, 10], 4),
    (_edge("rag_f32_d64", batch=5, t0=900, seg_len=33, window=20, top_k=5,
           dtype="f32", head_dim=64, n_features=64), [900, 33, 34, 1, 500], 0),
]


@PATHS
@pytest.mark.parametrize("wl,lens0,n_sink", RAGGED,
                         ids=[w.name for w, _, _ in RAGGED])
def test_ragged(wl, lens0, n_sink, path):
    _run(wl, 70, path, lens0=lens0, n_sink=n_sink)


@PATHS
def test_ragged_per_head_sinks(path):
    wl = _edge("rag_all", batch=3, n_q_heads=8, n_kv_heads=2, t0=1500,
               seg_len=32, window=40, top_k=3, n_features=256)
    _run(wl, 40, path, lens0=[1500, 700, 20], n_sink=3, per_head=True)


@PATHS
def test_ragged_append_equals_rebuild_bitwise(path):
    """Per-sequence segment closes give the bits of a one-shot rebuild."""
    wl = _edge("rag_grow", batch=3, t0=600, seg_len=40, window=40,
               n_features=256)
    ep = _run(wl, 90, path, lens0=[600, 333, 80], n_sink=2,
              check_steps={0, 89})
    lens = [600 + 90, 333 + 90, 80 + 90]
    fresh = radar.new_summaries(ep.cfg, ep.K.device)
    radar.build_index(ep.cfg, ep.K, ep.inp.omega, max(lens), fresh)
    torch.cuda.synchronize()
    for b, L in enumerate(lens):
        n_seg = (L - 2) // wl.seg_len
        assert torch.equal(fresh[b, :, :n_seg], ep.summ[b, :, :n_seg]), b


@PATHS
def test_invalid_lengths_give_nan(path):
    """Lengths outside [1, t] select nothing and return NaN; the other
    sequences of the batch are unaffected."""
    wl = _edge("rag_bad", batch=4, t0=800, seg_len=32, window=32, top_k=3)
    print(f"[case] invalid lengths path={path}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1)
    summ = radar.new_summaries(cfg, "cuda")
    radar.build_index(cfg, inp.K, inp.omega, wl.t0, summ)
    q = inp.q[0].contiguous()
    lens = torch.tensor([700, 0, 801, -5], dtype=torch.int64, device="cuda")
    sel = torch.zeros(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.int32,
                      device="cuda")
    sc = torch.zeros(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.float32,
                     device="cuda")
    radar.set_decode_path(path)
    try:
        out = radar.decode(cfg, q, inp.K, inp.V, inp.omega, summ, wl.t0,
                           wl.top_k, selected=sel, scores=sc, lens=lens)
        out_e = radar.decode_exact(cfg, q, inp.K, inp.V, wl.t0, wl.top_k,
                                   lens=lens)
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    torch.cuda.synchronize()
    for b in (1, 2, 3):
        assert bool(torch.isnan(out[b].float()).all()), b
        assert bool(torch.isnan(out_e[b].float()).all()), b
        assert bool((sel[b] == -1).all()) and bool(torch.isnan(sc[b]).all())
    # sequence 0 matches the oracle at length 700
    ws, n_cand = orc.window_split(700, wl.seg_len, wl.window)
    om = H.f64(inp.omega)
    for h in range(wl.n_q_heads):
        keys = H.f64(inp.K[0, h, :700])
        s64 = orc.segment_summaries(keys, om, wl.seg_len)
        ora = orc.segment_scores(orc.random_features(H.f64(q)[0, h], om),
                                 s64[:n_cand])
        H.check_selection(sel.cpu().numpy()[0, h], ora, wl.top_k, n_cand)
        toks = orc.attended_tokens(sel[0, h].tolist(), wl.seg_len, ws, 700)
        ref = orc.attend(H.f64(q)[0, h], keys, H.f64(inp.V[0, h, :700]), toks)
        assert H.rel_inf(H.f64(out)[0, h], ref) <= H.OUT_TOL[wl.dtype]


# --------------------------------------------------------------------------
# the exact selector and attend_selected with the options
# --------------------------------------------------------------------------
@pytest.mark.parametrize("per_head", [False, True], ids=["union", "per_head"])
def test_exact_with_options(per_head):
    wl = _edge("ex_opts", batch=3, n_q_heads=8, n_kv_heads=2, t0=2500,
               seg_len=64, window=70, top_k=4)
    n_sink, lens_l = 7, [2500, 901, 30]
    print(f"[case] exact with sinks / ragged per_head={per_head}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1, n_sink, per_head)
    q = inp.q[0].contiguous()
    lens = torch.tensor(lens_l, dtype=torch.int64, device="cuda")
    sel = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.int32,
                      device="cuda")
    sc = torch.empty_like(sel, dtype=torch.float32)
    out = radar.decode_exact(cfg, q, inp.K, inp.V, wl.t0, wl.top_k,
                             selected=sel, scores=sc, lens=lens)
    torch.cuda.synchronize()
    G, c = wl.group, wl.seg_len
    q64, sel_np, sc_np = H.f64(q), sel.cpu().numpy(), sc.cpu().numpy()
    for b, t in enumerate(lens_l):
        ws, n_cand = orc.window_split(t, c, wl.window, n_sink)
        k_eff = min(wl.top_k, n_cand)
        for g in range(wl.n_kv_heads):
            keys = H.f64(inp.K[b, g, :t])
            vals = H.f64(inp.V[b, g, :t])
            own, union = {}, set()
            for h in range(g * G, (g + 1) * G):
                lnb = orc.exact_segment_mass(q64[b, h], keys, c, n_cand,
                                             offset=n_sink)
                H.check_selection(sel_np[b, h], lnb, k_eff, n_cand,
                                  band_abs=1e-4)
                own[h] = [int(s) for s in sel_np[b, h, :k_eff]]
                union.update(own[h])
                if k_eff:
                    assert np.max(np.abs(sc_np[b, h, :k_eff] - lnb[own[h]])) <= 1e-4
            for h in range(g * G, (g + 1) * G):
                segs = own[h] if per_head else sorted(union)
                toks = orc.attended_tokens(segs, c, ws, t, n_sink)
                ref = orc.attend(q64[b, h], keys, vals, toks)
                assert H.rel_inf(H.f64(out)[b, h], ref) <= 1e-2, (b, h)


@pytest.mark.parametrize("per_head", [False, True], ids=["union", "per_head"])
def test_attend_selected_with_options(per_head):
    """Given ids (with a duplicate and out-of-range ids), sinks, ragged
    lengths; a head with no ids of its own under per-head attention and an
    empty window attends only the sinks."""
    wl = _edge("given", batch=2, n_q_heads=4, n_kv_heads=2, t0=1000,
               seg_len=50, window=0, top_k=3)
    n_sink, lens_l = 3, [1000 - 47, 503]    # (t - sinks) % c == 0: W empty
    print(f"[case] attend_selected options per_head={per_head}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1, n_sink, per_head)
    rng = np.random.default_rng(4)
    G, c, k = wl.group, wl.seg_len, wl.top_k
    sel = -np.ones((wl.batch, wl.n_q_heads, k), dtype=np.int32)
    for b, t in enumerate(lens_l):
        _, n_cand = orc.window_split(t, c, wl.window, n_sink)
        for h in range(wl.n_q_heads):
            sel[b, h] = rng.choice(n_cand, k, replace=False)
    sel[0, 1, 2] = sel[0, 1, 0]            # duplicate
    sel[1, 0, 1] = 10 ** 6                 # out of range
    sel[1, 3] = -1                         # a head with no ids
    q = inp.q[0].contiguous()
    out = radar.attend_selected(cfg, q, inp.K, inp.V,
                                torch.as_tensor(sel, device="cuda"), wl.t0,
                                lens=torch.tensor(lens_l, dtype=torch.int64,
                                                  device="cuda"))
    torch.cuda.synchronize()
    q64 = H.f64(q)
    for b, t in enumerate(lens_l):
        ws, n_cand = orc.window_split(t, c, wl.window, n_sink)
        assert ws == t
        for g in range(wl.n_kv_heads):
            ok = lambda s: 0 <= s < n_cand  # noqa: E731
            heads = range(g * G, (g + 1) * G)
            union = sorted({int(s) for h in heads for s in sel[b, h] if ok(s)})
            for h in heads:
                own = sorted({int(s) for s in sel[b, h] if ok(s)})
                toks = orc.attended_tokens(own if per_head else union, c, ws,
                                           t, n_sink)
                ref = orc.attend(q64[b, h], H.f64(inp.K[b, g, :t]),
                                 H.f64(inp.V[b, g, :t]), toks)
                assert H.rel_inf(H.f64(out)[b, h], ref) <= 1e-2, (b, h)
