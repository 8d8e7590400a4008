"""Exact segment search (radar_decode_exact) vs the fp64 oracle.

The exact selector ranks candidate segments by ln(beta_s), the log of the
segment's summed unnormalised attention weights (the selector of the
exact-search ablation, Section 3.3; beta as in Theorem 2's proof). Checks per
query head: the selected set equals the oracle's top-k_eff of ln(beta) up to
swaps inside an absolute band of 1e-4 around the k-th value; the returned
ln(beta) of each pick is within 1e-4 (absolute) of the oracle's; the output
matches exact attention over the group's union plus the window (2e-3 fp32,
1e-2 bf16).

The ln(beta) bound: the logits are fp32 dot products of the same (bf16 or
fp32) inputs the oracle reads, |error| <= d * 2^-24 * sum |q_i k_i| / sqrt(d)
~ 1e-5 for these unit-scale inputs; exp2 and log2 on the GPU are within a few
ulp, i.e. ~1e-6 relative to beta, ~1e-6 absolute in ln(beta).
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

LNB_TOL = 1e-4


def _edge(name, **kw):
    base = dict(batch=1, n_q_heads=2, n_kv_heads=2, head_dim=128, t0=300,
                seg_len=16, top_k=3, n_features=128, window=32, dtype="bf16",
                steps=1, keys="clustered", planted=2)
    base.update(kw)
    return Workload(name, **base)


CASES = [
    WORKLOADS["tiny"].scaled(name="tiny_x"),
    WORKLOADS["llama2_16k"].scaled(name="llama2_x", n_q_heads=4, n_kv_heads=4),
    WORKLOADS["gqa_64k"].scaled(name="gqa_64k_x", batch=2, n_q_heads=8,
                                n_kv_heads=2, t0=20000),
    # c = 724: not a multiple of the 64-token tile
    WORKLOADS["gqa_512k"].scaled(name="gqa_512k_x", n_q_heads=8, n_kv_heads=2,
                                 t0=36300),
    _edge("window_only", t0=20, window=64),
    _edge("all_selected", t0=150, window=16, top_k=64),
    _edge("c1_token_topk", t0=900, window=5, seg_len=1, top_k=7),
    _edge("c65_f32_d64", t0=700, window=65, seg_len=65, top_k=4, dtype="f32",
          head_dim=64),
    _edge("gqa8_f32_d128", n_q_heads=16, n_kv_heads=2, t0=3000, seg_len=128,
          window=128, top_k=4, dtype="f32"),
    _edge("b3_w0", batch=3, t0=1200, seg_len=48, window=0, top_k=6),
]


def _run_exact(wl):
    print(f"[case] exact {wl.name} B{wl.batch} Hq{wl.n_q_heads}/"
          f"{wl.n_kv_heads} d{wl.head_dim} t={wl.t0} c={wl.seg_len} "
          f"k={wl.top_k} w={wl.window} {wl.dtype}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1)
    t, c, G, k = wl.t0, wl.seg_len, wl.group, wl.top_k
    q = inp.q[0].contiguous()
    sel = torch.empty(wl.batch, wl.n_q_heads, k, dtype=torch.int32,
                      device="cuda")
    sc = torch.empty(wl.batch, wl.n_q_heads, k, dtype=torch.float32,
                     device="cuda")
    out = radar.decode_exact(cfg, q, inp.K, inp.V, t, k, selected=sel,
                             scores=sc)
    torch.cuda.synchronize()
    ws, n_cand = orc.window_split(t, c, wl.window)
    k_eff = min(k, n_cand)
    q64, out64 = H.f64(q), H.f64(out)
    sel_np, sc_np = sel.cpu().numpy(), sc.cpu().numpy()
    worst_out = worst_lnb = 0.0
    for b in range(wl.batch):
        for g in range(wl.n_kv_heads):
            keys = H.f64(inp.K[b, g, :t])
            vals = H.f64(inp.V[b, g, :t])
            union = set()
            for h in range(g * G, (g + 1) * G):
                lnb = orc.exact_segment_mass(q64[b, h], keys, c, n_cand)
                H.check_selection(sel_np[b, h], lnb, k_eff, n_cand,
                                  band_abs=LNB_TOL)
                picks = [int(s) for s in sel_np[b, h, :k_eff]]
                union.update(picks)
                if k_eff:
                    e = float(np.max(np.abs(sc_np[b, h, :k_eff] - lnb[picks])))
                    worst_lnb = max(worst_lnb, e)
                    assert e <= LNB_TOL, (b, h, e)
                    got = sc_np[b, h, :k_eff]
                    assert np.all(got[:-1] >= got[1:]), got
                assert np.all(np.isnan(sc_np[b, h, k_eff:]))
            toks = orc.attended_tokens(sorted(union), c, ws, t)
            for h in range(g * G, (g + 1) * G):
                ref = orc.attend(q64[b, h], keys, vals, toks)
                e = H.rel_inf(out64[b, h], ref)
                worst_out = max(worst_out, e)
                assert e <= H.OUT_TOL[wl.dtype], (b, h, e)
    print(f"  out_err={worst_out:.2e} lnb_err={worst_lnb:.2e}", flush=True)


@pytest.mark.parametrize("wl", CASES, ids=[w.name for w in CASES])
def test_exact_matches_oracle(wl):
    _run_exact(wl)


def test_exact_c1_is_token_topk():
    """With one-token segments the exact selector is the top-k of the raw
    logits (checked against the oracle's logits directly)."""
    wl = _edge("c1", t0=600, window=3, seg_len=1, top_k=9, dtype="f32",
               head_dim=64)
    print("[case] exact c=1 token top-k", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1)
    q = inp.q[0].contiguous()
    sel = torch.empty(1, 2, wl.top_k, dtype=torch.int32, device="cuda")
    radar.decode_exact(cfg, q, inp.K, inp.V, wl.t0, wl.top_k, selected=sel)
    torch.cuda.synchronize()
    ws, n_cand = orc.window_split(wl.t0, 1, wl.window)
    for h in range(2):
        lg = H.f64(inp.K[0, h, :n_cand]) @ H.f64(q)[0, h] / np.sqrt(64)
        want = np.argsort(-lg, kind="stable")[:wl.top_k]
        assert sorted(sel[0, h].tolist()) == sorted(want.tolist())


def test_exact_errors():
    wl = _edge("err")
    cfg = H.config_of(wl, 64)
    K = torch.zeros(1, 2, 64, 128, dtype=torch.bfloat16, device="cuda")
    q = torch.zeros(1, 2, 128, dtype=torch.bfloat16, device="cuda")
    out = torch.full_like(q, 3.0)
    with pytest.raises(radar.RadarError) as e:
        radar.decode_exact(cfg, q, K, K, 65, 2, out=out)
    assert e.value.status == 2
    with pytest.raises(radar.RadarError) as e:
        radar.decode_exact(cfg, q, K, K, 10, 300, out=out,
                           workspace=torch.empty(1 << 20, dtype=torch.uint8,
                                                 device="cuda"))
    assert e.value.status == 3
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())


MASS_CASES = [
    (_edge("mass_gqa4_sinks", batch=2, n_q_heads=8, n_kv_heads=2, t0=1500, seg_len=48,
           window=40), 3, [1500, 900]),
    (_edge("mass_f32_d64", head_dim=64, dtype="f32", t0=700, seg_len=65, window=65), 0, None),
    (_edge("mass_window_only", t0=20, window=64), 0, None),
    (WORKLOADS["gqa_512k"].scaled(name="mass_512k_x", n_q_heads=8, n_kv_heads=2,
                                  t0=36300), 0, None),
]


@pytest.mark.parametrize("wl,n_sink,lens", MASS_CASES, ids=[c[0].name for c in MASS_CASES])
def test_segment_mass_matches_oracle(wl, n_sink, lens):
    """radar_segment_mass: ln(beta) of every candidate segment and, at index
    n_cand, of the window and sinks, against the oracle (1e-4 absolute);
    an invalid length gives -inf at index 0 and leaves the rest alone."""
    print(f"[case] segment mass {wl.name} sinks={n_sink} lens={lens}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1, n_sink=n_sink)
    t = wl.t0
    q = inp.q[0].contiguous()
    lens_list = lens if lens is not None else [t] * wl.batch
    lens_dev = None if lens is None else torch.tensor(lens, dtype=torch.int64, device="cuda")
    ln = radar.segment_mass(cfg, q, inp.K, t, lens=lens_dev)
    torch.cuda.synchronize()
    got = ln.cpu().numpy()
    q64 = H.f64(q)
    G, c, d = wl.group, wl.seg_len, wl.head_dim
    for b in range(wl.batch):
        tb = lens_list[b]
        ws, n_cand = orc.window_split(tb, c, wl.window, n_sink)
        for g in range(wl.n_kv_heads):
            keys = H.f64(inp.K[b, g, :tb])
            rest = orc.attended_tokens([], c, ws, tb, n_sink)
            for h in range(g * G, (g + 1) * G):
                ref = orc.exact_segment_mass(q64[b, h], keys, c, n_cand, offset=n_sink)
                assert np.max(np.abs(got[b, h, :n_cand] - ref), initial=0.0) <= LNB_TOL
                lg = keys[rest] @ q64[b, h] / np.sqrt(d)
                ref_rest = lg.max() + np.log(np.exp(lg - lg.max()).sum()) if len(rest) else -np.inf
                if np.isfinite(ref_rest):
                    assert abs(got[b, h, n_cand] - ref_rest) <= LNB_TOL, (b, h)
                else:
                    assert got[b, h, n_cand] == -np.inf
                assert np.all(np.isnan(got[b, h, n_cand + 1:]))
    # an invalid length: -inf at index 0, nothing else written
    if wl.batch > 1:
        bad = torch.tensor([t] + [0] * (wl.batch - 1), dtype=torch.int64, device="cuda")
        ln2 = radar.segment_mass(cfg, q, inp.K, t, lens=bad)
        torch.cuda.synchronize()
        x = ln2.cpu().numpy()
        assert np.all(x[1:, :, 0] == -np.inf) and np.all(np.isnan(x[1:, :, 1:]))
