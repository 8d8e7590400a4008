"""Seeded random configurations vs the fp64 oracle.

Each case draws a shape (dtype, head_dim, group size, kv heads, batch,
features, segment length, window, k, sinks, GQA mode, ragged start lengths),
a decode path (a fifth of the cases the scored path) and the call form (radar_append + radar_decode, or one
radar_append_decode) from its own seed, then runs 3 decode steps through the
C ABI with the same acceptance as the core parity tests (tie band 1e-5 on
the Eq. 6 scores; outputs 2e-3 fp32 / 1e-2 bf16; summaries 1e-4), and one
exact-selector decode checked against the oracle's ln(beta) (band 1e-4).
Contexts stay small enough for the oracle to check every head.
"""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import _harness as H  # noqa: E402

import paper_2503_10571_amd as radar  # noqa: E402
from workloads import Workload  # noqa: E402
from oracle import radar_oracle as orc  # noqa: E402

pytestmark = pytest.mark.gpu

N_CASES = 300
PATHS = (radar.PATH_SPLIT, radar.PATH_FUSED, radar.PATH_SELECT, radar.PATH_AUTO)


def draw(seed):
    rng = np.random.default_rng(10_000 + seed)
    G = int(rng.choice([1, 2, 4, 8]))
    Hkv = int(rng.integers(1, 4))
    c = int(rng.choice([1, 7, 16, 33, 64, 100, 128, 200]))
    t0 = int(rng.integers(1, 3000))
    w = int(rng.choice([0, 5, 64, 150, 300]))
    # keep the candidates within the top-k stage's limit
    t0 = min(t0, 2000 * c + w)
    # at most the cache's capacity (t0 + 3 rows), as the config requires
    n_sink = min(int(rng.choice([0, 0, 1, 4, 70])), t0 + 3)
    wl = Workload(
        f"fuzz{seed}", batch=int(rng.integers(1, 4)), n_q_heads=G * Hkv,
        n_kv_heads=Hkv, head_dim=int(rng.choice([64, 128])), t0=t0, seg_len=c,
        top_k=int(rng.choice([1, 3, 8, 17, 40])),
        n_features=int(rng.choice([64, 128, 256, 512])), window=w,
        dtype=str(rng.choice(["f32", "bf16"])), steps=3,
        keys=str(rng.choice(["clustered", "gauss_scaled"])), planted=2)
    lens0 = None
    if wl.batch > 1 and rng.random() < 0.5:
        lens0 = [int(x) for x in rng.integers(1, t0 + 1, size=wl.batch)]
        lens0[0] = t0
    opt = dict(n_sink=n_sink, per_head=bool(rng.random() < 0.3), lens0=lens0)
    path = int(rng.choice(PATHS))
    # drawn last, so the earlier draws of a seed stay what they were
    opt["merged"] = bool(rng.random() < 0.5)
    opt["omega_bf16"] = bool(wl.dtype == "bf16" and rng.random() < 0.5)
    if rng.random() < 0.1:                    # the split path's chunked scores
        wl = wl.scaled(n_features=int(rng.choice([1024, 2048])))
    if rng.random() < 0.2:                    # the scored path
        path = radar.PATH_SCORED
    return wl, opt, path


@pytest.mark.parametrize("seed", range(N_CASES))
def test_fuzz_against_oracle(seed):
    wl, opt, path = draw(seed)
    print(f"[case] fuzz seed={seed} B{wl.batch} Hq{wl.n_q_heads}/{wl.n_kv_heads} "
          f"d{wl.head_dim} t0={wl.t0} c={wl.seg_len} k={wl.top_k} "
          f"n={wl.n_features} w={wl.window} {wl.dtype} path={path} {opt}",
          flush=True)
    ep = H.Episode(wl, 3, path=path, **opt)
    st = ep.run()
    assert st.heads > 0
    # the exact selector on the final cache, same options
    t = wl.t0 + 3
    lens = None if opt["lens0"] is None else [x + 3 for x in opt["lens0"]]
    q = ep.inp.q[2].contiguous()
    sel = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.int32,
                      device="cuda")
    lens_dev = None if lens is None else torch.tensor(lens, dtype=torch.int64,
                                                      device="cuda")
    out = radar.decode_exact(ep.cfg, q, ep.K, ep.V, t, wl.top_k, selected=sel,
                             lens=lens_dev)
    torch.cuda.synchronize()
    G, c, s0 = wl.group, wl.seg_len, opt["n_sink"]
    q64, sel_np, out64 = H.f64(q), sel.cpu().numpy(), H.f64(out)
    for (b, g) in ep.groups:
        tb = t if lens is None else lens[b]
        ws, n_cand = orc.window_split(tb, c, wl.window, s0)
        k_eff = min(wl.top_k, n_cand)
        keys, vals = ep.keys[(b, g)], ep.vals[(b, g)]
        own, union = {}, set()
        for h in range(g * G, (g + 1) * G):
            lnb = orc.exact_segment_mass(q64[b, h], keys[:tb], c, n_cand, offset=s0)
            H.check_selection(sel_np[b, h], lnb, k_eff, n_cand, band_abs=1e-4)
            own[h] = [int(x) for x in sel_np[b, h, :k_eff]]
            union.update(own[h])
        for h in range(g * G, (g + 1) * G):
            segs = own[h] if opt["per_head"] else sorted(union)
            toks = orc.attended_tokens(segs, c, ws, tb, s0)
            ref = orc.attend(q64[b, h], keys, vals, toks)
            assert H.rel_inf(out64[b, h], ref) <= H.OUT_TOL[wl.dtype], (b, h)
