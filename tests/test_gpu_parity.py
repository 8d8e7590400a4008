"""HIP path vs the fp64 oracle, through the C ABI, on the same seeded inputs.

Every case builds the index at t0 with radar_build_index, then runs
append + decode steps and checks selections (tie band 1e-5), selected scores,
outputs (2e-3 fp32 / 1e-2 bf16) and summaries against the oracle. The
workloads are the five decode configurations of the method's long-context
setting, checked in full where the oracle is fast enough and on sampled
(batch, kv head) groups at full size otherwise, plus edge cases: no candidate
segments, every segment selected, empty window, segment lengths that are not
multiples of the 64-token tile, grouped-query attention with G = 2, 4, 8,
d = 64 / 128 in both dtypes, n from 64 to 512.
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


def _announce(name):
    print(f"[case] {name}", flush=True)


PATHS = pytest.mark.parametrize("path", [radar.PATH_SPLIT, radar.PATH_FUSED,
                                 radar.PATH_SELECT,
                                 radar.PATH_SCORED],
                                ids=["split", "fused", "select", "scored"])


def _run(wl, steps, groups=None, check_steps=None, path=radar.PATH_AUTO):
    _announce(f"{wl.name} B{wl.batch} Hq{wl.n_q_heads}/{wl.n_kv_heads} "
              f"d{wl.head_dim} t0={wl.t0} c={wl.seg_len} k={wl.top_k} "
              f"n={wl.n_features} w={wl.window} {wl.dtype} steps={steps} "
              f"path={path}")
    ep = H.Episode(wl, steps, groups=groups, path=path)
    st = ep.run(check_steps=check_steps)
    print(f"  heads={st.heads} out_err={st.max_out_err:.2e} "
          f"score_err={st.max_score_err:.2e} summ_err={st.max_summ_err:.2e} "
          f"band_swaps={st.band_swaps}", flush=True)
    assert st.heads > 0
    return ep


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------
@PATHS
def test_tiny_full(path):
    """Tiny single-layer decode, fp32, all 32 steps, every head."""
    _run(WORKLOADS["tiny"], 32, path=path)


@PATHS
def test_llama2_16k_full_with_close(path):
    """Llama-2-7B-shaped layer at 16K, bf16: 130 steps (a segment closes at
    t = 16512), every head."""
    wl = WORKLOADS["llama2_16k"]
    _run(wl, 130, check_steps=set(range(0, 130, 8)) | {126, 127, 128, 129},
         path=path)


@PATHS
def test_mha_128k_scaled(path):
    wl = WORKLOADS["mha_128k"].scaled(name="mha_128k_s", batch=2, n_q_heads=4,
                                      n_kv_heads=4, t0=12800)
    _run(wl, 260, check_steps={0, 1, 2, 254, 255, 256, 259}, path=path)


@PATHS
def test_gqa_64k_scaled(path):
    wl = WORKLOADS["gqa_64k"].scaled(name="gqa_64k_s", batch=2, n_q_heads=8,
                                     n_kv_heads=2, t0=16384)
    _run(wl, 258, check_steps={0, 1, 255, 256, 257}, path=path)


@PATHS
def test_gqa_512k_scaled(path):
    wl = WORKLOADS["gqa_512k"].scaled(name="gqa_512k_s", n_q_heads=8,
                                      n_kv_heads=2, t0=36200)
    # c = 724: a segment closes at t = 36924 (step 723)
    _run(wl, 726, check_steps={0, 1, 400, 722, 723, 724, 725}, path=path)


@PATHS
@pytest.mark.parametrize("name,steps,ngroups", [
    ("mha_128k", 3, 3), ("gqa_64k", 3, 3), ("gqa_512k", 3, 2)])
def test_full_size_sampled(name, steps, ngroups, path):
    """Full-size workloads (the automatic path of the 128K MHA workload is
    the one the benchmark times); oracle checks on sampled (batch, kv head)
    groups."""
    wl = WORKLOADS[name]
    _run(wl, steps, groups=H.sample_groups(wl, ngroups, seed=1), path=path)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,steps,close_step,path", [
    ("mha_128k", 258, 255, radar.PATH_AUTO), ("mha_128k", 258, 255, radar.PATH_SPLIT),
    ("gqa_64k", 258, 255, radar.PATH_AUTO), ("gqa_512k", 614, 611, radar.PATH_AUTO)],
    ids=["mha_128k-auto", "mha_128k-split", "gqa_64k-auto", "gqa_512k-auto"])
def test_full_size_segment_close(name, steps, close_step, path):
    """Full-size workloads past their first segment close (the append at
    step close_step fills a segment: t = 131328 at 128K, 65792 at 64K GQA,
    524900 at 512K), on one sampled (batch, kv head) group: selections,
    scores and outputs checked against the oracle around the close, and the
    group's summaries (the closed segment's included) at the end."""
    wl = WORKLOADS[name]
    assert (wl.t0 + close_step + 1) % wl.seg_len == 0
    _run(wl, steps, groups=H.sample_groups(wl, 1, seed=2),
         check_steps={0, close_step - 1, close_step, close_step + 1, steps - 1},
         path=path)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("path", [radar.PATH_AUTO, radar.PATH_SPLIT, radar.PATH_SELECT,
                                  radar.PATH_SCORED, radar.PATH_FUSED],
                         ids=["auto", "split", "select", "scored", "fused"])
def test_paper_default_16k(path):
    """The paper's own settings (n = 2048, k = 64, w = 1024, c = 128) at its
    16K prefill on a GQA layer, at full size on two sampled groups, across a
    segment close (t = 16512 at step 127). (With 120 candidates the fused
    and select kernels take it too when forced.)"""
    wl = WORKLOADS["paper_16k"]
    _run(wl, 129, groups=H.sample_groups(wl, 2, seed=3),
         check_steps={0, 1, 126, 127, 128}, path=path)


@pytest.mark.parametrize("n,G,dtype", [(1024, 1, "bf16"), (2048, 4, "bf16"),
                                         (1024, 4, "f32"), (2048, 1, "f32"),
                                         (2048, 8, "bf16"), (2048, 2, "bf16")])
def test_large_feature_counts(n, G, dtype):
    """n = 1024 and 2048 (the paper's default feature count): the score
    passes read each summary row in feature chunks (the split path's score
    kernel and the fused and select kernels' phase 2); with four or more
    chunks the split path's score kernel spreads a row batch's chunks over
    2 or 4 waves (n = 1024 at G >= 4, n = 2048 at every G)."""
    wl = Workload(f"n{n}_g{G}", batch=2, n_q_heads=2 * G, n_kv_heads=2, head_dim=128,
                  t0=2100, seg_len=64, top_k=6, n_features=n, window=64, dtype=dtype,
                  steps=6, keys="clustered", planted=2)
    for path in (radar.PATH_SPLIT, radar.PATH_FUSED, radar.PATH_SELECT, radar.PATH_SCORED):
        _run(wl, 6, path=path)


def test_path_choice():
    """The fused path serves shapes with at least one (b, kv head) pair per
    CU, small steps, or few summary rows per pair (several workgroups per
    pair); the select path fp32 d = 128 caches with few rows; the scored
    path the other shapes with G <= 4 (many rows per pair, more than 1024
    candidates); G = 8 and fp32 d = 128 with many rows the split path."""
    def cfg(wl):
        return H.config_of(wl, wl.t0 + 1)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    mha = WORKLOADS["mha_128k"]
    assert mha.batch * mha.n_kv_heads >= n_cu
    assert radar.decode_path(cfg(mha), mha.t0 + 1, mha.top_k) == radar.PATH_FUSED
    g5 = WORKLOADS["gqa_512k"]
    assert radar.decode_path(cfg(g5), g5.t0 + 1, g5.top_k) == radar.PATH_SCORED
    pd = WORKLOADS["paper_16k"]
    assert radar.decode_path(cfg(pd), pd.t0 + 1, pd.top_k) == radar.PATH_SCORED
    f32_many = WORKLOADS["gqa_512k"].scaled(dtype="f32")
    assert radar.decode_path(cfg(f32_many), f32_many.t0 + 1, 32) == radar.PATH_SPLIT
    # a small step per pair (launch-bound): fused even with few pairs
    tiny = WORKLOADS["tiny"]
    assert radar.decode_path(cfg(tiny), tiny.t0 + 1, tiny.top_k) == radar.PATH_FUSED
    g8 = mha.scaled(n_q_heads=32, n_kv_heads=4, batch=128)
    assert radar.decode_path(cfg(g8), g8.t0 + 1, 16) == radar.PATH_SPLIT
    # few pairs with few summary rows each: fused, several workgroups a pair
    for name in ("llama2_16k", "gqa_64k"):
        w = WORKLOADS[name]
        assert radar.decode_path(cfg(w), w.t0 + 1, w.top_k) == radar.PATH_FUSED, name
    # the same with an fp32 cache at d = 128: select
    f32 = WORKLOADS["llama2_16k"].scaled(dtype="f32")
    assert radar.decode_path(cfg(f32), f32.t0 + 1, f32.top_k) == radar.PATH_SELECT
    radar.set_decode_path(radar.PATH_FUSED)
    try:
        assert radar.decode_path(cfg(g5), g5.t0 + 1, g5.top_k) == radar.PATH_FUSED
        many = mha.scaled(seg_len=64, window=64)           # 2047 candidates
        assert radar.decode_path(cfg(many), many.t0 + 1, 16) == radar.PATH_SPLIT
        wide = mha.scaled(n_features=2048)                  # the paper's n
        assert radar.decode_path(cfg(wide), wide.t0 + 1, 16) == radar.PATH_FUSED
        radar.set_decode_path(radar.PATH_SELECT)
        assert radar.decode_path(cfg(g5), g5.t0 + 1, g5.top_k) == radar.PATH_SELECT
        assert radar.decode_path(cfg(g8), g8.t0 + 1, 16) == radar.PATH_SPLIT
        assert radar.decode_path(cfg(wide), wide.t0 + 1, 16) == radar.PATH_SELECT
        radar.set_decode_path(radar.PATH_SCORED)
        assert radar.decode_path(cfg(mha), mha.t0 + 1, 16) == radar.PATH_SCORED
        assert radar.decode_path(cfg(many), many.t0 + 1, 16) == radar.PATH_SCORED
        assert radar.decode_path(cfg(g8), g8.t0 + 1, 16) == radar.PATH_SPLIT
        assert radar.decode_path(cfg(f32_many), f32_many.t0 + 1, 32) == radar.PATH_SPLIT
    finally:
        radar.set_decode_path(radar.PATH_AUTO)


# --------------------------------------------------------------------------
# edge cases
# --------------------------------------------------------------------------
def _edge(name, **kw):
    base = dict(batch=1, n_q_heads=2, n_kv_heads=2, head_dim=128, t0=300,
                seg_len=16, top_k=3, n_features=128, window=32, dtype="bf16",
                steps=1, keys="gauss_scaled", planted=2)
    base.update(kw)
    return Workload(name, **base)


EDGES = [
    # t <= w: no candidate segment, the window is everything
    _edge("window_only", t0=20, window=64, seg_len=16),
    # k >= n_cand: every candidate selected, exact full attention
    _edge("all_selected", t0=150, window=16, seg_len=16, top_k=64),
    # w = 0: Algorithm 1's buffer; t0 multiple of c gives W = {new token}
    _edge("w0", t0=256, window=0, seg_len=32, top_k=2),
    # segment lengths that are not multiples of the 64-token tile
    _edge("c100", t0=1000, window=100, seg_len=100, top_k=3),
    _edge("c65", t0=700, window=65, seg_len=65, top_k=4, dtype="f32",
          head_dim=64, n_features=64),
    _edge("c1", t0=900, window=5, seg_len=1, top_k=7, n_features=64),
    # grouped-query attention
    _edge("gqa2", n_q_heads=4, n_kv_heads=2, t0=2000, seg_len=64, window=64,
          top_k=5, keys="clustered"),
    _edge("gqa8", n_q_heads=16, n_kv_heads=2, t0=3000, seg_len=128,
          window=128, top_k=4, keys="clustered"),
    # head dims / dtypes / feature counts
    _edge("d64_bf16", head_dim=64, t0=1500, seg_len=64, window=64,
          n_features=256),
    _edge("d128_f32", head_dim=128, t0=1500, seg_len=64, window=64,
          dtype="f32", n_features=512),
    _edge("n512_b3", batch=3, t0=1200, seg_len=48, window=50, n_features=512,
          top_k=6, keys="clustered"),
    # the largest k the library takes, with more candidates than k
    _edge("k256", t0=1100, seg_len=4, window=16, top_k=256, n_features=64,
          keys="clustered"),
    # exactly the largest candidate count (2048 one-token segments)
    _edge("cand2048", t0=2055, seg_len=1, window=8, top_k=17, n_features=64,
          keys="clustered"),
    # a context that starts at one token and grows into segments
    _edge("t_one", t0=1, seg_len=4, window=4, top_k=2),
]


@PATHS
@pytest.mark.parametrize("wl", EDGES, ids=[w.name for w in EDGES])
def test_edge(wl, path):
    steps = 70 if wl.seg_len <= 64 else 8
    if wl.name == "cand2048":
        steps = 1                          # one more step would pass 2048
    _run(wl, steps, path=path)


# --------------------------------------------------------------------------
# properties
# --------------------------------------------------------------------------
def test_append_equals_rebuild_bitwise():
    """Summaries grown by appends equal a one-shot rebuild bit for bit (the
    segment close runs the build kernel's code path)."""
    wl = _edge("grow", t0=500, seg_len=48, window=48, n_features=256,
               keys="clustered", batch=2)
    ep = _run(wl, 100)
    t = wl.t0 + 100
    fresh = radar.new_summaries(ep.cfg, ep.K.device)
    radar.build_index(ep.cfg, ep.K, ep.inp.omega, t, fresh)
    torch.cuda.synchronize()
    n_seg = t // wl.seg_len
    assert torch.equal(fresh[:, :, :n_seg], ep.summ[:, :, :n_seg])


@pytest.mark.parametrize("c,d,n", [(129, 128, 256), (191, 64, 512), (255, 128, 64),
                                   (384, 128, 256)])
def test_build_tiles_ragged_segments(c, d, n):
    """bf16 keys in segments of at least 128 go through the index build in
    128-key tiles: segment lengths that end in a partial tile (1, 63, 127
    keys) or span three whole tiles, against the oracle's summaries at the
    prefix and after the appends that close a segment, and appends equal to
    a one-shot rebuild bit for bit."""
    steps = c + 2                          # at least one segment closes
    wl = _edge(f"build_c{c}", t0=6 * c + 5, seg_len=c, window=c, n_features=n,
               head_dim=d, keys="clustered", batch=2, n_kv_heads=2, n_q_heads=2,
               top_k=2)
    ep = _run(wl, steps, check_steps={0, steps - 1})
    t = wl.t0 + steps
    fresh = radar.new_summaries(ep.cfg, ep.K.device)
    radar.build_index(ep.cfg, ep.K, ep.inp.omega, t, fresh)
    torch.cuda.synchronize()
    n_seg = t // c
    assert n_seg == 7
    assert torch.equal(fresh[:, :, :n_seg], ep.summ[:, :, :n_seg])


def test_attend_selected_matches_oracle_selection():
    """The gather-attention stage on the oracle's own selection."""
    wl = _edge("hook", n_q_heads=8, n_kv_heads=2, t0=3000, seg_len=96,
               window=96, top_k=5, keys="clustered", n_features=256)
    _announce("attend_selected")
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1)
    t = wl.t0
    q = inp.q[0].contiguous()
    om = H.f64(inp.omega)
    ws, n_cand = orc.window_split(t, wl.seg_len, wl.window)
    G = wl.group
    sel = -np.ones((wl.batch, wl.n_q_heads, wl.top_k), dtype=np.int32)
    q64 = H.f64(q)
    summ = {}
    for b in range(wl.batch):
        for g in range(wl.n_kv_heads):
            summ[(b, g)] = orc.segment_summaries(H.f64(inp.K[b, g, :t]), om,
                                                 wl.seg_len)
            for h in range(g * G, (g + 1) * G):
                sc = orc.segment_scores(orc.random_features(q64[b, h], om),
                                        summ[(b, g)][:n_cand])
                s = orc.top_segments(sc, wl.top_k)
                sel[b, h, :len(s)] = s
    # plant duplicates and out-of-range ids: both must be ignored
    sel[0, 1, -1] = sel[0, 0, 0]
    sel[0, 2, -1] = n_cand + 3
    out = radar.attend_selected(cfg, q, inp.K, inp.V,
                                torch.as_tensor(sel, device="cuda"), t)
    torch.cuda.synchronize()
    got = H.f64(out)
    for b in range(wl.batch):
        for g in range(wl.n_kv_heads):
            ids = sorted({int(s) for s in sel[b, g * G:(g + 1) * G].ravel()
                          if 0 <= s < n_cand})
            toks = orc.attended_tokens(ids, wl.seg_len, ws, t)
            for h in range(g * G, (g + 1) * G):
                ref = orc.attend(q64[b, h], H.f64(inp.K[b, g, :t]),
                                 H.f64(inp.V[b, g, :t]), toks)
                assert H.rel_inf(got[b, h], ref) <= 1e-2


def test_decode_deterministic():
    """Two decodes of the same inputs give identical bits."""
    wl = _edge("det", n_q_heads=8, n_kv_heads=2, t0=5000, seg_len=128,
               window=128, top_k=6, keys="clustered", n_features=256)
    _announce("determinism")
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = H.config_of(wl, wl.t0 + 1)
    summ = radar.new_summaries(cfg, "cuda")
    radar.build_index(cfg, inp.K, inp.omega, wl.t0, summ)
    q = inp.q[0].contiguous()
    outs, sels = [], []
    for _ in range(2):
        sel = torch.full((wl.batch, wl.n_q_heads, wl.top_k), 7,
                         dtype=torch.int32, device="cuda")
        outs.append(radar.decode(cfg, q, inp.K, inp.V, inp.omega, summ,
                                 wl.t0, wl.top_k, selected=sel))
        sels.append(sel)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    assert torch.equal(sels[0], sels[1])


def test_errors_leave_outputs_untouched():
    """Rejected calls launch nothing."""
    wl = _edge("err")
    cfg = H.config_of(wl, 64)
    K = torch.zeros(1, 2, 64, 128, dtype=torch.bfloat16, device="cuda")
    om = torch.zeros(128, 128, device="cuda")
    summ = torch.full((1, 2, 4, 128), 5.0, device="cuda")
    with pytest.raises(radar.RadarError) as e:
        radar.build_index(cfg, K, om, 65, summ)
    assert e.value.status == 2
    q = torch.zeros(1, 2, 128, dtype=torch.bfloat16, device="cuda")
    out = torch.full_like(q, 3.0)
    with pytest.raises(radar.RadarError) as e:
        radar.decode(cfg, q, K, K, om, summ, 10, 300, out=out,
                     workspace=torch.empty(1 << 20, dtype=torch.uint8,
                                           device="cuda"))
    assert e.value.status == 3
    torch.cuda.synchronize()
    assert bool((summ == 5.0).all()) and bool((out == 3.0).all())


def test_binding_refuses_wrong_sizes():
    """A tensor whose size does not match the config is refused before any
    kernel could address past its end."""
    wl = _edge("sizes")
    cfg = H.config_of(wl, 64)
    K = torch.zeros(1, 2, 64, 128, dtype=torch.bfloat16, device="cuda")
    short = torch.zeros(1, 2, 63, 128, dtype=torch.bfloat16, device="cuda")
    om = torch.zeros(128, 128, device="cuda")
    summ = torch.zeros(1, 2, 4, 128, device="cuda")
    q = torch.zeros(1, 2, 128, dtype=torch.bfloat16, device="cuda")
    row = torch.zeros(1, 2, 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError, match="K holds"):
        radar.build_index(cfg, short, om, 10, summ)
    with pytest.raises(ValueError, match="summaries holds"):
        radar.build_index(cfg, K, om, 10, summ[:, :, :3].contiguous())
    with pytest.raises(ValueError, match="omega holds"):
        radar.build_index(cfg, K, om[:64].contiguous(), 10, summ)
    with pytest.raises(ValueError, match="V holds"):
        radar.decode(cfg, q, K, short, om, summ, 10, 2)
    with pytest.raises(ValueError, match="k_new holds"):
        radar.append(cfg, K, K, row[:, :1].contiguous(), row, om, 10, summ)
    with pytest.raises(ValueError, match="selected holds"):
        radar.decode(cfg, q, K, K, om, summ, 10, 4,
                     selected=torch.zeros(1, 2, 3, dtype=torch.int32,
                                          device="cuda"))
    with pytest.raises(ValueError, match="out holds"):
        radar.append_decode(cfg, q, K, K, row, row, om, summ, 10, 2,
                            out=q[:, :1].contiguous())


@PATHS
@pytest.mark.parametrize("k", [3, 6, 13])
def test_exact_ties_take_lower_index(path, k):
    """Identical segments have bit-identical summaries and scores; the
    selection must then be the oracle's order exactly: score descending,
    lower segment index first among equal scores."""
    _announce(f"exact ties k={k} path={path}")
    rng = np.random.default_rng(123 + k)
    d, c, n, n_types, reps = 64, 16, 128, 4, 8
    B, NH = 1, 2
    types = rng.standard_normal((NH, n_types, c, d)) * 0.4
    order = rng.permutation(n_types * reps) % n_types      # segment -> type
    t0 = n_types * reps * c + 5                              # + a ragged tail
    K = np.zeros((B, NH, t0 + 1, d))
    for h in range(NH):
        for s_, ty in enumerate(order):
            K[0, h, s_ * c:(s_ + 1) * c] = types[h, ty]
        K[0, h, n_types * reps * c:] = rng.standard_normal((t0 + 1 - n_types * reps * c, d)) * 0.4
    V = rng.standard_normal((B, NH, t0 + 1, d))
    q = rng.standard_normal((B, NH, d)) * 0.5
    om = rng.standard_normal((n, d))
    # both sides read the same values: the fp32 tensors the GPU gets, widened
    K, V, q, om = (x.astype(np.float32).astype(np.float64) for x in (K, V, q, om))
    wl = Workload("ties", B, NH, NH, d, t0, c, k, n, 5, "f32", 1, "gauss", 1)
    cfg = H.config_of(wl, t0 + 1)
    Kt = torch.tensor(K, dtype=torch.float32, device="cuda")
    Vt = torch.tensor(V, dtype=torch.float32, device="cuda")
    qt = torch.tensor(q, dtype=torch.float32, device="cuda")
    omt = torch.tensor(om, dtype=torch.float32, device="cuda")
    summ = radar.new_summaries(cfg, "cuda")
    t = t0
    radar.build_index(cfg, Kt, omt, t, summ)
    sel = torch.empty(B, NH, k, dtype=torch.int32, device="cuda")
    radar.set_decode_path(path)
    try:
        radar.decode(cfg, qt, Kt, Vt, omt, summ, t, k, selected=sel)
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    torch.cuda.synchronize()
    # the GPU's own summaries of identical segments must be identical
    sm = summ.cpu().numpy()
    for h in range(NH):
        for ty in range(n_types):
            segs = np.nonzero(order == ty)[0]
            for s_ in segs[1:]:
                assert np.array_equal(sm[0, h, s_], sm[0, h, segs[0]])
    ws, n_cand = orc.window_split(t, c, wl.window)
    for h in range(NH):
        summ64 = orc.segment_summaries(K[0, h, :t], om, c)
        sc = orc.segment_scores(orc.random_features(q[0, h], om), summ64[:n_cand])
        ref = orc.top_segments(sc, k)
        assert sel[0, h].cpu().numpy().tolist() == ref.tolist()
