"""radar_append_decode (one call per decode step) against the fp64 oracle and,
bit for bit, against radar_append followed by radar_decode.

The merged call runs the decode kernels of the two-call sequence and only
moves the k/v row write into the first per-(b, kv head) kernel of the path
(and the summary refresh after the decode), so its outputs, selections,
scores, cache rows and summaries must equal the two-call run's bits. The
oracle runs check the merged call itself with the core parity acceptance
(tie band 1e-5, outputs 2e-3 fp32 / 1e-2 bf16, summaries 1e-4). In the
"hot" runs every query is twice its own new key, so the row written in
the same call dominates the softmax: a stale read of it could not pass.
"""
import os
import sys

import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import _harness as H  # noqa: E402

import paper_2503_10571_amd as radar  # noqa: E402
import workloads  # noqa: E402
from workloads import Workload, WORKLOADS  # noqa: E402

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


def _oracle_run(wl, steps, path, check_steps=None, **opt):
    print(f"[case] merged {wl.name} B{wl.batch} Hq{wl.n_q_heads}/"
          f"{wl.n_kv_heads} d{wl.head_dim} t0={wl.t0} c={wl.seg_len} "
          f"k={wl.top_k} w={wl.window} {wl.dtype} steps={steps} path={path} "
          f"{opt}", flush=True)
    ep = H.Episode(wl, steps, path=path, merged=True, **opt)
    st = ep.run(check_steps=check_steps)
    print(f"  heads={st.heads} out_err={st.max_out_err:.2e} "
          f"score_err={st.max_score_err:.2e} summ_err={st.max_summ_err:.2e}",
          flush=True)
    assert st.heads > 0


# --------------------------------------------------------------------------
# against the oracle
# --------------------------------------------------------------------------
@PATHS
def test_tiny_merged(path):
    _oracle_run(WORKLOADS["tiny"], 32, path)


@PATHS
def test_llama2_16k_merged_with_close(path):
    """A segment closes at t = 16512; its summary is refreshed after that
    step's decode and is a candidate from the next closing window on."""
    _oracle_run(WORKLOADS["llama2_16k"], 130, path,
                check_steps=set(range(0, 130, 16)) | {126, 127, 128, 129})


@PATHS
def test_mha_128k_scaled_merged(path):
    wl = WORKLOADS["mha_128k"].scaled(name="mha_128k_s", batch=2, n_q_heads=4,
                                      n_kv_heads=4, t0=12800)
    _oracle_run(wl, 260, path, check_steps={0, 1, 255, 256, 259})


MERGED_EDGES = [
    # no window: the completed segment is a candidate at once (the call
    # appends, refreshes, then decodes)
    (_edge("m_w0", t0=600, seg_len=32, window=0, top_k=3), {}),
    # segment length not a multiple of the tile, one-token window
    (_edge("m_c100_w1", t0=1000, seg_len=100, window=1, top_k=2), {}),
    (_edge("m_rag_gqa_sink", batch=3, n_q_heads=8, n_kv_heads=2, t0=2000,
           seg_len=64, window=64, top_k=3),
     dict(lens0=[1999, 640, 10], n_sink=4)),
    (_edge("m_rag_ph_f32", batch=3, n_q_heads=8, n_kv_heads=2, t0=900,
           seg_len=33, window=20, top_k=4, dtype="f32", head_dim=64,
           n_features=64),
     dict(lens0=[900, 34, 1], per_head=True)),
]


@PATHS
@pytest.mark.parametrize("wl,opt", MERGED_EDGES,
                         ids=[w.name for w, _ in MERGED_EDGES])
def test_merged_edges(wl, opt, path):
    _oracle_run(wl, 70, path, **opt)


# --------------------------------------------------------------------------
# bit for bit against radar_append + radar_decode
# --------------------------------------------------------------------------
def _bits(x):
    return x.view(torch.int16) if x.element_size() == 2 else x.view(torch.int32)


def _drive(wl, cfg, inp, steps, path, merged, lens0=None, hot=False):
    """steps decode steps from the index at t0; returns every step's outputs
    plus the final cache and summaries."""
    dev = inp.K.device
    K, V = inp.K.clone(), inp.V.clone()
    summ = radar.new_summaries(cfg, dev)
    radar.build_index(cfg, K, inp.omega, wl.t0, summ)
    ws = radar.new_workspace(cfg, wl.top_k, dev)
    lens = [wl.t0] * wl.batch if lens0 is None else list(lens0)
    outs = []
    radar.set_decode_path(path)
    try:
        for i in range(steps):
            kn, vn = inp.k_new[i].contiguous(), inp.v_new[i].contiguous()
            if hot:
                q = (kn.float().repeat_interleave(wl.group, dim=1) * 2.0).to(
                    kn.dtype).contiguous()
            else:
                q = inp.q[i].contiguous()
            sel = torch.full((wl.batch, wl.n_q_heads, wl.top_k), 7,
                             dtype=torch.int32, device=dev)
            sc = torch.zeros(wl.batch, wl.n_q_heads, wl.top_k,
                             dtype=torch.float32, device=dev)
            pos = None if lens0 is None else \
                torch.tensor(lens, dtype=torch.int64, device=dev)
            t = max(lens) + 1
            if merged:
                out = radar.append_decode(cfg, q, K, V, kn, vn, inp.omega, summ,
                                          t, wl.top_k, selected=sel, scores=sc,
                                          workspace=ws, pos=pos)
            else:
                radar.append(cfg, K, V, kn, vn, inp.omega,
                             lens[0] if pos is None else 0, summ, pos=pos)
                lens_dev = None if pos is None else pos + 1
                out = radar.decode(cfg, q, K, V, inp.omega, summ, t, wl.top_k,
                                   selected=sel, scores=sc, workspace=ws,
                                   lens=lens_dev)
            outs.append((out, sel, sc))
            lens = [x + 1 for x in lens]
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    torch.cuda.synchronize()
    return outs, K, V, summ


def _compare(a, b):
    outs_a, Ka, Va, Sa = a
    outs_b, Kb, Vb, Sb = b
    for i, ((oa, sa, ca), (ob, sb, cb)) in enumerate(zip(outs_a, outs_b)):
        assert torch.equal(_bits(oa), _bits(ob)), ("out", i)
        assert torch.equal(sa, sb), ("selected", i)
        assert torch.equal(_bits(ca), _bits(cb)), ("scores", i)
    assert torch.equal(_bits(Ka), _bits(Kb))
    assert torch.equal(_bits(Va), _bits(Vb))
    assert torch.equal(_bits(Sa), _bits(Sb))


BITWISE = [
    (WORKLOADS["tiny"], 40, {}),
    (_edge("b_gqa4", batch=2, n_q_heads=8, n_kv_heads=2, t0=2000, seg_len=64,
           window=64, top_k=4, n_features=256), 70, {}),
    (_edge("b_w0", t0=700, seg_len=32, window=0, top_k=3), 40, {}),
    (_edge("b_sink_ph", batch=2, n_q_heads=4, n_kv_heads=2, t0=500,
           seg_len=16, window=20, top_k=3), 40, dict(n_sink=5, per_head=True)),
    (_edge("b_rag", batch=3, t0=600, seg_len=40, window=40, n_features=256),
     90, dict(lens0=[600, 333, 1], n_sink=2)),
]


@PATHS
@pytest.mark.parametrize("hot", [False, True], ids=["planted", "hot"])
@pytest.mark.parametrize("wl,steps,opt", BITWISE,
                         ids=[w.name for w, _, _ in BITWISE])
def test_merged_equals_two_calls_bitwise(wl, steps, opt, hot, path):
    print(f"[case] bitwise {wl.name} steps={steps} hot={hot} path={path} {opt}",
          flush=True)
    lens0 = opt.get("lens0")
    cfg = H.config_of(wl, wl.t0 + steps, opt.get("n_sink", 0),
                      opt.get("per_head", False))
    inp = workloads.make_inputs(wl, "cuda", steps=steps)
    a = _drive(wl, cfg, inp, steps, path, True, lens0, hot)
    b = _drive(wl, cfg, inp, steps, path, False, lens0, hot)
    _compare(a, b)


@PATHS
def test_merged_invalid_positions(path):
    """pos[b] = -1 writes nothing; pos[b] at or past the bound t writes its
    row but decodes nothing (NaN outputs, -1 ids, NaN scores); the other
    sequences match the two-call sequence bit for bit."""
    wl = _edge("m_bad", batch=4, t0=800, seg_len=32, window=32, top_k=3)
    print(f"[case] merged invalid positions path={path}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=200)     # capacity 1000
    cfg = H.config_of(wl, wl.t0 + 200)
    summ0 = radar.new_summaries(cfg, "cuda")
    radar.build_index(cfg, inp.K, inp.omega, wl.t0, summ0)
    pos = torch.tensor([700, -1, 900, 5], dtype=torch.int64, device="cuda")
    t_bound = 801
    kn, vn = inp.k_new[0].contiguous(), inp.v_new[0].contiguous()
    q = inp.q[0].contiguous()
    res = {}
    radar.set_decode_path(path)
    try:
        for merged in (True, False):
            K, V, summ = inp.K.clone(), inp.V.clone(), summ0.clone()
            sel = torch.zeros(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.int32,
                              device="cuda")
            sc = torch.zeros(wl.batch, wl.n_q_heads, wl.top_k,
                             dtype=torch.float32, device="cuda")
            if merged:
                out = radar.append_decode(cfg, q, K, V, kn, vn, inp.omega, summ,
                                          t_bound, wl.top_k, selected=sel,
                                          scores=sc, pos=pos)
            else:
                radar.append(cfg, K, V, kn, vn, inp.omega, 0, summ, pos=pos)
                out = radar.decode(cfg, q, K, V, inp.omega, summ, t_bound,
                                   wl.top_k, selected=sel, scores=sc,
                                   lens=pos + 1)
            res[merged] = (out, sel, sc, K, V, summ)
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    torch.cuda.synchronize()
    out, sel, sc, K, V, summ = res[True]
    for b in (1, 2):
        assert bool(torch.isnan(out[b].float()).all()), b
        assert bool((sel[b] == -1).all()) and bool(torch.isnan(sc[b]).all())
    assert torch.equal(K[2, :, 900], kn[2]) and torch.equal(V[2, :, 900], vn[2])
    assert torch.equal(K[1], inp.K[1]) and torch.equal(V[1], inp.V[1])
    ref = res[False]
    for x, y in zip(res[True], ref):
        assert torch.equal(_bits(x), _bits(y))


@pytest.mark.parametrize("schedule", ["fixed", "sqrt"])
def test_layer_step_equals_append_then_decode(schedule):
    """RadarLayer.step (one merged call, or append + restructure + decode
    when t reaches a perfect square) gives the bits of append() then
    decode()."""
    wl = _edge("layer", batch=2, n_q_heads=4, n_kv_heads=2, t0=1000,
               seg_len=32, window=32, top_k=4)
    steps = 40                         # crosses t = 1024 = 32^2
    print(f"[case] layer step schedule={schedule}", flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=steps)
    cfg = H.config_of(wl, wl.t0 + steps)
    outs = {}
    for merged in (True, False):
        layer = radar.RadarLayer(cfg, inp.omega, K=inp.K.clone(), V=inp.V.clone(),
                                 t=wl.t0, top_k=wl.top_k, schedule=schedule)
        got = []
        for i in range(steps):
            kn, vn = inp.k_new[i].contiguous(), inp.v_new[i].contiguous()
            q = inp.q[i].contiguous()
            if merged:
                got.append(layer.step(q, kn, vn))
            else:
                layer.append(kn, vn)
                got.append(layer.decode(q))
        torch.cuda.synchronize()
        outs[merged] = (got, layer)
    (ga, la), (gb, lb) = outs[True], outs[False]
    for i, (x, y) in enumerate(zip(ga, gb)):
        assert torch.equal(_bits(x), _bits(y)), i
    assert la.t == lb.t == wl.t0 + steps
    assert la.restructures == lb.restructures
    if schedule == "sqrt":
        assert la.restructures == 1
    assert torch.equal(_bits(la.summaries), _bits(lb.summaries))
