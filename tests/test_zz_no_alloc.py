"""radar_append_decode_noalloc (the decode's scratch in the library's own
device array, for callers that cannot allocate) against radar_append_decode
with a caller workspace, through the C ABI: the same kernels run, so outputs,
selections, scores, the appended cache rows and the summaries must be equal
bit for bit, on every decode path. Two workloads run back to back, the second
smaller than the first, so the second call finds the first one's contents in
the array; a ragged batch (per-sequence positions) and a segment close are
among the steps, and the noalloc steps are also checked against the fp64
oracle."""
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

PATHS = pytest.mark.parametrize("path", [radar.PATH_AUTO, radar.PATH_SPLIT,
                                         radar.PATH_FUSED, radar.PATH_SELECT,
                                         radar.PATH_SCORED],
                                ids=["auto", "split", "fused", "select", "scored"])


def _bits(x):
    return x.view(torch.int16 if x.element_size() == 2 else torch.int32)


def _steps(wl, inp, steps, noalloc, pos0=None):
    """`steps` merged decode steps from the index at t0; returns everything
    the calls wrote."""
    cfg = H.config_of(wl, wl.t0 + steps)
    K, V = inp.K.clone(), inp.V.clone()
    summ = radar.new_summaries(cfg, "cuda")
    radar.build_index(cfg, K, inp.omega, wl.t0, summ)
    ws = None if noalloc else radar.new_workspace(cfg, wl.top_k, "cuda")
    outs, sels, scs = [], [], []
    lens = list(pos0) if pos0 is not None else None
    t = wl.t0
    for i in range(steps):
        q = inp.q[i].contiguous()
        kn, vn = inp.k_new[i].contiguous(), inp.v_new[i].contiguous()
        out = torch.full_like(q, 7.0)
        sel = torch.full((wl.batch, wl.n_q_heads, wl.top_k), 9, dtype=torch.int32,
                         device="cuda")
        sc = torch.full((wl.batch, wl.n_q_heads, wl.top_k), 5.0, device="cuda")
        pos = None if lens is None else torch.tensor(lens, dtype=torch.int64,
                                                     device="cuda")
        t = t + 1 if lens is None else max(lens) + 1
        if noalloc:
            radar.append_decode_noalloc(cfg, q, K, V, kn, vn, inp.omega, summ, t,
                                        wl.top_k, out, selected=sel, scores=sc,
                                        pos=pos)
        else:
            radar.append_decode(cfg, q, K, V, kn, vn, inp.omega, summ, t, wl.top_k,
                                out=out, selected=sel, scores=sc, workspace=ws,
                                pos=pos)
        if lens is not None:
            lens = [x + 1 for x in lens]
        outs.append(out)
        sels.append(sel)
        scs.append(sc)
    torch.cuda.synchronize()
    return [torch.stack(outs), torch.stack(sels), torch.stack(scs), summ, K, V]


def _compare(wl, steps, path, pos0=None):
    print(f"[case] noalloc vs workspace: {wl.name} path={path} pos0={pos0}",
          flush=True)
    inp = workloads.make_inputs(wl, "cuda", steps=steps)
    radar.set_decode_path(path)
    try:
        ref = _steps(wl, inp, steps, noalloc=False, pos0=pos0)
        got = _steps(wl, inp, steps, noalloc=True, pos0=pos0)
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    for a, b, what in zip(ref, got, ("out", "selected", "scores", "summaries",
                                     "K", "V")):
        assert torch.equal(_bits(a), _bits(b)), (wl.name, what)


# the larger call first, then a smaller one that reuses the array
BIG = WORKLOADS["gqa_64k"].scaled(name="noalloc_big", batch=3, n_q_heads=8,
                                  n_kv_heads=2, t0=5100)     # closes at 5120
SMALL = WORKLOADS["llama2_16k"].scaled(name="noalloc_small", n_q_heads=4,
                                       n_kv_heads=4, t0=700)


@PATHS
def test_noalloc_equals_workspace_call(path):
    _compare(BIG, 24, path)
    _compare(SMALL, 6, path)


def test_noalloc_ragged_positions():
    """Per-sequence positions (pos) through the array, a segment close in
    one sequence only."""
    _compare(BIG, 8, radar.PATH_AUTO, pos0=[5100, 4093, 2500])


@pytest.mark.parametrize("path", [radar.PATH_SPLIT, radar.PATH_FUSED],
                         ids=["split", "fused"])
def test_noalloc_matches_oracle(path):
    """The noalloc steps against the fp64 oracle (the harness's acceptance)."""
    for wl, steps in ((BIG, 22), (SMALL, 4)):
        print(f"[case] noalloc vs oracle: {wl.name} path={path}", flush=True)
        ep = H.Episode(wl, steps, path=path, merged=True, noalloc=True)
        st = ep.run()
        assert st.heads > 0


def test_noalloc_refuses_a_shape_beyond_the_array():
    """A shape whose scratch exceeds the array is refused before any launch.
    The call goes straight to the C ABI with small real buffers (the library
    rejects it before it could address them): they stay as they were."""
    import ctypes
    cfg = radar.Config(batch=64, n_q_heads=32, n_kv_heads=32, head_dim=64,
                       n_features=64, seg_len=4, window=4, capacity=1 << 16,
                       dtype=torch.float32)
    assert radar.workspace_bytes(cfg, 64) > radar.NOALLOC_SCRATCH_BYTES
    buf = torch.full((1 << 16,), 3.0, device="cuda")
    out = torch.full((1 << 12,), 2.0, device="cuda")
    P = ctypes.c_void_p
    b = P(buf.data_ptr())
    st = radar.lib().radar_append_decode_noalloc(
        ctypes.byref(cfg.c_struct()), b, b, b, b, b, b, b, 2001, None, 64,
        P(out.data_ptr()), None, None, P(torch.cuda.current_stream().cuda_stream))
    assert st == 5                      # RADAR_EWORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 2.0).all()) and bool((buf == 3.0).all())
