"""Guard regions around every buffer the library reads or writes.

Each tensor the calls receive is a view into a larger allocation whose head
and tail hold a sentinel bit pattern (and so do the cache rows past the
last appended row and the summary rows past the last full segment). Every
call of the C ABI then runs on every decode path, on shapes at the
library's limits: k = 256, 2047 candidate segments, grouped-query heads
with per-head attention, attention sinks, per-sequence positions and
lengths with invalid entries, a fused path with several workgroups per pair
(partials in the workspace) and a segment close. Afterwards every sentinel
must be intact: nothing is written past the capacity, the summary rows, the
workspace size or the outputs' extent. This runs fixed code and is meant to
find nothing."""
import dataclasses
import math
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import _harness as H  # noqa: E402

import paper_2503_10571_amd as radar  # noqa: E402
import workloads  # noqa: E402
from workloads import Workload  # noqa: E402

pytestmark = pytest.mark.gpu

PAD = 4096                     # sentinel bytes before and after each buffer
# per element size: a NaN bit pattern for the float types
SENTINEL = {1: -0x5B, 2: 0x7FA5, 4: 0x7FA5A5A5, 8: 0x7FA5A5A5A5A5A5A5}
INT = {1: torch.int8, 2: torch.int16, 4: torch.int32, 8: torch.int64}


class Guarded:
    """A tensor of `shape` inside an allocation padded with sentinels."""

    def __init__(self, shape, dtype, init=None, device="cuda"):
        self.es = torch.empty(0, dtype=dtype).element_size()
        self.n = int(np.prod(shape))
        pe = PAD // self.es
        self.buf = torch.empty(self.n + 2 * pe, dtype=dtype, device=device)
        self.ibuf = self.buf.view(INT[self.es])
        self.ibuf.fill_(self._sent())
        self.pe = pe
        self.t = self.buf[pe:pe + self.n].view(shape)
        if init is not None:
            self.t.copy_(init)

    def _sent(self):
        return SENTINEL[self.es]

    def intact(self):
        s = self._sent()
        return bool((self.ibuf[:self.pe] == s).all()) and \
            bool((self.ibuf[self.pe + self.n:] == s).all())

    def region_is_sentinel(self, sl):
        """sl: a slice of the flat view that must still hold the sentinel."""
        return bool((self.ibuf[self.pe:self.pe + self.n][sl] == self._sent()).all())


def _case(name, **kw):
    base = dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=128, t0=600,
                seg_len=32, top_k=4, n_features=128, window=32, dtype="bf16",
                steps=8, keys="clustered", planted=2)
    base.update(kw)
    return Workload(name, **base)


CASES = [
    # k = 256 of 2047 one-token candidates, G = 8, ragged lengths
    (_case("k256_cand2048", n_q_heads=16, n_kv_heads=2, t0=2050, seg_len=1,
           window=8, top_k=256, n_features=64, steps=4), dict(n_sink=0, per_head=False)),
    # sinks, per-head GQA, fp32 cache at d = 64, c not a multiple of 64
    (_case("sinks_perhead_f32", batch=3, n_q_heads=8, n_kv_heads=2, head_dim=64,
           t0=900, seg_len=33, window=20, top_k=7, dtype="f32", steps=8),
     dict(n_sink=5, per_head=True)),
    # few pairs with a few hundred KB each: several workgroups per pair on
    # the fused path, a segment close at t = 4352
    (_case("gqa4_close", n_q_heads=8, n_kv_heads=2, t0=4331, seg_len=256,
           window=256, top_k=16, n_features=256, steps=24), dict(n_sink=0, per_head=False)),
]


@pytest.mark.parametrize("path", [radar.PATH_SPLIT, radar.PATH_FUSED, radar.PATH_SELECT,
                                  radar.PATH_SCORED],
                         ids=["split", "fused", "select", "scored"])
@pytest.mark.parametrize("wl,opt", CASES, ids=[c[0].name for c in CASES])
def test_no_write_outside_buffers(wl, opt, path):
    print(f"[case] canaries {wl.name} path={path}", flush=True)
    dev = "cuda"
    inp = workloads.make_inputs(wl, dev, steps=wl.steps)
    cap = wl.t0 + wl.steps
    cfg = H.config_of(wl, cap, n_sink=opt["n_sink"], per_head=opt["per_head"])
    B, Hq, Hkv, d, k = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.top_k
    dt = wl.torch_dtype()
    rows = cfg.summary_rows
    # the cache: rows [0, t0) hold the prefix; rows after it stay sentinel
    # until an append writes them
    K = Guarded((B, Hkv, cap, d), dt)
    V = Guarded((B, Hkv, cap, d), dt)
    K.t[:, :, :wl.t0] = inp.K[:, :, :wl.t0]
    V.t[:, :, :wl.t0] = inp.V[:, :, :wl.t0]
    summ = Guarded((B, Hkv, rows, wl.n_features), torch.float32)
    om = Guarded(tuple(inp.omega.shape), torch.float32, inp.omega)
    nws = radar.workspace_bytes(cfg, k)
    ws = Guarded((nws,), torch.uint8)
    q = Guarded((B, Hq, d), dt)
    kn = Guarded((B, Hkv, d), dt)
    vn = Guarded((B, Hkv, d), dt)
    out = Guarded((B, Hq, d), dt)
    sel = Guarded((B, Hq, k), torch.int32)
    sc = Guarded((B, Hq, k), torch.float32)
    lens = Guarded((B,), torch.int64)
    given = Guarded((B, Hq, k), torch.int32)
    every = [K, V, summ, om, ws, q, kn, vn, out, sel, sc, lens, given]

    radar.set_decode_path(path)
    try:
        radar.build_index(cfg, K.t, om.t, wl.t0, summ.t)
        t = wl.t0
        for i in range(wl.steps):
            q.t.copy_(inp.q[i])
            kn.t.copy_(inp.k_new[i])
            vn.t.copy_(inp.v_new[i])
            form = i % 4
            if form == 0:                        # append, then decode
                radar.append(cfg, K.t, V.t, kn.t, vn.t, om.t, t, summ.t)
                t += 1
                radar.decode(cfg, q.t, K.t, V.t, om.t, summ.t, t, k, out=out.t,
                             selected=sel.t, scores=sc.t, workspace=ws.t)
            elif form == 1:                      # the merged call
                t += 1
                radar.append_decode(cfg, q.t, K.t, V.t, kn.t, vn.t, om.t, summ.t,
                                    t, k, out=out.t, selected=sel.t, scores=sc.t,
                                    workspace=ws.t)
            elif form == 2:                      # ragged, one sequence invalid
                pos = [t] + [-5] * (B - 1)       # only sequence 0 appends
                lens.t.copy_(torch.tensor(pos, dtype=torch.int64))
                radar.append(cfg, K.t, V.t, kn.t, vn.t, om.t, 0, summ.t, pos=lens.t)
                t += 1
                lv = [t] + [0] * (B - 1)         # length 0: invalid, NaN out
                lens.t.copy_(torch.tensor(lv, dtype=torch.int64))
                radar.decode(cfg, q.t, K.t, V.t, om.t, summ.t, t, k, out=out.t,
                             selected=sel.t, scores=sc.t, workspace=ws.t,
                             lens=lens.t)
                # the other sequences' row t - 1 was skipped: fill it the
                # way the others will expect for the remaining steps
                if B > 1:
                    K.t[1:, :, t - 1] = kn.t[1:]
                    V.t[1:, :, t - 1] = vn.t[1:]
                    radar.build_index(cfg, K.t, om.t, t, summ.t)
            else:                                # no-alloc call, exact, given
                t += 1
                radar.append_decode_noalloc(cfg, q.t, K.t, V.t, kn.t, vn.t, om.t,
                                            summ.t, t, k, out.t, selected=sel.t,
                                            scores=sc.t)
                radar.decode_exact(cfg, q.t, K.t, V.t, t, k, out=out.t,
                                   selected=sel.t, scores=sc.t, workspace=ws.t)
                g = torch.randint(-3, 3000, (B, Hq, k), dtype=torch.int32)
                given.t.copy_(g)
                radar.attend_selected(cfg, q.t, K.t, V.t, given.t, t, out=out.t,
                                      workspace=ws.t)
        torch.cuda.synchronize()
    finally:
        radar.set_decode_path(radar.PATH_AUTO)
    names = ["K", "V", "summaries", "omega", "workspace", "q", "k_new", "v_new",
             "out", "selected", "scores", "lens", "given"]
    for g, nm in zip(every, names):
        assert g.intact(), nm
    # rows after the last appended one, and summary rows after the last full
    # segment, were never written
    n_seg = (t - opt["n_sink"]) // wl.seg_len
    for bh in range(B * Hkv):
        tail = slice(bh * cap * d + t * d, (bh + 1) * cap * d)
        assert K.region_is_sentinel(tail) and V.region_is_sentinel(tail), bh
        st = slice(bh * rows * wl.n_features + n_seg * wl.n_features,
                   (bh + 1) * rows * wl.n_features)
        assert summ.region_is_sentinel(st), bh
