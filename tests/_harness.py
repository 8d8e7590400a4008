"""Drive the HIP path through the C ABI and compare it with the fp64 oracle.

The HIP side runs through paper_2503_10571_amd (ctypes -> libradar.so); the
oracle side is oracle.radar_oracle on float64 copies of the same seeded inputs
(workloads.make_inputs). The two share nothing but those inputs.

Acceptance rules:
  * selected segments: equal as sets to the oracle's top-k_eff, except that
    segments whose oracle score lies within 1e-5 (relative) of the oracle's
    k-th score may be swapped for one another;
  * outputs: per (b, q head) max_i |o_i - o*_i| / max_i |o*_i| <= 2e-3 (fp32)
    or 1e-2 (bf16), where o* is the oracle's exact attention over the union
    the GPU selected plus the window (identical to the oracle's own output
    whenever the sets agree);
  * scores of the selected segments: relative error against the oracle's
    Eq. 6 values at most 1e-5 (the tie band: an error below it cannot move
    a segment across the band);
  * summaries: relative error per element <= 1e-4.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch

import paper_2503_10571_amd as radar
import workloads
from oracle import radar_oracle as orc

TIE_BAND = 1e-5
OUT_TOL = {"f32": 2e-3, "bf16": 1e-2}
SCORE_TOL = 1e-5
SUMM_TOL = 1e-4

# The largest errors and the band swaps seen by every check of this process
# (the GPU run's margins against the tolerances above; tests/conftest.py
# prints them at the end of the session).
MARGINS = {"episodes": 0, "heads": 0, "band_swaps": 0, "max_score_err": 0.0,
           "max_summ_err": 0.0, "max_out_err_f32": 0.0, "max_out_err_bf16": 0.0,
           "tolerances": {"score": SCORE_TOL, "summary": SUMM_TOL,
                          "out_f32": OUT_TOL["f32"], "out_bf16": OUT_TOL["bf16"],
                          "tie_band": TIE_BAND}}


def note_score_err(err):
    MARGINS["max_score_err"] = max(MARGINS["max_score_err"], float(err))


def config_of(wl: workloads.Workload, capacity: int, n_sink: int = 0,
              per_head: bool = False) -> radar.Config:
    return radar.Config(wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                        wl.n_features, wl.seg_len, wl.window, capacity,
                        wl.torch_dtype(), n_sink,
                        radar.GQA_PER_HEAD if per_head else radar.GQA_UNION)


def f64(x: torch.Tensor) -> np.ndarray:
    return x.detach().float().cpu().double().numpy()


def check_selection(gpu_sel, ora_scores, k_eff, n_cand, band_abs=None):
    """Tie-band set check for one query head. gpu_sel: the k ids (-1 pad).
    The band around the oracle's k-th score is relative (TIE_BAND) unless
    band_abs gives an absolute half-width (for log-scale scores)."""
    sel = [int(s) for s in gpu_sel if s >= 0]
    assert len(sel) == k_eff, (sel, k_eff)
    assert len(set(sel)) == k_eff, sel
    assert all(0 <= s < n_cand for s in sel), sel
    assert all(s == -1 for s in gpu_sel[k_eff:])
    if k_eff == 0:
        return 0
    order = orc.top_segments(ora_scores, k_eff)
    s_k = ora_scores[order[-1]]
    if band_abs is None:
        hi, lo = s_k * (1 + TIE_BAND), s_k * (1 - TIE_BAND)
    else:
        hi, lo = s_k + band_abs, s_k - band_abs
    must = {int(s) for s in np.nonzero(ora_scores > hi)[0]}
    assert must <= set(sel), ("missed", sorted(must - set(sel)))
    bad = [s for s in sel if ora_scores[s] < lo]
    assert not bad, ("outside band", bad, [ora_scores[s] for s in bad], s_k)
    return len(set(sel) ^ {int(s) for s in order})


def rel_inf(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30))


@dataclasses.dataclass
class Stats:
    heads: int = 0
    max_out_err: float = 0.0
    max_score_err: float = 0.0
    max_summ_err: float = 0.0
    band_swaps: int = 0

    def merge_out(self, e):
        self.max_out_err = max(self.max_out_err, e)


class Episode:
    """One workload run: build the index at t0, then `steps` x (append,
    decode). Oracle checks on the sampled (batch, kv head) groups.

    n_sink / per_head select the attention-sink and per-head GQA options.
    lens0 (one length <= t0 per sequence) makes the batch ragged: sequence b
    starts at length lens0[b] (its cache rows beyond are stale), appends at
    its own position and decodes at its own length. merged runs each step as
    one radar_append_decode call instead of radar_append + radar_decode.
    omega_bf16 passes Omega to the library as bf16 (bf16 workloads, whose
    Omega values are bf16 already; the oracle reads the same values)."""

    def __init__(self, wl, steps, groups=None, device="cuda",
                 path=radar.PATH_AUTO, n_sink=0, per_head=False, lens0=None,
                 merged=False, omega_bf16=False, noalloc=False, kv_host=False):
        self.wl = wl
        self.steps = steps
        self.path = path
        self.merged = merged
        self.noalloc = noalloc
        self.kv_host = kv_host
        assert merged or not noalloc
        self.n_sink, self.per_head = n_sink, per_head
        self.lens0 = list(lens0) if lens0 is not None else None
        self.inp = workloads.make_inputs(wl, device, steps=steps)
        self.cfg = config_of(wl, wl.t0 + steps, n_sink, per_head)
        self.omega_dev = self.inp.omega
        if omega_bf16:
            assert wl.dtype == "bf16"
            self.omega_dev = self.inp.omega.to(torch.bfloat16)
            assert torch.equal(self.omega_dev.float(), self.inp.omega)
            self.cfg = dataclasses.replace(self.cfg, omega_dtype=torch.bfloat16)
        B, Hkv = wl.batch, wl.n_kv_heads
        self.groups = groups if groups is not None else \
            [(b, g) for b in range(B) for g in range(Hkv)]
        self.omega64 = f64(self.inp.omega)
        self.keys = {}
        self.vals = {}
        self.summ64 = {}
        for (b, g) in self.groups:
            if self.lens0 is None:
                kk = f64(self.inp.keys_at(steps, b, g))
                vv = f64(self.inp.values_at(steps, b, g))
            else:
                L0 = self.lens0[b]
                kk = np.concatenate([f64(self.inp.K[b, g, :L0]),
                                     f64(self.inp.k_new[:steps, b, g])])
                vv = np.concatenate([f64(self.inp.V[b, g, :L0]),
                                     f64(self.inp.v_new[:steps, b, g])])
            self.keys[(b, g)] = kk
            self.vals[(b, g)] = vv
            self.summ64[(b, g)] = orc.segment_summaries(kk, self.omega64,
                                                        wl.seg_len,
                                                        offset=n_sink)
        self.stats = Stats()

    def run(self, check_steps=None):
        radar.set_decode_path(self.path)
        try:
            st = self._run(check_steps)
        finally:
            radar.set_decode_path(radar.PATH_AUTO)
            self._note_margins()
        return st

    def _note_margins(self):
        st = self.stats
        M = MARGINS
        M["episodes"] += 1
        M["heads"] += st.heads
        M["band_swaps"] += st.band_swaps
        M["max_score_err"] = max(M["max_score_err"], st.max_score_err)
        M["max_summ_err"] = max(M["max_summ_err"], st.max_summ_err)
        key = "max_out_err_" + self.wl.dtype
        M[key] = max(M[key], st.max_out_err)

    def _run(self, check_steps):
        wl, inp, cfg = self.wl, self.inp, self.cfg
        dev = inp.K.device
        if self.kv_host:
            # the cache in pinned host memory mapped for the device (the
            # kernels read it over the host link); everything else on the GPU
            K = torch.empty(inp.K.shape, dtype=inp.K.dtype, pin_memory=True)
            V = torch.empty(inp.V.shape, dtype=inp.V.dtype, pin_memory=True)
            K.copy_(inp.K)
            V.copy_(inp.V)
        else:
            K, V = inp.K.clone(), inp.V.clone()
        summ = radar.new_summaries(cfg, dev)
        radar.build_index(cfg, K, self.omega_dev, wl.t0, summ)
        lens = [wl.t0] * wl.batch if self.lens0 is None else list(self.lens0)
        self.check_summaries(summ, lens)
        ws = radar.new_workspace(cfg, wl.top_k, dev)
        sel = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.int32,
                          device=dev)
        sc = torch.empty(wl.batch, wl.n_q_heads, wl.top_k, dtype=torch.float32,
                         device=dev)
        out = torch.empty_like(inp.q[0])
        for i in range(self.steps):
            kn, vn = inp.k_new[i].contiguous(), inp.v_new[i].contiguous()
            q = inp.q[i].contiguous()
            pos = None if self.lens0 is None else \
                torch.tensor(lens, dtype=torch.int64, device=dev)
            if self.merged and self.noalloc:
                lens = [x + 1 for x in lens]
                radar.append_decode_noalloc(cfg, q, K, V, kn, vn, self.omega_dev,
                                            summ, max(lens), wl.top_k, out,
                                            selected=sel, scores=sc, pos=pos)
            elif self.merged:
                lens = [x + 1 for x in lens]
                radar.append_decode(cfg, q, K, V, kn, vn, self.omega_dev, summ,
                                    max(lens), wl.top_k, out=out, selected=sel,
                                    scores=sc, workspace=ws, pos=pos)
            else:
                radar.append(cfg, K, V, kn, vn, self.omega_dev,
                             lens[0] if pos is None else 0, summ, pos=pos)
                lens = [x + 1 for x in lens]
                lens_dev = None if self.lens0 is None else \
                    torch.tensor(lens, dtype=torch.int64, device=dev)
                radar.decode(cfg, q, K, V, self.omega_dev, summ, max(lens), wl.top_k,
                             out=out, selected=sel, scores=sc, workspace=ws,
                             lens=lens_dev)
            if check_steps is None or i in check_steps:
                torch.cuda.synchronize()
                self.check_step(i, lens, q, out, sel, sc)
        self.check_summaries(summ, lens)
        self.K, self.V, self.summ = K, V, summ
        return self.stats

    def check_summaries(self, summ, lens):
        c = self.wl.seg_len
        for (b, g) in self.groups:
            n_seg = max(0, lens[b] - self.n_sink) // c
            got = f64(summ[b, g, :n_seg])
            ref = self.summ64[(b, g)][:n_seg]
            err = float(np.max(np.abs(got - ref) / np.abs(ref))) if n_seg else 0.0
            self.stats.max_summ_err = max(self.stats.max_summ_err, err)
            assert err <= SUMM_TOL, (b, g, err)

    def check_step(self, i, lens, q, out, sel, sc):
        wl = self.wl
        G, c, d = wl.group, wl.seg_len, wl.head_dim
        q64 = f64(q)
        out64 = f64(out)
        sel_np = sel.cpu().numpy()
        sc_np = sc.cpu().numpy()
        for (b, g) in self.groups:
            t = lens[b]
            ws, n_cand = orc.window_split(t, c, wl.window, self.n_sink)
            k_eff = min(wl.top_k, n_cand)
            union = set()
            own = {}
            for h in range(g * G, (g + 1) * G):
                phi_q = orc.random_features(q64[b, h], self.omega64)
                ora_sc = orc.segment_scores(phi_q, self.summ64[(b, g)][:n_cand])
                self.stats.band_swaps += check_selection(sel_np[b, h], ora_sc,
                                                         k_eff, n_cand)
                picks = [int(s) for s in sel_np[b, h, :k_eff]]
                own[h] = picks
                union.update(picks)
                if k_eff:
                    ref = ora_sc[picks]
                    err = float(np.max(np.abs(sc_np[b, h, :k_eff] - ref) / ref))
                    self.stats.max_score_err = max(self.stats.max_score_err, err)
                    assert err <= SCORE_TOL, (i, b, h, err)
                    got_order = sc_np[b, h, :k_eff]
                    assert np.all(got_order[:-1] >= got_order[1:]), got_order
            for h in range(g * G, (g + 1) * G):
                segs = own[h] if self.per_head else sorted(union)
                toks = orc.attended_tokens(segs, c, ws, t, self.n_sink)
                ref = orc.attend(q64[b, h], self.keys[(b, g)],
                                 self.vals[(b, g)], toks)
                e = rel_inf(out64[b, h], ref)
                self.stats.merge_out(e)
                assert e <= OUT_TOL[wl.dtype], (i, b, h, e)
                self.stats.heads += 1


def sample_groups(wl, n, seed=0):
    rng = np.random.default_rng(seed)
    allg = [(b, g) for b in range(wl.batch) for g in range(wl.n_kv_heads)]
    idx = rng.choice(len(allg), size=min(n, len(allg)), replace=False)
    return [allg[i] for i in sorted(idx)]
