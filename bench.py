"""Decode throughput of the Radar path on one MI355X.

A step is one pass of the whole path for one token of every sequence: the
append (k/v row write, plus the summary refresh when a segment fills) and the
decode (phi(q), segment scores, top-k, union, gather attention, combine) for
every (batch, query head), as one radar_append_decode call (or, with
--merged 0, radar_append followed by radar_decode). Inputs are seeded
synthetic tensors already resident in HBM; the default workload is the
long-context MHA layer: batch 8, 32 heads, head_dim 128, 128K context,
segment length 256, top-16 segments, 256 random features, recent window 256,
bf16 K/V, clustered keys.

Prints one JSON line: tokens/s (batch x steps / time) with the algorithmic
HBM bytes of the step, the roofline of the gather-attention kernel (per-launch
algorithmic K/V bytes over its event-timed duration), the index build's MFMA
utilisation, and the fp64 oracle timed on a bounded sample on the host.
"""
from __future__ import annotations

import argparse
import ctypes
import dataclasses
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2503_10571_amd as radar  # noqa: E402
import workloads  # noqa: E402

METRIC = ("decode attention tokens/sec (all heads) + achieved HBM GB/s at "
          "128K context")
HOST_LINK_PEAK_GBPS = 63.0      # PCIe 5.0 x16, one direction
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def window_split(t, c, w):
    ws = c * (max(0, t - w) // c)
    return ws, ws // c


class Stepper:
    """Direct C-ABI calls with pre-marshalled arguments (the per-step host
    cost stays small next to the GPU time)."""

    def __init__(self, cfg, inp, K, V, summ, ws, out, k, omega, sqrt_schedule=False,
                 exact=False, merged=True, extra_layers=()):
        self.L = radar.lib()
        # further layers (K, V, summaries) the token also passes through;
        # each step decodes it in every layer in turn (fixed schedule)
        P0 = ctypes.c_void_p
        self.extra = [(P0(a.data_ptr()), P0(b.data_ptr()), P0(c.data_ptr()))
                      for a, b, c in extra_layers]
        self.sqrt = sqrt_schedule
        self.exact = exact
        self.merged = merged
        self.restructures = 0
        self.cfg_c = cfg.c_struct()
        self.cfgp = ctypes.byref(self.cfg_c)
        self.inp = inp
        P = ctypes.c_void_p
        self.K, self.V = P(K.data_ptr()), P(V.data_ptr())
        self.om = P(omega.data_ptr())
        self.summ = P(summ.data_ptr())
        self.ws, self.ws_n = P(ws.data_ptr()), ws.numel()
        self.out = P(out.data_ptr())
        self.k = k
        self.stream = P(torch.cuda.current_stream().cuda_stream)
        self.kn = [P(inp.k_new[i].data_ptr()) for i in range(inp.k_new.shape[0])]
        self.vn = [P(inp.v_new[i].data_ptr()) for i in range(inp.v_new.shape[0])]
        self.q = [P(inp.q[i].data_ptr()) for i in range(inp.q.shape[0])]
        self.t0 = inp.wl.t0

    def step(self, i, sel=None):
        t = self.t0 + i
        if self.merged and not self.exact:
            c = math.isqrt(t + 1) if self.sqrt else self.cfg_c.seg_len
            if c == self.cfg_c.seg_len:       # no restructure at this token
                if self.sqrt:
                    self.cfg_c.window = t + 1 - c * c
                st = self.L.radar_append_decode(
                    self.cfgp, self.q[i], self.K, self.V, self.kn[i], self.vn[i],
                    self.om, self.summ, t + 1, None, self.k, self.out, sel, None,
                    self.ws, self.ws_n, self.stream)
                for (Kl, Vl, Sl) in self.extra:
                    st = st or self.L.radar_append_decode(
                        self.cfgp, self.q[i], Kl, Vl, self.kn[i], self.vn[i],
                        self.om, Sl, t + 1, None, self.k, self.out, None, None,
                        self.ws, self.ws_n, self.stream)
                if st:
                    raise radar.RadarError("radar_append_decode", st)
                return
        st = self.L.radar_append(self.cfgp, self.K, self.V, self.kn[i],
                                 self.vn[i], self.om, t, None, self.summ,
                                 self.stream)
        if st:
            raise radar.RadarError("radar_append", st)
        if self.sqrt:
            # Algorithm 1: c = floor(sqrt(t + 1)), W = [c^2, t + 1); rebuild
            # the summaries when t + 1 is a perfect square
            c = math.isqrt(t + 1)
            if c != self.cfg_c.seg_len:
                self.cfg_c.seg_len = c
                st = self.L.radar_build_index(self.cfgp, self.K, self.om, t + 1,
                                              self.summ, self.stream)
                if st:
                    raise radar.RadarError("radar_build_index", st)
                self.restructures += 1
            self.cfg_c.window = t + 1 - c * c
        for (Kl, Vl, Sl) in self.extra:
            st = self.L.radar_append(self.cfgp, Kl, Vl, self.kn[i], self.vn[i],
                                     self.om, t, None, Sl, self.stream)
            st = st or self.L.radar_decode(self.cfgp, self.q[i], Kl, Vl, self.om, Sl,
                                           t + 1, None, self.k, self.out, None, None,
                                           self.ws, self.ws_n, self.stream)
            if st:
                raise radar.RadarError("radar_append / radar_decode", st)
        if self.exact:
            st = self.L.radar_decode_exact(self.cfgp, self.q[i], self.K, self.V,
                                           t + 1, None, self.k, self.out, sel,
                                           None, self.ws, self.ws_n, self.stream)
        else:
            st = self.L.radar_decode(self.cfgp, self.q[i], self.K, self.V,
                                     self.om, self.summ, t + 1, None, self.k,
                                     self.out, sel, None, self.ws, self.ws_n,
                                     self.stream)
        if st:
            raise radar.RadarError("radar_decode", st)


def phase_clock_pass(stp, W, Ksteps, gpu, max_wgs=8192):
    """The timed steps once more with the fused kernel's phase stamps on:
    per step, the stamps of every workgroup of its (last) fused-kernel
    launch. Returns µs figures: the spread of the workgroups' start, the
    launch's span (first entry to last merge), each workgroup's total, and
    per phase the mean and max over workgroups (means over the steps)."""
    S = radar.CLOCK_STAMPS
    clocks = torch.empty(max_wgs, S, dtype=torch.int64, device=gpu)
    khz = radar.wall_clock_khz()
    if khz <= 0:
        return None
    to_us = 1e3 / khz
    rows = []
    radar.set_phase_clock(clocks)
    try:
        for j in range(Ksteps):
            clocks.fill_(-1)
            stp.step(W + j)
            torch.cuda.synchronize()
            c = clocks.cpu().numpy()
            c = c[c[:, 0] >= 0]
            if len(c):
                rows.append(c.astype(np.float64))
    finally:
        radar.set_phase_clock(None)
    if not rows:
        return None
    acc = {"start_skew": [], "span": [], "wg_mean": [], "wg_max": []}
    ph = {name: ([], []) for name in radar.CLOCK_PHASES}
    for c in rows:
        acc["start_skew"].append((c[:, 0].max() - c[:, 0].min()) * to_us)
        acc["span"].append((c[:, 6].max() - c[:, 0].min()) * to_us)
        tot = (c[:, 6] - c[:, 0]) * to_us
        acc["wg_mean"].append(tot.mean())
        acc["wg_max"].append(tot.max())
        for i, name in enumerate(radar.CLOCK_PHASES, start=1):
            d = (c[:, i] - c[:, i - 1]) * to_us
            ph[name][0].append(d.mean())
            ph[name][1].append(d.max())
    r = lambda v: round(float(np.mean(v)), 2)
    return {"unit": "us", "clock_khz": khz, "steps": len(rows),
            "workgroups": int(len(rows[-1])),
            "start_skew": r(acc["start_skew"]), "span": r(acc["span"]),
            "workgroup_total": {"mean": r(acc["wg_mean"]), "max": r(acc["wg_max"])},
            "phases": {name: {"mean": r(v[0]), "max": r(v[1])} for name, v in ph.items()}}


def union_stats(us):
    """min / mean / max of the per-pair union sizes of every timed step, and
    the mean over steps of each step's mean / max."""
    a = np.stack([np.asarray(u, dtype=np.float64) for u in us])
    return {"min": int(a.min()), "mean": round(float(a.mean()), 2), "max": int(a.max()),
            "mean_over_max": round(float(np.mean(a.mean(1) / np.maximum(a.max(1), 1))), 4)}


def union_sizes(sel, G):
    """sel [B][Hq][k] int32 -> union size per (b, kv head) [B * Hkv]."""
    B, Hq, k = sel.shape
    Hkv = Hq // G
    g = sel.reshape(B, Hkv, G * k)
    out = np.empty(B * Hkv, dtype=np.int64)
    for i, row in enumerate(g.reshape(B * Hkv, G * k)):
        out[i] = len(set(int(x) for x in row if x >= 0))
    return out


def step_bytes(wl, t, U, s_kv, sqrt_schedule=False, exact=False, s_om=4, n_sink=0):
    """Algorithmic HBM bytes of one step whose decode runs at length t (the
    append wrote row t - 1). U: union size per (b, kv head).
    Returns (whole step, decode call, K/V gather, candidate-key scan, row
    append, summary rows read); with exact=True the selection scans every candidate key
    instead of reading phi(q)'s inputs and the summaries. s_om: bytes per
    Omega entry; n_sink: attention-sink rows, always attended, after which
    the segments and the window start."""
    d, n = wl.head_dim, wl.n_features
    if sqrt_schedule:
        c, w = radar.schedule_sqrt(t)
    else:
        c, w = wl.seg_len, wl.window
    te = t - n_sink                    # tokens after the sinks
    ws, n_cand = window_split(te, c, w)
    W = te - ws
    BH = wl.batch * wl.n_kv_heads
    summ = BH * n_cand * n * 4
    kv = int(np.sum(U * c + W + n_sink)) * d * 2 * s_kv
    qo = wl.batch * wl.n_q_heads * d * 2 * s_kv
    om = n * d * s_om
    app = BH * 4 * d * s_kv            # read k_new, v_new; write both rows
    close = BH * (c * d * s_kv + n * 4) if te % c == 0 else 0
    if sqrt_schedule and w == 0:       # restructure: all t keys re-summarised
        close += BH * (t * d * s_kv + (t // c) * n * 4)
    scan = BH * n_cand * c * d * s_kv
    decode = (scan if exact else summ + om) + kv + qo
    return decode + app + close, decode, kv, scan, app, (0 if exact else summ)


def run_signature(line):
    """What fixes the HBM traffic of a launch relative to its algorithmic
    bytes besides the kernel source: the workload and the call form (the
    step range only scales both, one row per step)."""
    cfg = line["config"]
    sig = {"decode_path": cfg["decode_path"], "schedule": cfg["schedule"],
           "calls": cfg["calls"], "selector": cfg["selector"],
           "omega": cfg["omega"]}
    if cfg.get("kv", "device") != "device":
        sig["kv"] = cfg["kv"]
    if cfg.get("n_features_override"):
        sig["n_features"] = cfg["n_features"]
    for key, default in (("gqa_mode", "union"), ("n_sink", 0), ("layers", 1)):
        if cfg.get(key, default) != default:
            sig[key] = cfg[key]
    return sig


def source_sha256():
    """One hash over every file the library is built from."""
    import hashlib
    from paper_2503_10571_amd import _build
    h = hashlib.sha256()
    for path in _build.sources():
        h.update(os.path.relpath(path, ROOT).encode())
        h.update(open(path, "rb").read())
    return h.hexdigest()


def measured_traffic(kernel, workload, line, alg_bytes_per_launch, profiles=None):
    """HBM traffic per launch of `kernel` from the committed rocprofv3
    counter record: the record's FETCH_SIZE + WRITE_SIZE bytes (each divided
    by the scale a 1 GiB copy kernel shows) over its algorithmic bytes,
    times this run's algorithmic bytes per launch. FETCH_SIZE counts L2
    misses, so bytes served by the Infinity Cache count as traffic too.
    Returns (bytes, ratio), or None when there is no record, the library's
    sources have changed since it was taken, or it was taken with another
    call form."""
    path = os.path.join(profiles or os.path.join(ROOT, "profiles"),
                        f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("sources_sha256") != source_sha256():
        return None
    if rec.get("run") != run_signature(line):
        return None
    ratio = float(rec["traffic_ratio"])
    return int(ratio * alg_bytes_per_launch), ratio


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 0) for i in threadpool_info()
             if i.get("user_api") == "blas"]
        if n:
            return int(max(n))
    except Exception:
        pass
    return int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))


def _widen(x):
    """A torch tensor (fp32, or bf16 carried as its raw 16-bit words) as
    float64 numpy."""
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def _as_words(t):
    t = t.contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.float().numpy()


def oracle_worker(job):
    """The fp64 oracle on some (batch, q head) pairs of a workload, one BLAS
    thread: per decode step a segment-close refresh when one is due, then
    phi(q), scores, top-k and exact attention. Repeats its pass over the
    steps until min_s seconds of work (at most max_s). Returns (head-steps,
    seconds). Module level so that a process pool can run it."""
    try:
        from threadpoolctl import threadpool_limits
    except Exception:
        threadpool_limits = None
    if threadpool_limits is not None:
        with threadpool_limits(1):
            return _oracle_run(job)
    return _oracle_run(job)


def _oracle_run(job):
    from oracle import radar_oracle as orc
    (t0, first_step, n_steps, c, w, top_k, sqrt_schedule, om_words, pairs,
     min_s, max_s) = job
    om = _widen(om_words)
    state = []
    for (keys_w, vals_w, qs_w) in pairs:
        keys, vals, qs = _widen(keys_w), _widen(vals_w), _widen(qs_w)
        t_start = t0 + first_step
        c0 = orc.sqrt_schedule(t_start)[0] if sqrt_schedule else c
        summ = orc.segment_summaries(keys[:t_start], om, c0)  # index (untimed)
        state.append([keys, vals, qs, summ, summ])
    done, passes = 0, 0
    t_begin = time.perf_counter()
    while True:
        for st in state:
            st[3] = st[4]
        for i in range(n_steps):
            t = t0 + first_step + i + 1
            cs, ww = orc.sqrt_schedule(t) if sqrt_schedule else (c, w)
            for st in state:
                keys, vals, qs, summ, _ = st
                if sqrt_schedule and ww == 0:   # restructure at a square
                    st[3] = summ = orc.segment_summaries(keys[:t], om, cs)
                elif not sqrt_schedule and t % c == 0:
                    # the appended row closed a segment
                    new = orc.segment_summaries(keys[:t], om, c, first=t // c - 1)
                    st[3] = summ = np.concatenate([summ, new], 0)
                ws, n_cand = orc.window_split(t, cs, ww)
                phi_q = orc.random_features(qs[i], om)
                _, sel = orc.decode_head(phi_q, summ, n_cand, top_k)
                toks = orc.attended_tokens(sel, cs, ws, t)
                orc.attend(qs[i], keys, vals, toks)
                done += 1
            if time.perf_counter() - t_begin > max_s:
                break
        passes += 1
        el = time.perf_counter() - t_begin
        if el >= min_s or el > max_s:
            break
    return done, time.perf_counter() - t_begin


def cpu_baseline(wl, inp, first_step, n_steps, n_heads=4, min_s=8.0, max_s=20.0,
                 sqrt_schedule=False, workers=None):
    """The fp64 oracle (as it stands) timed on the host on a bounded sample
    of the timed steps: sampled (batch, q head) pairs, each decoded over the
    timed steps. Two timings, each scaled to the workload's tokens/s over
    all heads: one process with one BLAS thread on `n_heads` pairs, and a
    pool of one-thread worker processes, one per usable core (at most 16),
    each on its own pair; `value` is the pool's. The oracle's per-head loop
    is serial Python, so the pool is how it uses the cores."""
    import multiprocessing as mp
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") \
        else (os.cpu_count() or 1)
    P = max(1, min(cores, 16)) if workers is None else workers
    total = wl.batch * wl.n_q_heads
    rng = np.random.default_rng(5)
    n_pick = min(total, max(n_heads, P))
    pick = (np.arange(total) if n_pick >= total
            else np.sort(rng.choice(total, n_pick, replace=False)))
    pairs = [(int(i) // wl.n_q_heads, int(i) % wl.n_q_heads) for i in pick]
    last = first_step + n_steps
    data = []
    for b, h in pairs:
        g = h // wl.group
        data.append((_as_words(inp.keys_at(last, b, g)), _as_words(inp.values_at(last, b, g)),
                     _as_words(inp.q[first_step:last, b, h])))
    om = _as_words(inp.omega)
    common = (wl.t0, first_step, n_steps, wl.seg_len, wl.window, wl.top_k,
              sqrt_schedule, om)

    def per_token(done, sec):
        return wl.batch / (sec / done * total)

    # one process, one thread
    d1, s1 = oracle_worker(common + (data[:n_heads], min_s, max_s))
    one = per_token(d1, s1)
    # one worker per core, a pair each (the pairs cycle when there are fewer)
    jobs = [common + ([data[i % len(data)]], min_s, max_s) for i in range(P)]
    ctx = mp.get_context("spawn")
    t_begin = time.perf_counter()
    with ctx.Pool(P) as pool:
        res = pool.map(oracle_worker, jobs)
    wall = time.perf_counter() - t_begin
    done = sum(r[0] for r in res)
    busy = max(r[1] for r in res)
    allc = per_token(done, busy)
    return {"value": allc, "unit": "tokens/s", "cores": P, "kind": "oracle",
            "value_1_thread": one, "cores_affinity": cores,
            "cpu_count": os.cpu_count(), "blas_threads_per_process": 1,
            "sample": (f"{P} one-thread worker processes, each decoding one "
                       f"(batch, q head) pair ({len(data)} distinct pairs of "
                       f"{total}) over the {n_steps} timed steps until "
                       f"{min_s:.0f} s of work ({done} head-steps in "
                       f"{busy:.1f} s per worker, {wall:.1f} s with start-up); "
                       f"value_1_thread: one process, one thread, {min(n_heads, len(data))} "
                       f"pairs, {d1} head-steps in {s1:.1f} s; both scaled to all "
                       f"{total} heads; each pair's index build before the "
                       "sample is untimed")}


def recall_sweep(wl):
    """Recall of Radar's selection against the exact segment search at the
    workload's context length, for n in 64..2048 and k in 1..64, over the
    first decode query of the workload's inputs."""
    from paper_2503_10571_amd import recall
    log(f"[recall] generating {wl.name} inputs")
    inp = workloads.make_inputs(wl, "cuda", steps=1)
    cfg = radar.Config(wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                       wl.n_features, wl.seg_len, wl.window, wl.t0 + 1,
                       wl.torch_dtype())
    omegas = {n: workloads.make_omega(n, wl.head_dim, seed=1000 + n,
                                      dtype=wl.dtype, device="cuda")
              for n in (64, 128, 256, 512, 1024, 2048)}
    ks = [1, 2, 4, 8, 16, 32, 64]
    rows = recall.sweep(cfg, inp.q[0].contiguous(), inp.K, inp.V, wl.t0,
                        omegas, ks)
    for r in rows:
        r["workload"] = wl.name
        print(json.dumps(r), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default: the workload's step count)")
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default="mha_128k",
                    choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--cpu-baseline", type=int, default=1)
    ap.add_argument("--cpu-heads", type=int, default=4)
    ap.add_argument("--calibrate-copy", type=int, default=1,
                    help="also run a plain 1 GiB read+write elementwise "
                         "kernel: this GPU's copy bandwidth (and the counter "
                         "calibration for HBM traffic)")
    ap.add_argument("--merged", type=int, default=1,
                    help="1: one radar_append_decode call per step (the row "
                         "write runs inside the decode's first kernel); 0: "
                         "radar_append then radar_decode")
    ap.add_argument("--kernel-events", default="separate",
                    choices=["inline", "separate"],
                    help="per-kernel HIP event timing (the roofline's kernel "
                         "duration): separate = on a second pass over the same "
                         "steps, so the timed steps carry no event overhead; "
                         "inline = on the timed steps themselves (the event "
                         "pairs add host work per launch, which slows short "
                         "steps)")
    ap.add_argument("--graph", type=int, default=0,
                    help="1: capture the timed steps (the same library calls "
                         "as the eager loop) into one HIP graph and time its "
                         "replay, so host launch overhead is not timed; 0: "
                         "time the eager launches")
    ap.add_argument("--peaks", type=int, default=1,
                    help="measure the sustained bf16 MFMA and exp2 rates "
                         "(the index build's two resources)")
    ap.add_argument("--build-reps", type=int, default=3)
    ap.add_argument("--build-warmup", type=int, default=4,
                    help="untimed index builds before the timed ones")
    ap.add_argument("--path", default="auto",
                    choices=["auto", "split", "fused", "select", "scored"],
                    help="decode path (auto: the library's choice)")
    ap.add_argument("--selector", default="radar", choices=["radar", "exact"],
                    help="radar: Eq. 6 scores (the method); exact: the exact "
                         "segment search, every candidate key scanned")
    ap.add_argument("--recall", action="store_true",
                    help="instead of timing: recall of Radar's selection "
                         "against the exact search over n and k, one JSON "
                         "line per (n, k)")
    ap.add_argument("--gqa-mode", default="union", choices=["union", "per_head"],
                    help="grouped query heads attend their group's union, or "
                         "each its own selection")
    ap.add_argument("--sinks", type=int, default=0,
                    help="attention-sink rows at the start of the cache")
    ap.add_argument("--n-features", type=int, default=0,
                    help="random features n instead of the workload's "
                         "(64 ... 2048)")
    ap.add_argument("--kv-host", type=int, default=0,
                    help="1: the K/V cache in pinned host memory mapped for "
                         "the GPU; the decode gathers the selected segments "
                         "over the host link (reported as host_link)")
    ap.add_argument("--omega", default="auto", choices=["auto", "f32"],
                    help="auto: Omega passed as bf16 for bf16 caches (their "
                         "projection rounds it to bf16 anyway; same results, "
                         "half the Omega bytes), fp32 otherwise; f32: always "
                         "fp32")
    ap.add_argument("--layers", type=int, default=1,
                    help="layers the token passes through each step, each with "
                         "its own K/V cache and summaries (the same contents): "
                         "with two or more, a step's working set no longer "
                         "fits the Infinity Cache between its visits, as in a "
                         "multi-layer decode; tokens/s counts one token "
                         "through all layers")
    ap.add_argument("--phase-clock", type=int, default=0,
                    help="also replay the timed steps with the fused kernel's "
                         "per-workgroup phase stamps on (radar_set_phase_clock) "
                         "and report each phase's duration")
    ap.add_argument("--cold-pass", type=int, default=1,
                    help="also time the dominant kernel with the Infinity "
                         "Cache and L2 swept between steps (a 1 GiB "
                         "read-modify-write outside the event bracket)")
    ap.add_argument("--schedule", default="fixed", choices=["fixed", "sqrt"],
                    help="fixed: the workload's segment length and window; "
                         "sqrt: Algorithm 1's restructuring (c = sqrt(t) at "
                         "perfect squares, W = [c^2, t)), rebuilds timed")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the decode path runs on a single "
              "device (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if args.sinks and args.schedule == "sqrt":
        print("bench.py: --sinks with --schedule sqrt is not measured (the byte "
              "model's restructure term has no sinks)", file=sys.stderr)
        sys.exit(2)
    if args.layers < 1 or (args.layers > 1 and (args.schedule != "fixed" or
                                                  args.selector != "radar" or
                                                  args.kv_host or args.graph)):
        print("bench.py: --layers > 1 runs the fixed schedule, the radar selector "
              "and a device cache, eagerly", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    radar.set_decode_path({"auto": radar.PATH_AUTO, "split": radar.PATH_SPLIT,
                           "fused": radar.PATH_FUSED, "select": radar.PATH_SELECT,
                           "scored": radar.PATH_SCORED}[args.path])
    wl = workloads.WORKLOADS[args.workload]
    if args.n_features:
        # another feature count on the same keys and queries (Omega drawn at
        # that size)
        wl = wl.scaled(n_features=args.n_features)
    if args.recall:
        recall_sweep(wl)
        return
    exact = args.selector == "exact"
    W = args.warmup
    Ksteps = args.steps if args.steps is not None else wl.steps
    total = W + Ksteps
    log(f"[bench] generating {wl.name} inputs ({total} steps)")
    inp = workloads.make_inputs(wl, "cuda", steps=total)
    if args.schedule == "sqrt":
        c0, w0 = radar.schedule_sqrt(wl.t0)
        wl = wl.scaled(seg_len=c0, window=w0)
    omega = inp.omega
    if args.omega == "auto" and wl.dtype == "bf16":
        omega = inp.omega.to(torch.bfloat16)    # exact: the values are bf16
        assert torch.equal(omega.float(), inp.omega)
    cfg = radar.Config(wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                       wl.n_features, wl.seg_len, wl.window, wl.t0 + total,
                       wl.torch_dtype(), n_sink=args.sinks,
                       gqa_mode=(radar.GQA_PER_HEAD if args.gqa_mode == "per_head"
                                 else radar.GQA_UNION),
                       omega_dtype=omega.dtype)
    s_kv = 2 if wl.dtype == "bf16" else 4
    s_om = omega.element_size()
    K, V = inp.K, inp.V
    gpu = inp.K.device
    if args.kv_host:
        # the K/V cache in pinned host memory mapped for the GPU: the decode
        # reads only the selected segments, the window and the sinks over
        # the host link (the summaries, Omega and the workspace stay on the
        # GPU)
        K = torch.empty(inp.K.shape, dtype=inp.K.dtype, pin_memory=True)
        V = torch.empty(inp.V.shape, dtype=inp.V.dtype, pin_memory=True)
        K.copy_(inp.K)
        V.copy_(inp.V)
    summ = radar.new_summaries(cfg, gpu)
    if args.schedule == "sqrt":
        # the largest scratch any step of the run needs (window up to 2c)
        need = max(radar.workspace_bytes(
            dataclasses.replace(cfg, seg_len=radar.schedule_sqrt(t)[0],
                                window=radar.schedule_sqrt(t)[1]), wl.top_k)
            for t in range(wl.t0, wl.t0 + total + 1))
        ws = torch.empty(need, dtype=torch.uint8, device=gpu)
    else:
        ws = radar.new_workspace(cfg, wl.top_k, gpu)
    out = torch.empty_like(inp.q[0])
    torch.cuda.synchronize()

    # ---- index build (Eq. 4-5 over the whole prefix) --------------------
    log("[bench] index build")
    # untimed builds first: the first few run slower (about 3.3 against
    # 2.9 ms at the 128K shape) until the GPU has settled under load
    for _ in range(max(1, args.build_warmup)):
        radar.build_index(cfg, K, omega, wl.t0, summ)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.build_reps):
        radar.build_index(cfg, K, omega, wl.t0, summ)
    e1.record()
    torch.cuda.synchronize()
    build_ms = e0.elapsed_time(e1) / args.build_reps
    n_keys = wl.batch * wl.n_kv_heads * (wl.t0 // wl.seg_len) * wl.seg_len
    build_flop = 2.0 * n_keys * wl.n_features * wl.head_dim
    build_tflops = build_flop / (build_ms * 1e-3) / 1e12
    build_exps = n_keys * wl.n_features / (build_ms * 1e-3) / 1e12   # 10^12 / s

    # ---- decode steps ----------------------------------------------------
    merged = bool(args.merged) and not exact
    extra_layers = []
    for _ in range(args.layers - 1):
        # another layer: its own copy of the cache and of the summaries
        Kl, Vl, Sl = K.clone(), V.clone(), summ.clone()
        extra_layers.append((Kl, Vl, Sl))
    torch.cuda.synchronize()
    stp = Stepper(cfg, inp, K, V, summ, ws, out, wl.top_k, omega,
                  sqrt_schedule=args.schedule == "sqrt", exact=exact,
                  merged=merged, extra_layers=extra_layers)
    sel_log = torch.empty(Ksteps, wl.batch, wl.n_q_heads, wl.top_k,
                          dtype=torch.int32, device=gpu)
    log(f"[bench] warmup {W} steps")
    for i in range(W):
        stp.step(i)
    torch.cuda.synchronize()
    t_timed = wl.t0 + W
    seg_timed, win_timed = stp.cfg_c.seg_len, stp.cfg_c.window
    restr_before = stp.restructures

    def rewind():
        # the steps are replayed from the same state: their appends rewrite
        # the same rows, their refreshes the same summaries; the sqrt
        # schedule needs its (c, w) and summaries of the pass's start
        if args.schedule == "sqrt":
            stp.cfg_c.seg_len, stp.cfg_c.window = seg_timed, win_timed
            radar.build_index(dataclasses.replace(cfg, seg_len=seg_timed,
                                                  window=win_timed),
                              K, omega, t_timed, summ)
        torch.cuda.synchronize()

    def profiled_pass(flush=None):
        # flush: a buffer swept (read and written) between steps, outside the
        # kernels' event brackets, so that every step starts with the
        # Infinity Cache and the L2s holding none of the step's data
        radar.profile_enable(True)
        for j in range(Ksteps):
            if flush is not None:
                flush.add_(1)
            stp.step(W + j)
        torch.cuda.synchronize()
        p = radar.profile_read()
        radar.profile_enable(False)
        return p

    inline = args.kernel_events == "inline" and not args.graph
    if inline:
        # an untimed profiled pass first: it creates the event pairs the
        # timed pass then reuses, so no event is created while timing
        profiled_pass()
        rewind()
        restr_before = stp.restructures
    log(f"[bench] timing {Ksteps} steps" + (" (graph replay)" if args.graph else ""))
    sel_ptrs = [ctypes.c_void_p(sel_log[j].data_ptr()) for j in range(Ksteps)]
    if args.graph:
        # capture records the launches without running them; the replay runs
        # exactly the steps the eager loop would
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            stp.stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
            for j in range(Ksteps):
                stp.step(W + j, sel_ptrs[j])
        stp.stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        e0.record()
        graph.replay()
        e1.record()
    else:
        # inline: every launch of the timed steps is bracketed by HIP events
        # (hipExtLaunchKernel) on its own stream
        radar.profile_enable(inline)
        e0.record()
        for j in range(Ksteps):
            stp.step(W + j, sel_ptrs[j])
        e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    ms_step = ms / Ksteps
    restructures = stp.restructures - restr_before
    if inline:
        prof = radar.profile_read()
        radar.profile_enable(False)
    else:
        # the same steps again with every kernel bracketed by HIP events
        rewind()
        prof = profiled_pass()
    phases = None
    if args.phase_clock:
        log("[bench] phase-clock pass")
        rewind()
        phases = phase_clock_pass(stp, W, Ksteps, gpu)
    prof_cold = None
    if args.cold_pass and not args.kv_host:
        log("[bench] cold pass: 1 GiB swept between steps")
        rewind()
        flush = torch.zeros(1 << 28, dtype=torch.int32, device=gpu)
        prof_cold = profiled_pass(flush)
        del flush

    # ---- algorithmic bytes ------------------------------------------------
    sel_np = sel_log.cpu().numpy()
    tot_bytes, dec_bytes, kv_bytes, scan_bytes, summ_bytes = 0, 0, 0, 0, 0
    NL = args.layers           # every layer moves the same bytes
    u_all = []
    for j in range(Ksteps):
        t = wl.t0 + W + j + 1
        U = union_sizes(sel_np[j], wl.group)
        u_all.append(U)
        b_all, b_dec, b_kv, b_scan, b_app, b_summ = (NL * x for x in step_bytes(
            wl, t, U, s_kv, sqrt_schedule=args.schedule == "sqrt", exact=exact,
            s_om=s_om, n_sink=args.sinks))
        tot_bytes += b_all
        # with the merged call the fused kernel also does the row append
        dec_bytes += b_dec + (b_app if merged else 0)
        kv_bytes += b_kv
        scan_bytes += b_scan
        summ_bytes += b_summ
    step_gbps = tot_bytes / (ms * 1e-3) / 1e9
    path = radar.decode_path(dataclasses.replace(cfg, seg_len=seg_timed,
                                                 window=win_timed),
                             wl.t0 + W + 1, wl.top_k)
    # dominant kernel: the fused decode (all decode bytes), or on the split
    # path the longer of the gather attention (the K/V bytes) and the score
    # pass (the summary rows; the longer one for large n)
    if exact:
        # the exact selector runs the split path; its key scan dominates
        path = radar.PATH_SPLIT
        dom, dom_name, dom_bytes = "score", "k_segment_mass", scan_bytes
    elif path == radar.PATH_FUSED:
        dom, dom_name, dom_bytes = "fused", "k_decode_fused", dec_bytes
    elif path == radar.PATH_SCORED:
        # the fused kernel from its top-k on: the K/V gather (and the rows the
        # merged call appends)
        dom, dom_name = "scored", "k_decode_fused_scored"
        dom_bytes = kv_bytes + (NL * Ksteps * wl.batch * wl.n_kv_heads * 4 * wl.head_dim
                                * s_kv if merged else 0)
    else:
        dom, dom_name, dom_bytes = "attend", "k_attend", kv_bytes
        avg = {k: prof[k][0] / max(prof[k][1], 1) for k in ("attend", "score")}
        if prof["score"][1] and avg["score"] > avg["attend"]:
            dom, dom_name, dom_bytes = "score", "k_score", summ_bytes
    dom_ms, dom_n = prof[dom]
    dom_avg_ms = dom_ms / max(dom_n, 1)
    per_launch = dom_bytes / (Ksteps * NL)     # one launch per layer and step
    dom_gbps = per_launch / (dom_avg_ms * 1e-3) / 1e9
    tokens_s = wl.batch * Ksteps / (ms * 1e-3)
    cold = None
    if prof_cold is not None and prof_cold[dom][1]:
        c_avg = prof_cold[dom][0] / prof_cold[dom][1]
        c_gbps = per_launch / (c_avg * 1e-3) / 1e9
        cold = {"avg_us": round(c_avg * 1e3, 2), "achieved": round(c_gbps, 1),
                "frac": round(c_gbps / HBM_PEAK_GBPS, 4),
                "sweep": "1 GiB read and written between steps, outside the "
                         "event bracket (evicts the 256 MB Infinity Cache and "
                         "the L2s)"}

    kern = {k: {"avg_us": round(v[0] / max(v[1], 1) * 1e3, 2), "launches": v[1]}
            for k, v in prof.items() if v[1]}
    log("[bench] kernels: " + json.dumps(kern))

    cpu = None
    # the oracle's timing covers the default options only
    if args.cpu_baseline and not exact and args.sinks == 0 and args.gqa_mode == "union" \
            and NL == 1:
        log("[bench] cpu baseline (fp64 oracle)")
        cpu = cpu_baseline(wl, inp, W, Ksteps, n_heads=args.cpu_heads,
                           sqrt_schedule=args.schedule == "sqrt")

    copy_gbps = None
    if args.calibrate_copy:
        # torch.neg over 1 GiB fp32: reads 1 GiB, writes 1 GiB
        x = torch.ones(1 << 28, dtype=torch.float32, device=gpu)
        y = torch.empty_like(x)
        torch.neg(x, out=y)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(5):
            torch.neg(x, out=y)
        e1.record()
        torch.cuda.synchronize()
        copy_gbps = 2 * x.numel() * 4 * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9
        log(f"[bench] copy kernel (1 GiB read + 1 GiB write): {copy_gbps:.1f} GB/s")
        del x, y

    peaks = radar.peak_rates() if args.peaks else None
    read_gbps = None
    if args.peaks:
        del extra_layers
        stp.extra = []
        torch.cuda.empty_cache()
        read_gbps = radar.peak_read_gbps()
        log(f"[bench] non-temporal read stream: {read_gbps:.1f} GB/s")

    line = {
        "metric": METRIC,
        "value": round(tokens_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": Ksteps,
        "warmup": W,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {
            "workload": (f"{wl.name}: batch {wl.batch}, {wl.n_q_heads} q / "
                         f"{wl.n_kv_heads} kv heads, head_dim {wl.head_dim}, "
                         f"context {wl.t0}+, c {wl.seg_len}, top-k "
                         f"{wl.top_k}, n {wl.n_features}, window {wl.window}, "
                         f"{wl.dtype} K/V, {wl.keys} keys"),
            "batch": wl.batch, "context": wl.t0, "seg_len": wl.seg_len,
            "top_k": wl.top_k, "n_features": wl.n_features,
            "window": wl.window,
            "decode_path": {radar.PATH_SPLIT: "split", radar.PATH_FUSED: "fused",
                            radar.PATH_SELECT: "select",
                            radar.PATH_SCORED: "scored"}.get(path, "?"),
            "schedule": args.schedule,
            "launch": "hip graph replay" if args.graph else "eager",
            "kernel_events": ("inline" if args.kernel_events == "inline" and not args.graph
                              else "separate pass"),
            "calls": ("radar_append_decode" if merged
                      else "radar_append + radar_decode"),
            "selector": args.selector,
            "omega": "bf16" if s_om == 2 else "f32",
            "kv": "pinned host memory" if args.kv_host else "device",
            "n_features_override": bool(args.n_features),
            "gqa_mode": args.gqa_mode,
            "n_sink": args.sinks,
            "restructures": restructures,
            "layers": NL,
        },
        "hbm_GBps": round(step_gbps, 1),
        "hbm_frac": round(step_gbps / HBM_PEAK_GBPS, 4),
        "bytes_per_step": int(tot_bytes // Ksteps),
        "roofline": {
            "kernel": dom_name,
            "bound": "hbm",
            "achieved": round(dom_gbps, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(dom_gbps / HBM_PEAK_GBPS, 4),
            "traffic": None,              # filled in below
            "bytes_per_launch": int(per_launch),
            "avg_us": round(dom_avg_ms * 1e3, 2),
            "cold_cache": cold,
        },
        "phase_clock": phases,
        "kernels_us": {k: v["avg_us"] for k, v in kern.items()},
        # segments attended per (b, kv head) over the timed steps: a pair's
        # share of the attention is proportional to it, so mean / max bounds
        # how evenly the pairs' workgroups finish
        "union_segments": union_stats(u_all),
        "index_build": {
            "ms": round(build_ms, 3),
            "warmup_builds": max(1, args.build_warmup),
            "tflops": round(build_tflops, 1),
            "mfma_frac": round(build_tflops / BF16_MFMA_PEAK_TFLOPS, 4),
            "keys": n_keys,
            "exp2_T_per_s": round(build_exps, 3),
            "mfma_peak_measured_tflops": round(peaks["mfma_tflops"], 1) if peaks else None,
            "mfma_frac_of_measured": round(build_tflops / peaks["mfma_tflops"], 4) if peaks else None,
            "exp2_peak_measured_T_per_s": round(peaks["exp_T_per_s"], 3) if peaks else None,
            "exp2_frac_of_measured": round(build_exps / peaks["exp_T_per_s"], 4) if peaks else None,
        },
        "cpu_baseline": cpu,
    }
    tr = measured_traffic(dom_name, wl.name, line, per_launch)
    if tr is not None:
        line["roofline"]["traffic"] = tr[0]
        line["roofline"]["traffic_ratio"] = round(tr[1], 4)
        line["roofline"]["traffic_counter"] = (
            "rocprofv3 FETCH_SIZE + WRITE_SIZE (L2-miss bytes: Infinity Cache "
            "hits count too), scaled by a copy kernel's reading")
    if read_gbps is not None:
        line["roofline"]["read_peak_GBps"] = round(read_gbps, 1)
        line["roofline"]["frac_of_read_peak"] = round(dom_gbps / read_gbps, 4)
    if args.kv_host:
        # the K/V rows each step gathers (selected segments, window, sinks)
        # cross the host link; its reference rate is PCIe 5.0 x16, one way
        kv_step = kv_bytes / Ksteps
        line["host_link"] = {
            "kv_bytes_per_step": int(kv_step),
            "achieved": round(kv_step / (ms_step * 1e-3) / 1e9, 2),
            "peak": HOST_LINK_PEAK_GBPS, "unit": "GB/s",
            "frac": round(kv_step / (ms_step * 1e-3) / 1e9 / HOST_LINK_PEAK_GBPS, 4),
        }
    if copy_gbps is not None:
        line["copy_GBps"] = round(copy_gbps, 1)
        line["roofline"]["frac_of_copy"] = round(dom_gbps / copy_gbps, 4)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
