"""Radar decode path on MI355X: Python binding of the C ABI in include/radar.h.

The binding only marshals arguments: every step of the path (index build,
append, phi(q), segment scores, top-k, union, gather-attention, combine) runs
in the HIP kernels of libradar.so. torch supplies device memory and the
stream (the current torch stream of the tensors' device). There is no CPU
fallback: a missing library raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libradar.so")

ABI_VERSION = 7
# bytes of the library's own decode scratch (RADAR_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 32 << 20
RADAR_F32, RADAR_BF16 = 0, 1
GQA_UNION, GQA_PER_HEAD = 0, 1
STATUS = {0: "ok", 1: "invalid argument", 2: "position outside the cache capacity",
          3: "shape outside the instantiated kernels", 4: "HIP launch failed",
          5: "workspace missing or too small"}


class RadarError(RuntimeError):
    def __init__(self, fn, status, detail=""):
        self.status = status
        msg = f"{fn}: {STATUS.get(status, status)}"
        if detail:
            msg += f" ({detail})"
        super().__init__(msg)


class _Config(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("n_features", ctypes.c_int32), ("seg_len", ctypes.c_int32),
                ("window", ctypes.c_int32), ("capacity", ctypes.c_int64),
                ("kv_dtype", ctypes.c_int32), ("n_sink", ctypes.c_int32),
                ("gqa_mode", ctypes.c_int32), ("omega_dtype", ctypes.c_int32)]


@dataclasses.dataclass(frozen=True)
class Config:
    """Shape of one Radar layer (mirrors radar_config). n_sink: leading
    attention-sink tokens (always attended, in no segment); gqa_mode:
    GQA_UNION (each query head attends its group's union) or GQA_PER_HEAD
    (its own selection); omega_dtype: the element type of the Omega tensor
    passed to every call (torch.bfloat16 only with a bf16 cache, whose
    projection rounds Omega to bf16 anyway: the same results from half the
    Omega bytes)."""
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_features: int
    seg_len: int
    window: int
    capacity: int
    dtype: torch.dtype = torch.bfloat16
    n_sink: int = 0
    gqa_mode: int = GQA_UNION
    omega_dtype: torch.dtype = torch.float32

    def c_struct(self) -> _Config:
        codes = {torch.float32: RADAR_F32, torch.bfloat16: RADAR_BF16}
        return _Config(self.batch, self.n_q_heads, self.n_kv_heads,
                       self.head_dim, self.n_features, self.seg_len,
                       self.window, self.capacity, codes[self.dtype], self.n_sink,
                       self.gqa_mode, codes[self.omega_dtype])

    @property
    def summary_rows(self) -> int:
        return self.capacity // self.seg_len


_lib = None
_P = ctypes.c_void_p


def lib() -> ctypes.CDLL:
    """The loaded libradar.so (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2503_10571_amd._build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        L.radar_abi_version.restype = ctypes.c_int32
        if L.radar_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI {L.radar_abi_version()}, "
                               f"this binding expects {ABI_VERSION}: rebuild it")
        cfgp = ctypes.POINTER(_Config)
        i64, i32, sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
        L.radar_build_index.argtypes = [cfgp, _P, _P, i64, _P, _P]
        L.radar_append.argtypes = [cfgp, _P, _P, _P, _P, _P, i64, _P, _P, _P]
        L.radar_decode.argtypes = [cfgp, _P, _P, _P, _P, _P, i64, _P, i32, _P,
                                   _P, _P, _P, sz, _P]
        L.radar_decode_exact.argtypes = [cfgp, _P, _P, _P, i64, _P, i32, _P, _P,
                                         _P, _P, sz, _P]
        L.radar_append_decode.argtypes = [cfgp, _P, _P, _P, _P, _P, _P, _P, i64,
                                          _P, i32, _P, _P, _P, _P, sz, _P]
        L.radar_append_decode_noalloc.argtypes = [cfgp, _P, _P, _P, _P, _P, _P,
                                                  _P, i64, _P, i32, _P, _P, _P, _P]
        L.radar_segment_mass.argtypes = [cfgp, _P, _P, i64, _P, _P, _P]
        L.radar_decode_workspace_bytes.argtypes = [cfgp, i32]
        L.radar_decode_workspace_bytes.restype = sz
        L.radar_attend_selected.argtypes = [cfgp, _P, _P, _P, _P, i32, i64, _P,
                                            _P, _P, sz, _P]
        L.radar_status_string.argtypes = [ctypes.c_int]
        L.radar_status_string.restype = ctypes.c_char_p
        L.radar_last_error.restype = ctypes.c_char_p
        L.radar_profile_enable.argtypes = [i32]
        L.radar_set_phase_clock.argtypes = [_P, i32]
        L.radar_wall_clock_khz.restype = i64
        L.radar_schedule_sqrt.argtypes = [i64, ctypes.POINTER(i32),
                                          ctypes.POINTER(i32)]
        L.radar_schedule_sqrt.restype = ctypes.c_int
        L.radar_set_decode_path.argtypes = [i32]
        L.radar_set_decode_path.restype = ctypes.c_int
        L.radar_decode_path.argtypes = [cfgp, i64, i32]
        L.radar_decode_path.restype = i32
        L.radar_profile_read.argtypes = [ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_int64), i32]
        L.radar_peak_sink_floats.restype = sz
        L.radar_peak_mfma.argtypes = [i32, _P, ctypes.POINTER(ctypes.c_double), _P]
        L.radar_peak_read.argtypes = [_P, sz, _P, _P]
        L.radar_peak_read.restype = ctypes.c_int
        L.radar_peak_exp.argtypes = [i32, _P, ctypes.POINTER(ctypes.c_double), _P]
        for fn in ("radar_peak_mfma", "radar_peak_exp"):
            getattr(L, fn).restype = ctypes.c_int
        for fn in ("radar_build_index", "radar_append", "radar_decode",
                   "radar_append_decode", "radar_append_decode_noalloc",
                   "radar_decode_exact", "radar_segment_mass",
                   "radar_attend_selected",
                   "radar_profile_enable", "radar_profile_read"):
            getattr(L, fn).restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(x):
    return None if x is None else ctypes.c_void_p(x.data_ptr())


def _stream(x):
    return ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream)


def _check(fn, st):
    if st != 0:
        detail = lib().radar_last_error().decode() if st == 4 else ""
        raise RadarError(fn, st, detail)


class _PtrAttr(ctypes.Structure):
    # hipPointerAttribute_t
    _fields_ = [("type", ctypes.c_int), ("device", ctypes.c_int),
                ("devicePointer", ctypes.c_void_p), ("hostPointer", ctypes.c_void_p),
                ("isManaged", ctypes.c_int), ("allocationFlags", ctypes.c_uint)]


_hip_rt = None


def _device_mapped(x) -> bool:
    """A pinned host tensor whose pages the GPU reaches at the same address
    (hipHostMalloc memory, as torch's pin_memory=True allocates it)."""
    global _hip_rt
    if not x.is_pinned():
        return False
    if _hip_rt is None:
        _hip_rt = ctypes.CDLL("libamdhip64.so")
    a = _PtrAttr()
    st = _hip_rt.hipPointerGetAttributes(ctypes.byref(a), ctypes.c_void_p(x.data_ptr()))
    return st == 0 and a.devicePointer == x.data_ptr()


def _need(x, dtype, name, numel=None, at_least=False, host_ok=False):
    """Device, dtype and layout checks; numel: the element count the kernels
    address for this argument (exactly, or at least with at_least), so that
    a tensor of the wrong size is refused before any kernel reads or writes
    past its end. host_ok also accepts pinned host memory mapped for the
    device (the K/V cache only)."""
    if not x.is_cuda and not (host_ok and _device_mapped(x)):
        raise ValueError(f"{name} must be a device tensor" +
                         (" or pinned host memory mapped for the device" if host_ok else ""))
    if x.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {x.dtype}")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and (x.numel() < numel if at_least else x.numel() != numel):
        raise ValueError(f"{name} holds {x.numel()} elements, the config needs "
                         f"{'at least ' if at_least else ''}{numel}")


def _cache(cfg, K, V=None):
    """K and V may sit in device memory or in pinned, device-mapped host
    memory (the decode then reads only the selected segments' rows, and the
    window's, over the host link)."""
    n = cfg.batch * cfg.n_kv_heads * cfg.capacity * cfg.head_dim
    _need(K, cfg.dtype, "K", n, host_ok=True)
    if V is not None:
        _need(V, cfg.dtype, "V", n, host_ok=True)


def _rows(cfg, k_new, v_new):
    n = cfg.batch * cfg.n_kv_heads * cfg.head_dim
    _need(k_new, cfg.dtype, "k_new", n)
    _need(v_new, cfg.dtype, "v_new", n)


def _query(cfg, q):
    _need(q, cfg.dtype, "q", cfg.batch * cfg.n_q_heads * cfg.head_dim)


def _omega(cfg, omega):
    _need(omega, cfg.omega_dtype, "omega", cfg.n_features * cfg.head_dim)


def _summ(cfg, summaries):
    rows = max(1, cfg.summary_rows)
    _need(summaries, torch.float32, "summaries",
          cfg.batch * cfg.n_kv_heads * rows * cfg.n_features, at_least=True)


def workspace_bytes(cfg: Config, k: int) -> int:
    return int(lib().radar_decode_workspace_bytes(ctypes.byref(cfg.c_struct()), k))


def new_workspace(cfg: Config, k: int, device) -> torch.Tensor:
    n = workspace_bytes(cfg, k)
    if n == 0:
        raise RadarError("radar_decode_workspace_bytes", 1)
    return torch.empty(n, dtype=torch.uint8, device=device)


def new_summaries(cfg: Config, device) -> torch.Tensor:
    return torch.zeros(cfg.batch, cfg.n_kv_heads, max(1, cfg.summary_rows),
                       cfg.n_features, dtype=torch.float32, device=device)


def build_index(cfg: Config, K, omega, t: int, summaries) -> None:
    """radar_build_index: summaries of the floor(t / c) full segments."""
    _cache(cfg, K); _omega(cfg, omega); _summ(cfg, summaries)
    _check("radar_build_index", lib().radar_build_index(
        ctypes.byref(cfg.c_struct()), _ptr(K), _ptr(omega), t, _ptr(summaries),
        _stream(summaries)))


def _lens(x, cfg: Config, name):
    """Optional per-sequence int64 [B] device array."""
    if x is None:
        return None
    _need(x, torch.int64, name)
    if x.numel() != cfg.batch:
        raise ValueError(f"{name} must hold batch = {cfg.batch} lengths")
    return x


def append(cfg: Config, K, V, k_new, v_new, omega, t: int, summaries,
           pos=None) -> None:
    """radar_append: write row t (or row pos[b] of sequence b); refresh the
    summary of a segment the row completes."""
    _cache(cfg, K, V); _rows(cfg, k_new, v_new)
    _omega(cfg, omega); _summ(cfg, summaries)
    pos = _lens(pos, cfg, "pos")
    _check("radar_append", lib().radar_append(
        ctypes.byref(cfg.c_struct()), _ptr(K), _ptr(V), _ptr(k_new), _ptr(v_new),
        _ptr(omega), t, _ptr(pos), _ptr(summaries), _stream(summaries)))


def _outputs(cfg, q, k, out, selected, scores, workspace):
    if out is None:
        out = torch.empty_like(q)
    _need(out, cfg.dtype, "out", cfg.batch * cfg.n_q_heads * cfg.head_dim)
    if workspace is None:
        workspace = new_workspace(cfg, k, q.device)
    _need(workspace, torch.uint8, "workspace")
    n_sel = cfg.batch * cfg.n_q_heads * k
    if selected is not None:
        _need(selected, torch.int32, "selected", n_sel, at_least=True)
    if scores is not None:
        _need(scores, torch.float32, "scores", n_sel, at_least=True)
    return out, workspace


def decode(cfg: Config, q, K, V, omega, summaries, t: int, k: int, out=None,
           selected=None, scores=None, workspace=None, lens=None):
    """radar_decode: one query per (b, q head) at context length t (or at
    lens[b] <= t per sequence). Returns out (and writes the optional
    selected / scores tensors)."""
    _query(cfg, q); _cache(cfg, K, V); _omega(cfg, omega); _summ(cfg, summaries)
    lens = _lens(lens, cfg, "lens")
    out, workspace = _outputs(cfg, q, k, out, selected, scores, workspace)
    _check("radar_decode", lib().radar_decode(
        ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(K), _ptr(V), _ptr(omega),
        _ptr(summaries), t, _ptr(lens), k, _ptr(out), _ptr(selected),
        _ptr(scores), _ptr(workspace), workspace.numel(), _stream(q)))
    return out


def append_decode(cfg: Config, q, K, V, k_new, v_new, omega, summaries,
                  t: int, k: int, out=None, selected=None, scores=None,
                  workspace=None, pos=None):
    """radar_append_decode: append row t - 1 (row pos[b] of sequence b) and
    decode at context length t (pos[b] + 1, bounded by t) in one call, the
    same result as append(..., t - 1, pos=pos) then decode(..., t,
    lens=pos + 1). Returns out."""
    _query(cfg, q); _cache(cfg, K, V); _rows(cfg, k_new, v_new)
    _omega(cfg, omega); _summ(cfg, summaries)
    pos = _lens(pos, cfg, "pos")
    out, workspace = _outputs(cfg, q, k, out, selected, scores, workspace)
    _check("radar_append_decode", lib().radar_append_decode(
        ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(K), _ptr(V), _ptr(k_new),
        _ptr(v_new), _ptr(omega), _ptr(summaries), t, _ptr(pos), k, _ptr(out),
        _ptr(selected), _ptr(scores), _ptr(workspace), workspace.numel(),
        _stream(q)))
    return out


def append_decode_noalloc(cfg: Config, q, K, V, k_new, v_new, omega, summaries,
                          t: int, k: int, out, selected=None, scores=None,
                          pos=None):
    """radar_append_decode_noalloc: append_decode() with the decode's scratch
    in the library's own device array instead of a workspace (for callers
    that cannot allocate: nothing is allocated here either, so `out` must be
    given). Calls that may overlap on one GPU must be serialised."""
    _query(cfg, q); _cache(cfg, K, V); _rows(cfg, k_new, v_new)
    _omega(cfg, omega); _summ(cfg, summaries)
    pos = _lens(pos, cfg, "pos")
    if out is None:
        raise ValueError("out must be given (this call allocates nothing)")
    _need(out, cfg.dtype, "out", cfg.batch * cfg.n_q_heads * cfg.head_dim)
    n_sel = cfg.batch * cfg.n_q_heads * k
    if selected is not None:
        _need(selected, torch.int32, "selected", n_sel, at_least=True)
    if scores is not None:
        _need(scores, torch.float32, "scores", n_sel, at_least=True)
    _check("radar_append_decode_noalloc", lib().radar_append_decode_noalloc(
        ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(K), _ptr(V), _ptr(k_new),
        _ptr(v_new), _ptr(omega), _ptr(summaries), t, _ptr(pos), k, _ptr(out),
        _ptr(selected), _ptr(scores), _stream(q)))
    return out


def decode_exact(cfg: Config, q, K, V, t: int, k: int, out=None,
                 selected=None, scores=None, workspace=None, lens=None):
    """radar_decode_exact: top-k segments by exact attention mass, then the
    same attention as decode(). scores receives ln(beta) of the picks."""
    _query(cfg, q); _cache(cfg, K, V)
    lens = _lens(lens, cfg, "lens")
    out, workspace = _outputs(cfg, q, k, out, selected, scores, workspace)
    _check("radar_decode_exact", lib().radar_decode_exact(
        ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(K), _ptr(V), t, _ptr(lens),
        k, _ptr(out), _ptr(selected), _ptr(scores), _ptr(workspace),
        workspace.numel(), _stream(q)))
    return out


def segment_mass(cfg: Config, q, K, t: int, lens=None, out=None):
    """radar_segment_mass: ln(beta_s) of every candidate segment and, at
    index n_cand, of the window and sinks, per (b, q head):
    [B][Hq][capacity / c + 1] fp32 (entries after n_cand unwritten)."""
    _query(cfg, q); _cache(cfg, K)
    lens = _lens(lens, cfg, "lens")
    rows = cfg.summary_rows + 1
    if out is None:
        out = torch.full((cfg.batch, cfg.n_q_heads, rows), float("nan"),
                         dtype=torch.float32, device=q.device)
    _need(out, torch.float32, "ln_beta", cfg.batch * cfg.n_q_heads * rows)
    _check("radar_segment_mass", lib().radar_segment_mass(
        ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(K), t, _ptr(lens), _ptr(out),
        _stream(q)))
    return out


def attend_selected(cfg: Config, q, K, V, selected, t: int, out=None,
                    workspace=None, lens=None):
    """radar_attend_selected: exact attention over given segment ids plus
    the sinks and W."""
    _query(cfg, q); _cache(cfg, K, V)
    k = selected.shape[-1]
    _need(selected, torch.int32, "selected", cfg.batch * cfg.n_q_heads * k)
    lens = _lens(lens, cfg, "lens")
    out, workspace = _outputs(cfg, q, k, out, None, None, workspace)
    _check("radar_attend_selected", lib().radar_attend_selected(
        ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(K), _ptr(V), _ptr(selected),
        k, t, _ptr(lens), _ptr(out), _ptr(workspace), workspace.numel(),
        _stream(q)))
    return out


KERNELS = ("append", "build", "phi_q", "score", "topk", "attend", "combine",
           "fused", "select", "scored")


def schedule_sqrt(t: int):
    """Algorithm 1's restructuring schedule at context length t: (segment
    length c = floor(sqrt(t)), window t - c^2)."""
    c, w = ctypes.c_int32(), ctypes.c_int32()
    _check("radar_schedule_sqrt", lib().radar_schedule_sqrt(t, ctypes.byref(c),
                                                            ctypes.byref(w)))
    return c.value, w.value


PATH_AUTO, PATH_SPLIT, PATH_FUSED, PATH_SELECT, PATH_SCORED = 0, 1, 2, 3, 4


def set_decode_path(path: int) -> None:
    """Force the split, fused, select or scored decode path on this thread
    (PATH_AUTO = automatic)."""
    _check("radar_set_decode_path", lib().radar_set_decode_path(path))


def decode_path(cfg: Config, t: int, k: int) -> int:
    """The path radar_decode takes for this shape, t and k."""
    return int(lib().radar_decode_path(ctypes.byref(cfg.c_struct()), t, k))


def profile_enable(on: bool) -> None:
    """Bracket every library kernel with a HIP event pair (measurement only)."""
    _check("radar_profile_enable", lib().radar_profile_enable(1 if on else 0))


def profile_read() -> dict:
    """{kernel: (total ms, launches)} of the kernels recorded since the last
    read; waits for them to finish."""
    n = len(KERNELS)
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int64 * n)()
    _check("radar_profile_read", lib().radar_profile_read(ms, cnt, n))
    return {k: (ms[i], cnt[i]) for i, k in enumerate(KERNELS)}


CLOCK_STAMPS = 8
# radar_set_phase_clock's stamps: the phase that ends at stamp i (i >= 1)
CLOCK_PHASES = ("phi_q", "scores", "topk_window", "union", "segment_tiles", "merge")


def set_phase_clock(clocks=None) -> None:
    """radar_set_phase_clock (measurement only): while `clocks` (a device
    int64 tensor [max_wgs][CLOCK_STAMPS]) is set, every fused-kernel launch
    from this thread writes its workgroups' phase stamps there; None stops."""
    if clocks is None:
        _check("radar_set_phase_clock", lib().radar_set_phase_clock(None, 0))
        return
    if (clocks.dtype != torch.int64 or clocks.dim() != 2 or
            clocks.shape[1] != CLOCK_STAMPS or not clocks.is_cuda or
            not clocks.is_contiguous()):
        raise ValueError("clocks: a contiguous device int64 tensor [max_wgs][8]")
    _check("radar_set_phase_clock",
           lib().radar_set_phase_clock(_ptr(clocks), clocks.shape[0]))


def wall_clock_khz() -> int:
    """Rate of the clock behind the phase stamps (kHz)."""
    return int(lib().radar_wall_clock_khz())


def peak_rates(device="cuda", iters=4096) -> dict:
    """Measured sustained dense bf16 MFMA rate (TFLOP/s) and exp2 rate
    (10^12 / s) of this GPU, from the library's measurement microkernels
    (measurement only)."""
    L = lib()
    sink = torch.empty(int(L.radar_peak_sink_floats()), dtype=torch.float32,
                       device=device)
    st = ctypes.c_void_p(torch.cuda.current_stream(sink.device).cuda_stream)
    out = {}
    for name, fn, n in (("mfma_tflops", L.radar_peak_mfma, iters),
                        ("exp_T_per_s", L.radar_peak_exp, iters * 4)):
        work = ctypes.c_double()
        _check(fn.__name__, fn(n, _ptr(sink), ctypes.byref(work), st))    # warm
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            _check(fn.__name__, fn(n, _ptr(sink), ctypes.byref(work), st))
        e1.record()
        torch.cuda.synchronize()
        sec = e0.elapsed_time(e1) / 3 * 1e-3
        out[name] = work.value / sec / 1e12
    return out


def peak_read_gbps(device="cuda", nbytes=4 << 30, reps=5) -> float:
    """Measured HBM read rate (GB/s) of one pass of non-temporal 16-byte
    loads over a fresh `nbytes` buffer, the loads the decode kernels stream
    with (measurement only)."""
    L = lib()
    sink = torch.empty(int(L.radar_peak_sink_floats()), dtype=torch.float32,
                       device=device)
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device=device)
    st = ctypes.c_void_p(torch.cuda.current_stream(sink.device).cuda_stream)
    _check("radar_peak_read", L.radar_peak_read(_ptr(buf), nbytes, _ptr(sink), st))
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        _check("radar_peak_read", L.radar_peak_read(_ptr(buf), nbytes, _ptr(sink), st))
    e1.record()
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) / reps * 1e-3
    del buf
    return nbytes / sec / 1e9


class RadarLayer:
    """Device state of one Radar layer: K/V cache, summaries, Omega and a
    decode workspace, driven through the C ABI (append, then decode, or
    both in one step).

    schedule="fixed" keeps cfg.seg_len and cfg.window. schedule="sqrt"
    follows Algorithm 1's restructuring: at every perfect-square context
    length the summaries are rebuilt with c = sqrt(t), and each decode
    attends the c restructured segments' top-k plus the buffer [c^2, t)."""

    def __init__(self, cfg: Config, omega, K=None, V=None, t: int = 0,
                 top_k: int = 16, device="cuda", schedule: str = "fixed"):
        if schedule not in ("fixed", "sqrt"):
            raise ValueError(schedule)
        self.cfg, self.k, self.schedule = cfg, top_k, schedule
        # summaries and workspace live on the GPU; K and V may be given in
        # pinned, device-mapped host memory
        if K is None:
            self.device = torch.device(device)
        elif K.is_cuda:
            self.device = K.device
        else:
            self.device = torch.device("cuda")
        shape = (cfg.batch, cfg.n_kv_heads, cfg.capacity, cfg.head_dim)
        self.K = K if K is not None else torch.zeros(shape, dtype=cfg.dtype, device=device)
        self.V = V if V is not None else torch.zeros(shape, dtype=cfg.dtype, device=device)
        self.omega = omega
        self.t = t
        if schedule == "sqrt":
            c0 = schedule_sqrt(max(t, 1))[0]
            rows = cfg.capacity // c0              # the smallest c comes first
            self.summaries = torch.zeros(cfg.batch, cfg.n_kv_heads, rows,
                                         cfg.n_features, dtype=torch.float32,
                                         device=self.device)
            self.cfg = self._cfg_at(max(t, 1))
        else:
            self.summaries = new_summaries(cfg, self.device)
        self.workspace = new_workspace(self.cfg, top_k, self.device)
        self.restructures = 0
        if t > 0:
            build_index(self.cfg, self.K, omega, t, self.summaries)

    def _cfg_at(self, t):
        c, w = schedule_sqrt(t)
        return dataclasses.replace(self.cfg, seg_len=c, window=w)

    def append(self, k_new, v_new):
        append(self.cfg, self.K, self.V, k_new, v_new, self.omega, self.t,
               self.summaries)
        self.t += 1
        if self.schedule == "sqrt":
            c_old = self.cfg.seg_len
            self.cfg = self._cfg_at(self.t)
            if self.cfg.seg_len != c_old:          # t is a perfect square
                build_index(self.cfg, self.K, self.omega, self.t,
                            self.summaries)
                self.restructures += 1

    def decode(self, q, out=None, selected=None, scores=None):
        self._fit_workspace()
        return decode(self.cfg, q, self.K, self.V, self.omega, self.summaries,
                      self.t, self.k, out=out, selected=selected, scores=scores,
                      workspace=self.workspace)

    def step(self, q, k_new, v_new, out=None, selected=None, scores=None):
        """append(k_new, v_new) then decode(q), as one radar_append_decode
        call unless the sqrt schedule restructures at this token."""
        if self.schedule == "sqrt" and self._cfg_at(self.t + 1).seg_len != self.cfg.seg_len:
            self.append(k_new, v_new)
            return self.decode(q, out=out, selected=selected, scores=scores)
        if self.schedule == "sqrt":
            self.cfg = self._cfg_at(self.t + 1)
        self._fit_workspace()
        self.t += 1
        return append_decode(self.cfg, q, self.K, self.V, k_new, v_new,
                             self.omega, self.summaries, self.t, self.k,
                             out=out, selected=selected, scores=scores,
                             workspace=self.workspace)

    def _fit_workspace(self):
        # the scratch size follows the window, which grows between
        # restructures under the sqrt schedule
        if workspace_bytes(self.cfg, self.k) > self.workspace.numel():
            self.workspace = new_workspace(self.cfg, self.k, self.device)
