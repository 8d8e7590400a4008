"""The C ABI on the CPU: the library loads, exports every function that
include/radar.h declares, sizes workspaces, and rejects bad arguments with
the documented status codes before anything reaches the GPU (every call here
fails validation, so no kernel is launched)."""
import ctypes
import os
import re

import pytest

import paper_2503_10571_amd as radar
from paper_2503_10571_amd import _build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "radar.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(radar.LIB_PATH):
        _build.build_library()
    return radar.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(radar_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert {"radar_build_index", "radar_append", "radar_decode",
            "radar_decode_workspace_bytes", "radar_attend_selected",
            "radar_status_string", "radar_last_error",
            "radar_abi_version"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_version_and_strings(L):
    assert L.radar_abi_version() == radar.ABI_VERSION == 7
    for st in range(6):
        assert L.radar_status_string(st).decode()
    assert L.radar_last_error() is not None


def test_config_layout_matches_the_header(tmp_path):
    """The binding's ctypes mirror of radar_config has the C compiler's size
    and field offsets (a C program built from the header prints them)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "layout.c"
    src.write_text(
        "#include <stddef.h>\n#include <stdio.h>\n#include \"radar.h\"\n"
        "int main(void) {\n"
        "  printf(\"%zu\", sizeof(radar_config));\n"
        + "".join(f"  printf(\" %zu\", offsetof(radar_config, {f}));\n"
                  for f, _ in radar._Config._fields_)
        + "  return 0;\n}\n")
    exe = tmp_path / "layout"
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    r = subprocess.run([gcc, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                        "-I", os.path.join(rocm, "include"), str(src), "-o", str(exe)],
                       capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("header does not compile here: " + r.stderr[-300:])
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True,
                                          text=True, check=True).stdout.split()]
    want = [ctypes.sizeof(radar._Config)] + [getattr(radar._Config, f).offset
                                             for f, _ in radar._Config._fields_]
    assert got == want


def _cfg(**kw):
    base = dict(batch=8, n_q_heads=32, n_kv_heads=32, head_dim=128,
                n_features=256, seg_len=256, window=256, capacity=131584)
    base.update(kw)
    return radar.Config(**base)


def test_workspace_bytes(L):
    import torch
    cfg = _cfg()
    n16 = radar.workspace_bytes(cfg, 16)
    n32 = radar.workspace_bytes(cfg, 32)
    assert 0 < n16 < n32
    # phi(q) + scores + union + partials: a few MB at the 128K shape
    assert n16 < 64 << 20
    assert radar.workspace_bytes(cfg, 0) == 0
    assert radar.workspace_bytes(cfg, 257) == 0
    assert radar.workspace_bytes(_cfg(n_q_heads=24, n_kv_heads=8), 16) == 0  # G=3
    assert radar.workspace_bytes(_cfg(head_dim=96), 16) == 0
    assert radar.workspace_bytes(_cfg(n_features=100), 16) == 0
    assert radar.workspace_bytes(_cfg(n_features=2048), 16) > n16
    assert radar.workspace_bytes(_cfg(dtype=torch.float32), 16) > 0
    # a bf16 Omega with a bf16 cache; refused with an fp32 cache
    assert radar.workspace_bytes(_cfg(omega_dtype=torch.bfloat16), 16) == n16
    assert radar.workspace_bytes(_cfg(dtype=torch.float32,
                                      omega_dtype=torch.bfloat16), 16) == 0


def _P(v):
    return ctypes.c_void_p(v)


def test_validation_before_launch(L):
    cfg = _cfg().c_struct()
    good = _P(0x1000)
    odd = _P(0x1008)
    null = None
    by = ctypes.byref
    # null config / pointers
    assert L.radar_build_index(None, good, good, 10, good, None) == 1
    assert L.radar_build_index(by(cfg), null, good, 10, good, None) == 1
    # misaligned
    assert L.radar_build_index(by(cfg), odd, good, 10, good, None) == 1
    # t outside [1, capacity]
    assert L.radar_build_index(by(cfg), good, good, 0, good, None) == 2
    assert L.radar_build_index(by(cfg), good, good, 131585, good, None) == 2
    # append position outside [0, capacity)
    ap = [by(cfg), good, good, good, good, good]
    assert L.radar_append(*ap, 131584, null, good, None) == 2
    assert L.radar_append(*ap, -1, null, good, None) == 2
    assert L.radar_append(*ap, 5, odd, good, None) == 1      # misaligned pos
    ws = L.radar_decode_workspace_bytes(by(cfg), 16)
    args = [by(cfg), good, good, good, good, good]
    # k out of range
    assert L.radar_decode(*args, 1000, null, 0, good, None, None, good, ws, None) == 3
    assert L.radar_decode(*args, 1000, null, 300, good, None, None, good, ws, None) == 3
    # t out of range
    assert L.radar_decode(*args, 0, null, 16, good, None, None, good, ws, None) == 2
    # misaligned lens
    assert L.radar_decode(*args, 1000, odd, 16, good, None, None, good, ws, None) == 1
    # workspace missing / too small
    assert L.radar_decode(*args, 1000, null, 16, good, None, None, None, ws, None) == 5
    assert L.radar_decode(*args, 1000, null, 16, good, None, None, good, ws - 1,
                          None) == 5
    # too many candidate segments for the top-k stage
    big = _cfg(seg_len=16, window=16, capacity=1 << 20).c_struct()
    wsb = L.radar_decode_workspace_bytes(by(big), 16)
    assert L.radar_decode(by(big), good, good, good, good, good, 40000, null, 16,
                          good, None, None, good, wsb, None) == 3
    # bad shapes
    for bad in (_cfg(batch=0), _cfg(n_q_heads=30), _cfg(seg_len=0),
                _cfg(window=-1), _cfg(capacity=0), _cfg(n_sink=-1),
                _cfg(n_sink=131585), _cfg(gqa_mode=2)):
        assert L.radar_build_index(by(bad.c_struct()), good, good, 1, good,
                                   None) == 1
    # Omega element type: fp32 or bf16, bf16 only with a bf16 cache
    import torch
    for bad_omega in (2, -1):
        c = _cfg().c_struct()
        c.omega_dtype = bad_omega
        assert L.radar_build_index(by(c), good, good, 1, good, None) == 1
        assert L.radar_decode_workspace_bytes(by(c), 16) == 0
    c = _cfg(dtype=torch.float32, omega_dtype=torch.bfloat16).c_struct()
    assert L.radar_build_index(by(c), good, good, 1, good, None) == 1
    assert L.radar_append(by(c), good, good, good, good, good, 5, null, good,
                          None) == 1
    for bad in (_cfg(head_dim=256), _cfg(n_features=4096), _cfg(n_features=768),
                _cfg(n_q_heads=96, n_kv_heads=32), _cfg(capacity=1 << 31),
                _cfg(batch=2048, n_q_heads=32, n_kv_heads=32)):
        assert L.radar_build_index(by(bad.c_struct()), good, good, 1, good,
                                   None) == 3
    # decode_exact: same checks as decode
    ex = [by(cfg), good, good, good]
    assert L.radar_decode_exact(*ex, 1000, null, 0, good, None, None, good, ws,
                                None) == 3
    assert L.radar_decode_exact(*ex, 131585, null, 16, good, None, None, good,
                                ws, None) == 2
    assert L.radar_decode_exact(*ex, 1000, null, 16, null, None, None, good, ws,
                                None) == 1
    assert L.radar_decode_exact(*ex, 1000, null, 16, good, None, None, good,
                                ws - 1, None) == 5
    assert L.radar_decode_exact(by(big), good, good, good, 40000, null, 16, good,
                                None, None, good, wsb, None) == 3
    # attend_selected
    assert L.radar_attend_selected(by(cfg), good, good, good, null, 4, 100,
                                   null, good, good, ws, None) == 1
    assert L.radar_attend_selected(by(cfg), good, good, good, good, 0, 100,
                                   null, good, good, ws, None) == 3
    # append_decode: append's and decode's checks, t is the length after
    # the append
    ad = [by(cfg), good, good, good, good, good, good, good]
    assert L.radar_append_decode(None, good, good, good, good, good, good, good,
                                 1000, null, 16, good, None, None, good, ws,
                                 None) == 1
    assert L.radar_append_decode(by(cfg), null, good, good, good, good, good,
                                 good, 1000, null, 16, good, None, None, good,
                                 ws, None) == 1
    assert L.radar_append_decode(by(cfg), good, good, good, null, good, good,
                                 good, 1000, null, 16, good, None, None, good,
                                 ws, None) == 1
    assert L.radar_append_decode(*ad, 0, null, 16, good, None, None, good, ws,
                                 None) == 2
    assert L.radar_append_decode(*ad, 131585, null, 16, good, None, None, good,
                                 ws, None) == 2
    assert L.radar_append_decode(*ad, 1000, odd, 16, good, None, None, good, ws,
                                 None) == 1
    assert L.radar_append_decode(*ad, 1000, null, 0, good, None, None, good, ws,
                                 None) == 3
    assert L.radar_append_decode(*ad, 1000, null, 16, good, None, None, good,
                                 ws - 1, None) == 5
    assert L.radar_append_decode(*ad, 1000, null, 16, null, None, None, good,
                                 ws, None) == 1
    # append_decode_noalloc: the same checks (a bad config or k fails
    # before the scratch is looked up), and a shape whose scratch exceeds the
    # library's array is refused
    assert L.radar_append_decode_noalloc(None, good, good, good, good, good,
                                         good, good, 1000, null, 16, good,
                                         None, None, None) == 1
    assert L.radar_append_decode_noalloc(*ad, 1000, null, 0, good, None, None,
                                         None) == 3
    assert L.radar_append_decode_noalloc(*ad, 1000, null, 300, good, None,
                                         None, None) == 3
    huge = _cfg(batch=64, capacity=1 << 20).c_struct()
    assert L.radar_decode_workspace_bytes(by(huge), 16) > radar.NOALLOC_SCRATCH_BYTES
    assert L.radar_append_decode_noalloc(by(huge), good, good, good, good, good,
                                         good, good, 1000, null, 16, good,
                                         None, None, None) == 5
    # segment_mass: pointers, t, candidates
    assert L.radar_segment_mass(by(cfg), good, good, 1000, null, null, None) == 1
    assert L.radar_segment_mass(by(cfg), good, odd, 1000, null, good, None) == 1
    assert L.radar_segment_mass(by(cfg), good, good, 0, null, good, None) == 2
    assert L.radar_segment_mass(by(cfg), good, good, 131585, null, good, None) == 2
    assert L.radar_segment_mass(by(big), good, good, 40000, null, good, None) == 3
    # measurement microkernels
    work = ctypes.c_double()
    assert L.radar_peak_mfma(0, good, by(work), None) == 1
    assert L.radar_peak_exp(16, null, by(work), None) == 1
    assert L.radar_peak_exp(16, odd, by(work), None) == 1
    assert L.radar_peak_read(good, 0, good, None) == 1
    assert L.radar_peak_read(good, 24, good, None) == 1
    assert L.radar_peak_read(odd, 32, good, None) == 1
    # sinks widen the scratch for the attention partials
    assert radar.workspace_bytes(_cfg(n_sink=4096), 16) > \
        radar.workspace_bytes(_cfg(), 16)


def test_product_path_has_no_fallback(monkeypatch, tmp_path):
    """Without the built library the binding raises instead of computing."""
    monkeypatch.setattr(radar, "_lib", None)
    monkeypatch.setattr(radar, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        radar.lib()


def test_noalloc_scratch_size_matches_the_header():
    """The binding's copy of RADAR_NOALLOC_SCRATCH_BYTES is the header's, and
    it holds the decode workspace of every benchmark workload."""
    import workloads
    text = open(HEADER).read()
    m = re.search(r"#define RADAR_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)",
                  text)
    assert m, "macro not found"
    assert int(m.group(1)) << int(m.group(2)) == radar.NOALLOC_SCRATCH_BYTES


def test_noalloc_scratch_holds_every_workload(L):
    import workloads
    import torch
    for wl in workloads.WORKLOADS.values():
        cfg = radar.Config(wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                           wl.n_features, wl.seg_len, wl.window, wl.capacity + 64,
                           wl.torch_dtype())
        assert 0 < radar.workspace_bytes(cfg, wl.top_k) <= radar.NOALLOC_SCRATCH_BYTES, wl.name
