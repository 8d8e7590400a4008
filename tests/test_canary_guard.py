"""The guard regions of the GPU canary test, exercised on the CPU: a write
past either end of a guarded view, or into the unwritten tail of a cache,
must be seen."""
import os
import sys

import torch

sys.path.insert(0, os.path.dirname(__file__))
from test_gpu_canaries import Guarded  # noqa: E402


def test_guard_sees_writes_past_either_end():
    for dtype in (torch.float32, torch.bfloat16, torch.int32, torch.uint8, torch.int64):
        g = Guarded((3, 5), dtype, device="cpu")
        g.t.zero_()
        assert g.intact()
        g.buf[g.pe - 1] = 0                       # one element before the view
        assert not g.intact()
        g = Guarded((3, 5), dtype, device="cpu")
        g.buf[g.pe + g.n] = 1                     # one element after it
        assert not g.intact()


def test_guard_sees_a_write_into_an_unwritten_tail():
    g = Guarded((2, 10, 4), torch.float32, device="cpu")
    g.t[:, :6] = 1.0                              # rows 0..5 written
    tail = slice(6 * 4, 10 * 4)                   # rows 6..9 of the first head
    assert g.region_is_sentinel(tail)
    g.t[0, 7, 2] = 0.0
    assert not g.region_is_sentinel(tail)
