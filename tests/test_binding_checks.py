"""The Python binding checks every device buffer before its pointer reaches
the library (which cannot see buffer sizes): a host tensor, a wrong dtype, a
non-contiguous view or an undersized buffer raises SiftError, and the
library is never called.  Runs on the CPU: the library entry points are
replaced by a stub that fails the test if reached."""

import numpy as np
import pytest
import torch

import paper_2606_09441_amd._lib as L
from paper_2606_09441_amd import Plan, SiftError

INFO = {"num_tokens": 288, "num_segments": 3, "num_tiles": 18, "num_q_heads": 2,
        "num_kv_heads": 1, "head_dim": 64, "tile": 16, "num_work_units": 4, "num_rows": 36,
        "list_capacity": 342, "la_bytes": 20, "ca_bytes": 4, "scratch_bytes": 0}


class _NoLib:
    def __getattr__(self, name):
        raise AssertionError(f"library entry {name} reached with a bad buffer")


@pytest.fixture
def plan(monkeypatch):
    monkeypatch.setattr(L, "lib", lambda: _NoLib())
    p = Plan.__new__(Plan)
    p._h = None
    p.device = None
    p.info = dict(INFO)
    return p


def _u8(n):
    return torch.zeros(n, dtype=torch.uint8)


def _i32(n):
    return torch.zeros(n, dtype=torch.int32)


def _status(fn, *a, **kw):
    with pytest.raises(SiftError) as e:
        fn(*a, **kw)
    return e.value.status


def test_require_rules():
    assert _status(L.require, "f", None, "x", "uint8", 1) == 1
    assert _status(L.require, "f", np.zeros(4, np.uint8), "x", "uint8", 1) == 4
    assert _status(L.require, "f", _i32(8), "x", "uint8", 1) == 4          # dtype
    assert _status(L.require, "f", _i32(8)[::2], "x", "int32", 1) == 2     # not contiguous
    assert _status(L.require, "f", _u8(3), "x", "uint8", 4) == 5           # too small
    assert _status(L.require, "f", _u8(4), "x", "uint8", 4) == 4           # host memory
    L.require("f", None, "x", "uint8", 0)                                  # optional, absent


def test_decode_checks_bitmaps_and_lists(plan):
    la, ca = _u8(20), _u8(4)
    assert _status(plan.decode, _u8(19), ca) == 5                 # bitmap built for other sizes
    assert _status(plan.decode, la, _u8(3)) in (4, 5)
    assert _status(plan.decode, la.to(torch.int32), ca) == 4
    assert _status(plan.decode, la, ca) == 4                       # host tensors
    assert _status(plan.decode, la, ca, row_ptr=_i32(36), col_idx=_i32(342)) in (4, 5)
    assert _status(plan.decode_internal, _u8(19), ca) == 5
    assert _status(plan.run, None, None, None, _u8(10), ca) == 5


def test_attention_and_paged_check_their_buffers(plan):
    assert _status(plan.attention, None, None, None, _i32(36), _i32(10)) == 5      # row_ptr short
    assert _status(plan.attention, None, None, None, _i32(37).to(torch.int64), _i32(10)) == 4
    la, ca = _u8(20), _u8(4)
    assert _status(plan.run_paged, None, None, None, _i32(17), la, ca) in (4, 5)
    assert _status(plan.run_paged, None, None, None, None, _u8(1), ca) == 5


def test_one_shot_checks_bitmaps(monkeypatch):
    q = torch.zeros(288, 2, 64)
    # a host q is refused before anything else
    assert _status(L.sparse_prefill, q, q, q, [0, 128, 256, 288], [0, 3], _u8(20), _u8(4),
                   tile=16) == 4


def test_bitmap_bytes_follow_section_4_3():
    # documents of 128 tokens at T = 16: P = 8, LA ceil(72/16) = 5 bytes, CA 1 byte, per head
    assert L.bitmap_bytes([0, 128, 256, 288], [0, 3], 2, 16) == (2 * 2 * 5, 2 * 2 * 1)
    assert L.bitmap_bytes([0, 40], [0, 1], 4, 16) == (0, 0)        # a query alone
