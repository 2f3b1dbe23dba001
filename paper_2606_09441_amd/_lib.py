"""ctypes binding of libsift (include/sift.h).  Marshalling only: every step
of the hot path runs in the library's HIP kernels; torch provides device
memory and the current stream."""

from __future__ import annotations

import ctypes
import math
import os
import re

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsift.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "sift.h")

SIFT_F32 = 0
SIFT_BF16 = 1

STATUS = {
    0: "SIFT_OK", 1: "SIFT_E_NULL", 2: "SIFT_E_SHAPE", 3: "SIFT_E_LAYOUT",
    4: "SIFT_E_UNSUPPORTED", 5: "SIFT_E_CAPACITY", 6: "SIFT_E_HIP", 7: "SIFT_E_PLAN",
}


class SiftError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: {STATUS.get(status, status)} ({msg})")
        self.status = status


class SiftTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("tokens", ctypes.c_int32),
                ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32)]


class SiftLayout(ctypes.Structure):
    _fields_ = [("num_prompts", ctypes.c_int32),
                ("prompt_seg_ptr", ctypes.POINTER(ctypes.c_int32)),
                ("seg_offsets", ctypes.POINTER(ctypes.c_int32))]


class SiftPlanInfo(ctypes.Structure):
    _fields_ = [("num_tokens", ctypes.c_int32), ("num_segments", ctypes.c_int32),
                ("num_tiles", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("tile", ctypes.c_int32), ("num_work_units", ctypes.c_int32),
                ("num_rows", ctypes.c_int64), ("list_capacity", ctypes.c_int64),
                ("la_bytes", ctypes.c_int64), ("ca_bytes", ctypes.c_int64),
                ("scratch_bytes", ctypes.c_int64)]


_P = ctypes.c_void_p
_SIGS = {
    "sift_status_string": (ctypes.c_char_p, [ctypes.c_int32]),
    "sift_plan_create": (ctypes.c_int, [ctypes.POINTER(SiftLayout), ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(_P)]),
    "sift_plan_destroy": (ctypes.c_int, [_P]),
    "sift_plan_get_info": (ctypes.c_int, [_P, ctypes.POINTER(SiftPlanInfo)]),
    "sift_plan_exact_passes": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int64)]),
    "sift_plan_decode_tiles": (ctypes.c_int, [_P, _P, _P, _P, _P, ctypes.c_int64, _P]),
    "sift_decode_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(SiftLayout), ctypes.c_int32,
                                                   ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]),
    "sift_decode_tiles": (ctypes.c_int, [ctypes.POINTER(SiftLayout), _P, _P, ctypes.c_int32,
                                         ctypes.c_int32, _P, _P, ctypes.c_int64, _P,
                                         ctypes.c_size_t, _P]),
    "sift_sparse_attention": (ctypes.c_int, [_P, ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftTensor),
                                             ctypes.POINTER(SiftTensor), _P, _P, ctypes.c_int64,
                                             ctypes.c_float, ctypes.POINTER(SiftTensor), _P]),
    "sift_plan_decode": (ctypes.c_int, [_P, _P, _P, _P]),
    "sift_plan_attention": (ctypes.c_int, [_P, ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftTensor),
                                           ctypes.POINTER(SiftTensor), ctypes.c_float,
                                           ctypes.POINTER(SiftTensor), _P]),
    "sift_plan_run": (ctypes.c_int, [_P, ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftTensor),
                                     ctypes.POINTER(SiftTensor), _P, _P, ctypes.c_float,
                                     ctypes.POINTER(SiftTensor), _P]),
    "sift_plan_run_paged": (ctypes.c_int, [_P, ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftTensor),
                                           ctypes.POINTER(SiftTensor), _P, _P, _P, ctypes.c_float,
                                           ctypes.POINTER(SiftTensor), _P]),
    "sift_sparse_prefill": (ctypes.c_int, [ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftTensor),
                                           ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftLayout),
                                           _P, _P, ctypes.c_int32, ctypes.POINTER(SiftTensor), _P]),
    "sift_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(SiftLayout), ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_int32, ctypes.c_int32,
                                            ctypes.POINTER(ctypes.c_size_t)]),
    "sift_sparse_prefill_ex": (ctypes.c_int, [ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftTensor),
                                              ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftLayout),
                                              _P, _P, ctypes.c_int32, ctypes.c_float, _P,
                                              ctypes.c_size_t, ctypes.POINTER(SiftTensor), _P]),
    "sift_sparse_prefill_static": (ctypes.c_int, [ctypes.POINTER(SiftTensor),
                                                  ctypes.POINTER(SiftTensor),
                                                  ctypes.POINTER(SiftTensor),
                                                  ctypes.POINTER(SiftLayout), _P, _P,
                                                  ctypes.c_int32, ctypes.c_float,
                                                  ctypes.POINTER(SiftTensor), _P]),
    "sift_static_scratch_bytes": (ctypes.c_size_t, []),
    "sift_rope": (ctypes.c_int, [ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftTensor), _P, _P, _P]),
    "sift_extract_sizes": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t),
                                          ctypes.POINTER(ctypes.c_size_t)]),
    "sift_extract_bits": (ctypes.c_int, [ctypes.POINTER(SiftTensor), ctypes.POINTER(SiftTensor),
                                         ctypes.c_int32, _P, ctypes.c_int32, ctypes.c_double,
                                         ctypes.c_double, ctypes.c_double, ctypes.c_float, _P, _P, _P,
                                         ctypes.c_size_t, _P]),
}

_lib = None


def header_functions() -> list[str]:
    """Names of the functions include/sift.h declares."""
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sift_[a-z_]+)\s*\(", text)))


def lib() -> ctypes.CDLL:
    """Load libsift.so once.  Raises if it has not been built: there is no
    fallback path."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2606_09441_amd.build` (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def check(fn: str, status: int) -> None:
    if status != 0:
        msg = lib().sift_status_string(status).decode()
        raise SiftError(fn, status, msg)


# ----------------------------------------------------------------------------
# torch marshalling
# ----------------------------------------------------------------------------


def _torch():
    import torch
    return torch


def tensor_desc(t) -> SiftTensor:
    torch = _torch()
    if not getattr(t, "is_cuda", False):
        raise SiftError("tensor_desc", 4, "tensors must be in GPU memory")
    if t.dim() != 3:
        raise ValueError("expected a [tokens, heads, head_dim] tensor")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    if t.dtype == torch.bfloat16:
        dt = SIFT_BF16
    elif t.dtype == torch.float32:
        dt = SIFT_F32
    else:
        raise ValueError(f"unsupported dtype {t.dtype}")
    return SiftTensor(t.data_ptr(), dt, t.shape[0], t.shape[1], t.shape[2])


def require(fn: str, t, name: str, dtype: str, min_numel: int, device=None) -> None:
    """Check a device buffer before its pointer goes to the library, which
    cannot see buffer sizes: a GPU tensor (on `device` when given), of
    `dtype` ("uint8", "int32", "float32"), contiguous, with at least
    min_numel elements.  Raises SiftError otherwise."""
    torch = _torch()
    want = {"uint8": torch.uint8, "int32": torch.int32, "float32": torch.float32}[dtype]
    if t is None:
        if min_numel > 0:
            raise SiftError(fn, 1, f"{name} is required")
        return
    if not isinstance(t, torch.Tensor):
        raise SiftError(fn, 4, f"{name} must be a torch tensor")
    if t.dtype != want:
        raise SiftError(fn, 4, f"{name} must be {dtype}, not {t.dtype}")
    if not t.is_contiguous():
        raise SiftError(fn, 2, f"{name} must be contiguous")
    if t.numel() < min_numel:
        raise SiftError(fn, 5, f"{name} holds {t.numel()} elements, needs {min_numel}")
    if not t.is_cuda:
        raise SiftError(fn, 4, f"{name} must be a GPU tensor")
    if device is not None and t.device != device:
        raise SiftError(fn, 7, f"{name} is on {t.device}, the plan on {device}")


def bitmap_bytes(seg_offsets, prompt_seg_ptr, num_q_heads: int, tile: int) -> tuple[int, int]:
    """(LA bytes, CA bytes) the bit-vector buffers of a layout hold, from the
    library (sift_extract_sizes over the layout's documents in order)."""
    so = np.asarray(seg_offsets, dtype=np.int64)
    ps = np.asarray(prompt_seg_ptr, dtype=np.int64)
    lens = [int(so[s + 1] - so[s]) for b in range(len(ps) - 1)
            for s in range(int(ps[b]), int(ps[b + 1]) - 1)]
    if not lens:
        return 0, 0
    if min(lens) < 1:
        raise SiftError("bitmap_bytes", 3, "documents must hold at least one token")
    offs = np.ascontiguousarray(np.concatenate([[0], np.cumsum(lens)]).astype(np.int32))
    la, ca = ctypes.c_size_t(), ctypes.c_size_t()
    check("sift_extract_sizes", lib().sift_extract_sizes(len(lens), offs.ctypes.data_as(_P),
                                                         num_q_heads, tile, ctypes.byref(la),
                                                         ctypes.byref(ca), None))
    return la.value, ca.value


def layout_struct(seg_offsets, prompt_seg_ptr):
    so = np.ascontiguousarray(np.asarray(seg_offsets, dtype=np.int32))
    ps = np.ascontiguousarray(np.asarray(prompt_seg_ptr, dtype=np.int32))
    lay = SiftLayout(len(ps) - 1, ps.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                     so.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    return lay, (so, ps)  # keep the arrays alive with the struct


def _stream_ptr(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


class Plan:
    """A validated prompt layout with its device tables (sift_plan_*)."""

    def __init__(self, seg_offsets, prompt_seg_ptr, num_q_heads, num_kv_heads, head_dim, tile=64):
        self._h = None
        lay, keep = layout_struct(seg_offsets, prompt_seg_ptr)
        h = ctypes.c_void_p()
        check("sift_plan_create", lib().sift_plan_create(ctypes.byref(lay), num_q_heads, num_kv_heads,
                                                         head_dim, tile, ctypes.byref(h)))
        self._h = h
        torch = _torch()
        self.device = torch.device("cuda", torch.cuda.current_device())
        inf = SiftPlanInfo()
        check("sift_plan_get_info", lib().sift_plan_get_info(self._h, ctypes.byref(inf)))
        self.info = {name: getattr(inf, name) for name, _ in SiftPlanInfo._fields_}

    def close(self):
        if self._h is not None:
            check("sift_plan_destroy", lib().sift_plan_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def _bits(self, fn, la, ca):
        require(fn, la, "local_bitmap", "uint8", self.info["la_bytes"], self.device)
        require(fn, ca, "cross_bitmap", "uint8", self.info["ca_bytes"], self.device)

    def decode(self, la, ca, row_ptr=None, col_idx=None, stream=None):
        """Decoded lists (Section 5.1) as device int32 tensors (row_ptr, col_idx)."""
        torch = _torch()
        self._bits("sift_plan_decode_tiles", la, ca)
        dev = la.device
        if row_ptr is None:
            row_ptr = torch.empty(self.info["num_rows"] + 1, dtype=torch.int32, device=dev)
        if col_idx is None:
            col_idx = torch.empty(max(1, self.info["list_capacity"]), dtype=torch.int32, device=dev)
        require("sift_plan_decode_tiles", row_ptr, "row_ptr", "int32", self.info["num_rows"] + 1,
                self.device)
        require("sift_plan_decode_tiles", col_idx, "col_idx", "int32", self.info["list_capacity"],
                self.device)
        check("sift_plan_decode_tiles", lib().sift_plan_decode_tiles(
            self._h, _ptr(la), _ptr(ca), _ptr(row_ptr), _ptr(col_idx), col_idx.numel(),
            _stream_ptr(stream)))
        return row_ptr, col_idx

    def attention(self, q, k, v, row_ptr, col_idx, scale=None, out=None, out_dtype=None, stream=None):
        """Sparse attention over given lists (Section 5.2)."""
        torch = _torch()
        require("sift_sparse_attention", row_ptr, "row_ptr", "int32", self.info["num_rows"] + 1,
                self.device)
        require("sift_sparse_attention", col_idx, "col_idx", "int32", 0, self.device)
        if out is None:
            out = torch.empty(q.shape, dtype=out_dtype or q.dtype, device=q.device)
        qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
        check("sift_sparse_attention", lib().sift_sparse_attention(
            self._h, ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), _ptr(row_ptr),
            _ptr(col_idx), col_idx.numel(), ctypes.c_float(0.0 if scale is None else scale),
            ctypes.byref(od), _stream_ptr(stream)))
        return out

    def exact_passes(self) -> int:
        """Attention launches on this plan that needed the exact second pass
        (sift_plan_exact_passes; waits for the plan's last stream)."""
        n = ctypes.c_int64()
        check("sift_plan_exact_passes", lib().sift_plan_exact_passes(self._h, ctypes.byref(n)))
        return n.value

    def decode_internal(self, la, ca, stream=None):
        """Decode into the plan's own scratch (sift_plan_decode)."""
        self._bits("sift_plan_decode", la, ca)
        check("sift_plan_decode", lib().sift_plan_decode(self._h, _ptr(la), _ptr(ca),
                                                         _stream_ptr(stream)))

    def attention_internal(self, q, k, v, scale=None, out=None, out_dtype=None, stream=None):
        """Attention over the plan's last decode (sift_plan_attention)."""
        torch = _torch()
        if out is None:
            out = torch.empty(q.shape, dtype=out_dtype or q.dtype, device=q.device)
        qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
        check("sift_plan_attention", lib().sift_plan_attention(
            self._h, ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd),
            ctypes.c_float(0.0 if scale is None else scale), ctypes.byref(od), _stream_ptr(stream)))
        return out

    def run(self, q, k, v, la, ca, scale=None, out=None, out_dtype=None, stream=None):
        """Decode + attention for one layer (sift_plan_run)."""
        torch = _torch()
        self._bits("sift_plan_run", la, ca)
        if out is None:
            out = torch.empty(q.shape, dtype=out_dtype or q.dtype, device=q.device)
        qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
        check("sift_plan_run", lib().sift_plan_run(
            self._h, ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), _ptr(la), _ptr(ca),
            ctypes.c_float(0.0 if scale is None else scale), ctypes.byref(od), _stream_ptr(stream)))
        return out

    def run_paged(self, q, k_pages, v_pages, page_table, la, ca, scale=None, out=None,
                  out_dtype=None, stream=None):
        """Decode + attention with K/V in a page pool (sift_plan_run_paged):
        k_pages/v_pages [num_pages * T, Hkv, D], page_table int32 [num_tiles]."""
        torch = _torch()
        self._bits("sift_plan_run_paged", la, ca)
        require("sift_plan_run_paged", page_table, "page_table", "int32", self.info["num_tiles"],
                self.device)
        if out is None:
            out = torch.empty(q.shape, dtype=out_dtype or q.dtype, device=q.device)
        qd, kd, vd, od = tensor_desc(q), tensor_desc(k_pages), tensor_desc(v_pages), tensor_desc(out)
        check("sift_plan_run_paged", lib().sift_plan_run_paged(
            self._h, ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), _ptr(page_table),
            _ptr(la), _ptr(ca), ctypes.c_float(0.0 if scale is None else scale), ctypes.byref(od),
            _stream_ptr(stream)))
        return out


def sparse_prefill(q, k, v, seg_offsets, prompt_seg_ptr, la, ca, tile=64, out=None, stream=None):
    """One-shot sift_sparse_prefill: stream-ordered scratch, decode and attention
    enqueued on the stream; returns without waiting."""
    torch = _torch()
    _check_bits("sift_sparse_prefill", q, la, ca, seg_offsets, prompt_seg_ptr, tile)
    if out is None:
        out = torch.empty_like(q)
    lay, keep = layout_struct(seg_offsets, prompt_seg_ptr)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
    check("sift_sparse_prefill", lib().sift_sparse_prefill(
        ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), ctypes.byref(lay), _ptr(la), _ptr(ca),
        tile, ctypes.byref(od), _stream_ptr(stream)))
    return out


def _check_bits(fn, q, la, ca, seg_offsets, prompt_seg_ptr, tile):
    """The bit-vector buffers of a one-shot call, against the layout's sizes."""
    if not getattr(q, "is_cuda", False):
        raise SiftError(fn, 4, "q must be a GPU tensor")
    la_n, ca_n = bitmap_bytes(seg_offsets, prompt_seg_ptr, q.shape[1], tile)
    require(fn, la, "local_bitmap", "uint8", la_n, q.device)
    require(fn, ca, "cross_bitmap", "uint8", ca_n, q.device)


def workspace_bytes(seg_offsets, prompt_seg_ptr, num_q_heads, num_kv_heads, head_dim, tile=64):
    """Device workspace bytes of sparse_prefill_ex (sift_workspace_bytes)."""
    lay, keep = layout_struct(seg_offsets, prompt_seg_ptr)
    n = ctypes.c_size_t()
    check("sift_workspace_bytes", lib().sift_workspace_bytes(
        ctypes.byref(lay), num_q_heads, num_kv_heads, head_dim, tile, ctypes.byref(n)))
    return n.value


def sparse_prefill_ex(q, k, v, seg_offsets, prompt_seg_ptr, la, ca, tile=64, scale=None,
                      workspace=None, out=None, stream=None):
    """One-shot form with the caller's scale and workspace (sift_sparse_prefill_ex):
    no device allocation in the library; returns once the work is enqueued.
    workspace: a uint8 device tensor of at least workspace_bytes(...) bytes
    (allocated here when None)."""
    torch = _torch()
    _check_bits("sift_sparse_prefill_ex", q, la, ca, seg_offsets, prompt_seg_ptr, tile)
    if out is None:
        out = torch.empty_like(q)
    n = workspace_bytes(seg_offsets, prompt_seg_ptr, q.shape[1], k.shape[1], q.shape[2], tile)
    if workspace is None:
        workspace = torch.empty(max(n, 1), dtype=torch.uint8, device=q.device)
    require("sift_sparse_prefill_ex", workspace, "workspace", "uint8", n, q.device)
    lay, keep = layout_struct(seg_offsets, prompt_seg_ptr)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
    check("sift_sparse_prefill_ex", lib().sift_sparse_prefill_ex(
        ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), ctypes.byref(lay), _ptr(la), _ptr(ca),
        tile, ctypes.c_float(0.0 if scale is None else scale), _ptr(workspace),
        workspace.numel() * workspace.element_size(), ctypes.byref(od), _stream_ptr(stream)))
    return out


def sparse_prefill_static(q, k, v, seg_offsets, prompt_seg_ptr, la, ca, tile=64, scale=None,
                          out=None, stream=None):
    """The one-shot form on the library's static device scratch
    (sift_sparse_prefill_static): nothing is allocated on the device; calls
    on one GPU must not overlap."""
    torch = _torch()
    _check_bits("sift_sparse_prefill_static", q, la, ca, seg_offsets, prompt_seg_ptr, tile)
    if out is None:
        out = torch.empty_like(q)
    lay, keep = layout_struct(seg_offsets, prompt_seg_ptr)
    qd, kd, vd, od = tensor_desc(q), tensor_desc(k), tensor_desc(v), tensor_desc(out)
    check("sift_sparse_prefill_static", lib().sift_sparse_prefill_static(
        ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), ctypes.byref(lay), _ptr(la), _ptr(ca),
        tile, ctypes.c_float(0.0 if scale is None else scale), ctypes.byref(od),
        _stream_ptr(stream)))
    return out


def static_scratch_bytes() -> int:
    """Bytes of the static scratch of sparse_prefill_static (per GPU)."""
    return int(lib().sift_static_scratch_bytes())


def decode_workspace_bytes(seg_offsets, prompt_seg_ptr, num_q_heads, tile=64):
    """Device workspace bytes of decode_tiles (sift_decode_workspace_bytes)."""
    lay, keep = layout_struct(seg_offsets, prompt_seg_ptr)
    n = ctypes.c_size_t()
    check("sift_decode_workspace_bytes", lib().sift_decode_workspace_bytes(
        ctypes.byref(lay), num_q_heads, tile, ctypes.byref(n)))
    return n.value


def list_capacity(seg_offsets, prompt_seg_ptr, num_q_heads, tile=64):
    """Hq x (causal tiles of all prompts): the col_idx size that bounds any
    decode of this layout."""
    so = np.asarray(seg_offsets, dtype=np.int64)
    ps = np.asarray(prompt_seg_ptr, dtype=np.int64)
    total = 0
    for b in range(len(ps) - 1):
        before = 0
        for s in range(int(ps[b]), int(ps[b + 1])):
            P = -(-int(so[s + 1] - so[s]) // tile)
            total += P * before + P * (P + 1) // 2
            before += P
    return num_q_heads * total


def decode_tiles(seg_offsets, prompt_seg_ptr, la, ca, num_q_heads, tile=64, row_ptr=None,
                 col_idx=None, workspace=None, stream=None):
    """Decoded lists without a plan (sift_decode_tiles): (row_ptr, col_idx)
    device int32 tensors; workspace is allocated here when None."""
    torch = _torch()
    fn = "sift_decode_tiles"
    dev = la.device if la is not None else ca.device
    la_n, ca_n = bitmap_bytes(seg_offsets, prompt_seg_ptr, num_q_heads, tile)
    require(fn, la, "local_bitmap", "uint8", la_n)
    require(fn, ca, "cross_bitmap", "uint8", ca_n)
    M = sum(-(-int(seg_offsets[s + 1] - seg_offsets[s]) // tile)
            for s in range(len(seg_offsets) - 1))
    cap = list_capacity(seg_offsets, prompt_seg_ptr, num_q_heads, tile)
    if row_ptr is None:
        row_ptr = torch.empty(num_q_heads * M + 1, dtype=torch.int32, device=dev)
    if col_idx is None:
        col_idx = torch.empty(max(1, cap), dtype=torch.int32, device=dev)
    n = decode_workspace_bytes(seg_offsets, prompt_seg_ptr, num_q_heads, tile)
    if workspace is None:
        workspace = torch.empty(max(n, 1), dtype=torch.uint8, device=dev)
    require(fn, row_ptr, "row_ptr", "int32", num_q_heads * M + 1, dev)
    require(fn, col_idx, "col_idx", "int32", cap, dev)
    require(fn, workspace, "workspace", "uint8", n, dev)
    lay, keep = layout_struct(seg_offsets, prompt_seg_ptr)
    check(fn, lib().sift_decode_tiles(ctypes.byref(lay), _ptr(la), _ptr(ca), tile, num_q_heads,
                                      _ptr(row_ptr), _ptr(col_idx), col_idx.numel(),
                                      _ptr(workspace), workspace.numel(), _stream_ptr(stream)))
    return row_ptr, col_idx


def extract_sizes(doc_offsets, num_q_heads, tile):
    """(LA bytes, CA bytes, workspace bytes) of sift_extract_bits."""
    import numpy as np
    offs = np.ascontiguousarray(np.asarray(doc_offsets, dtype=np.int32))
    la, ca, ws = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    check("sift_extract_sizes", lib().sift_extract_sizes(
        len(offs) - 1, offs.ctypes.data_as(_P), num_q_heads, tile, ctypes.byref(la), ctypes.byref(ca),
        ctypes.byref(ws)))
    return la.value, ca.value, ws.value


def extract_bits(q, k, doc_offsets, tile=64, alpha=0.001, beta=0.01, gamma=0.1, scale=None,
                 workspace=None, stream=None):
    """Offline metadata of documents prefilled alone (sift_extract_bits).

    q [tokens, Hq, D] and k [tokens, Hkv, D] are bf16 on the GPU; doc_offsets
    (host, [N+1]) delimit the documents.  Returns (la, ca) uint8 device
    tensors in the layout the online path reads."""
    import numpy as np
    torch = _torch()
    offs = np.ascontiguousarray(np.asarray(doc_offsets, dtype=np.int32))
    la_n, ca_n, ws_n = extract_sizes(offs, q.shape[1], tile)
    la = torch.empty(max(la_n, 1), dtype=torch.uint8, device=q.device)
    ca = torch.empty(max(ca_n, 1), dtype=torch.uint8, device=q.device)
    if workspace is None or workspace.numel() < ws_n:
        workspace = torch.empty(max(ws_n, 1), dtype=torch.uint8, device=q.device)
    qd, kd = tensor_desc(q), tensor_desc(k)
    require("sift_extract_bits", workspace, "workspace", "uint8", ws_n, q.device)
    check("sift_extract_bits", lib().sift_extract_bits(
        ctypes.byref(qd), ctypes.byref(kd), len(offs) - 1, offs.ctypes.data_as(_P), tile,
        float(alpha), float(beta), float(gamma), ctypes.c_float(0.0 if scale is None else scale),
        _ptr(la), _ptr(ca), _ptr(workspace), workspace.numel(), _stream_ptr(stream)))
    return la[:la_n], ca[:ca_n]


def rope_(q, k, positions, inv_freq, stream=None):
    """In-place rotary embedding of bf16 q and k (sift_rope)."""
    qd, kd = tensor_desc(q), tensor_desc(k)
    require("sift_rope", positions, "positions", "int32", q.shape[0], q.device)
    require("sift_rope", inv_freq, "inv_freq", "float32", q.shape[2] // 2, q.device)
    check("sift_rope", lib().sift_rope(ctypes.byref(qd), ctypes.byref(kd), _ptr(positions),
                                       _ptr(inv_freq), _stream_ptr(stream)))
    return q, k


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)
