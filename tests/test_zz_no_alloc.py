"""GPU: sift_sparse_prefill_static, the one-shot form on the library's
static device scratch (for callers that cannot allocate), against
sift_sparse_prefill_ex on a caller workspace: outputs bit-identical on two
calls in a row, the second with a smaller input (the scratch keeps the first
call's contents), plus the oracle's tolerance and the capacity refusal."""

import ctypes

import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import BF16_TOL, F32_TOL, device, max_abs, oracle_layout, say
from oracle import sift_oracle as O
import paper_2606_09441_amd._lib as L

pytestmark = pytest.mark.gpu


def _dev(wl):
    dev = device()
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    t = lambda x: torch.from_numpy(x).to(dev).to(dt).contiguous()
    la = torch.from_numpy(wl.la if wl.la.size else np.zeros(1, np.uint8)).to(dev)
    ca = torch.from_numpy(wl.ca if wl.ca.size else np.zeros(1, np.uint8)).to(dev)
    return t(wl.q), t(wl.k), t(wl.v), la, ca


def _static(wl, q, k, v, la, ca, out):
    """Through the C ABI directly."""
    lay, keep = L.layout_struct(wl.seg_offsets, wl.prompt_seg_ptr)
    qd, kd, vd, od = (L.tensor_desc(x) for x in (q, k, v, out))
    return L.lib().sift_sparse_prefill_static(
        ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(vd), ctypes.byref(lay),
        ctypes.c_void_p(la.data_ptr()), ctypes.c_void_p(ca.data_ptr()), wl.tile,
        ctypes.c_float(0.0), ctypes.byref(od),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


@pytest.mark.parametrize("dtype,tile", [("bf16", 64), ("bf16", 16), ("f32", 32)])
def test_static_matches_workspace_form_twice(dtype, tile):
    from paper_2606_09441_amd import sparse_prefill_ex
    d = 128 if dtype == "bf16" else 64
    big = W.custom([[300, 64, 129, 75], [5], [200, 131, 70]], tile=tile, hq=8, hkv=2, d=d,
                   dtype=dtype, seed=21, p_la=0.4, p_ca=0.3)
    small = W.custom([[70, 33]], tile=tile, hq=8, hkv=2, d=d, dtype=dtype, seed=22)
    tol = BF16_TOL if dtype == "bf16" else F32_TOL
    for tag, wl in (("first, larger", big), ("second, smaller", small)):
        say(f"[static] {dtype} T={tile} {tag}: tokens={wl.tokens}")
        q, k, v, la, ca = _dev(wl)
        out = torch.empty_like(q)
        st = _static(wl, q, k, v, la, ca, out)
        assert st == 0, L.STATUS.get(st, st)
        ref_ex = sparse_prefill_ex(q, k, v, wl.seg_offsets, wl.prompt_seg_ptr, la, ca, tile=tile)
        torch.cuda.synchronize()
        assert torch.equal(out, ref_ex), f"{tag}: static scratch output differs from workspace output"
        err = max_abs(out.float().cpu().numpy(),
                      O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca))
        say(f"[static] {dtype} T={tile} {tag}: equal to the workspace form, max-abs {err:.3e}")
        assert err <= tol


def test_static_refuses_layouts_beyond_its_scratch():
    need = L.workspace_bytes([0, 2048 * 32 + 512], [0, 1], 48, 8, 128, 16)
    assert need > L.static_scratch_bytes()
    wl_so, wl_ps = np.array([0, 2048 * 32 + 512], np.int32), np.array([0, 1], np.int32)
    dev = device()
    n = 2048 * 32 + 512
    q = torch.empty((n, 48, 128), dtype=torch.bfloat16, device=dev)
    k = torch.empty((n, 8, 128), dtype=torch.bfloat16, device=dev)
    lay, keep = L.layout_struct(wl_so, wl_ps)
    qd, kd = L.tensor_desc(q), L.tensor_desc(k)
    st = L.lib().sift_sparse_prefill_static(ctypes.byref(qd), ctypes.byref(kd), ctypes.byref(kd),
                                             ctypes.byref(lay), None, None, 16, ctypes.c_float(0.0),
                                             ctypes.byref(qd), None)
    assert st == 5
    say("[static] a 64K query-only layout at T=16 is refused: SIFT_E_CAPACITY")
