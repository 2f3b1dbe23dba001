"""GPU: the one-shot form with the caller's softmax scale and workspace
(sift_sparse_prefill_ex, sift_workspace_bytes).

It computes what sift_sparse_prefill computes (Sections 4 and 5): the same
outputs bit for bit at the default scale, the oracle's at another scale,
and one workspace serves consecutive calls of different layouts on one
stream."""

import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import BF16_TOL, F32_TOL, device, max_abs, oracle_layout, say
from oracle import sift_oracle as O

pytestmark = pytest.mark.gpu


def _dev(wl):
    dev = device()
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    t = lambda x: torch.from_numpy(x).to(dev).to(dt).contiguous()
    la = torch.from_numpy(wl.la if wl.la.size else np.zeros(1, np.uint8)).to(dev)
    ca = torch.from_numpy(wl.ca if wl.ca.size else np.zeros(1, np.uint8)).to(dev)
    return t(wl.q), t(wl.k), t(wl.v), la, ca


def test_prefill_ex_matches_prefill_bit_for_bit():
    from paper_2606_09441_amd import sparse_prefill, sparse_prefill_ex
    wl = W.custom([[300, 64, 129, 75], [5], [200, 131, 70]], tile=64, hq=8, hkv=2, d=128,
                  dtype="bf16", seed=31, p_la=0.4, p_ca=0.3)
    q, k, v, la, ca = _dev(wl)
    a = sparse_prefill(q, k, v, wl.seg_offsets, wl.prompt_seg_ptr, la, ca, tile=64)
    b = sparse_prefill_ex(q, k, v, wl.seg_offsets, wl.prompt_seg_ptr, la, ca, tile=64)
    torch.cuda.synchronize()
    say(f"[ex] bf16 T=64: equal {torch.equal(a, b)}")
    assert torch.equal(a, b)


@pytest.mark.parametrize("tile,d,dtype", [(16, 64, "f32"), (64, 128, "bf16"), (32, 128, "bf16")])
def test_prefill_ex_scale_against_oracle(tile, d, dtype):
    from paper_2606_09441_amd import sparse_prefill_ex
    wl = W.custom([[150, 64, 40], [33, 17]], tile=tile, hq=4, hkv=2, d=d, dtype=dtype,
                  seed=tile + d, p_la=0.5, p_ca=0.5)
    q, k, v, la, ca = _dev(wl)
    scale = 0.05
    out = sparse_prefill_ex(q, k, v, wl.seg_offsets, wl.prompt_seg_ptr, la, ca, tile=tile,
                            scale=scale)
    torch.cuda.synchronize()
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca, scale=scale)
    err = max_abs(out.float().cpu().numpy(), ref)
    tol = BF16_TOL if dtype == "bf16" else F32_TOL
    say(f"[ex] {dtype} T={tile} D={d} scale {scale}: max-abs {err:.3e}")
    assert err <= tol


def test_one_workspace_serves_consecutive_calls():
    """Two layouts, one workspace sized for the larger, three calls on one
    stream without waiting in between: each output equals its own one-shot
    result."""
    from paper_2606_09441_amd import sparse_prefill, sparse_prefill_ex, workspace_bytes
    big = W.custom([[256, 192, 100], [64, 64, 64]], tile=64, hq=4, hkv=1, d=128, dtype="bf16",
                   seed=5)
    small = W.custom([[70, 33]], tile=64, hq=4, hkv=1, d=128, dtype="bf16", seed=6)
    need = [workspace_bytes(w.seg_offsets, w.prompt_seg_ptr, 4, 1, 128, 64) for w in (big, small)]
    assert need[0] > need[1] > 0
    ws = torch.empty(need[0], dtype=torch.uint8, device=device())
    outs, refs = [], []
    for w in (big, small, big):
        q, k, v, la, ca = _dev(w)
        outs.append(sparse_prefill_ex(q, k, v, w.seg_offsets, w.prompt_seg_ptr, la, ca, tile=64,
                                      workspace=ws))
        refs.append((q, k, v, la, ca, w))
    torch.cuda.synchronize()
    for o, (q, k, v, la, ca, w) in zip(outs, refs):
        r = sparse_prefill(q, k, v, w.seg_offsets, w.prompt_seg_ptr, la, ca, tile=64)
        torch.cuda.synchronize()
        assert torch.equal(o, r)
    say(f"[ex] one workspace of {need[0]} bytes, 3 calls: equal")


@pytest.mark.parametrize("name,kw", [("tiny", {}), ("llama8b_4k", {}), ("custom16", {}),
                                     ("custom128", {})])
def test_layout_form_decode(name, kw):
    """sift_decode_tiles (layout, bit vectors, tile, caller workspace; no
    plan) gives the oracle's lists bit for bit, like the plan's decode."""
    from gpu_helpers import oracle_csr
    from paper_2606_09441_amd import decode_tiles
    if name.startswith("custom"):
        t = int(name[6:])
        wl = W.custom([[300, 64, 129, 75], [5], [1, 64, 0]], tile=t, hq=4, hkv=2, d=64,
                      dtype="f32", seed=t, p_la=0.4, p_ca=0.3)
    else:
        wl = W.make(name, **kw)
    dev = device()
    la = torch.from_numpy(wl.la if wl.la.size else np.zeros(1, np.uint8)).to(dev)
    ca = torch.from_numpy(wl.ca if wl.ca.size else np.zeros(1, np.uint8)).to(dev)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        rp, ci = decode_tiles(wl.seg_offsets, wl.prompt_seg_ptr, la, ca, wl.hq, tile=wl.tile,
                              stream=s)
    s.synchronize()
    rp = rp.cpu().numpy().astype(np.int64)
    ci = ci[: int(rp[-1])].cpu().numpy().astype(np.int64)
    erp, eci = oracle_csr(wl)
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci)
    say(f"[ex] layout-form decode {wl.name} T={wl.tile}: nnz={ci.size} bit-exact")


def test_one_shot_forms_are_stream_ordered():
    """The one-shot forms enqueue everything on the caller's stream: on a
    side stream, several calls queued back to back without a wait (the
    stream-ordered scratch of sift_sparse_prefill, one workspace for
    sift_sparse_prefill_ex) give the plan run's outputs."""
    from paper_2606_09441_amd import Plan, sparse_prefill, sparse_prefill_ex, workspace_bytes
    wl = W.custom([[256, 192, 100], [64, 64, 64]], tile=64, hq=4, hkv=1, d=128, dtype="bf16",
                  seed=5)
    q, k, v, la, ca = _dev(wl)
    with Plan(wl.seg_offsets, wl.prompt_seg_ptr, 4, 1, 128, 64) as plan:
        ref = plan.run(q, k, v, la, ca)
        torch.cuda.synchronize()
    n = workspace_bytes(wl.seg_offsets, wl.prompt_seg_ptr, 4, 1, 128, 64)
    ws = torch.empty(n, dtype=torch.uint8, device=q.device)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    outs = []
    with torch.cuda.stream(s):
        for i in range(6):
            if i % 2:
                outs.append(sparse_prefill_ex(q, k, v, wl.seg_offsets, wl.prompt_seg_ptr, la, ca,
                                              tile=64, workspace=ws, stream=s))
            else:
                outs.append(sparse_prefill(q, k, v, wl.seg_offsets, wl.prompt_seg_ptr, la, ca,
                                           tile=64, stream=s))
    s.synchronize()
    for o in outs:
        assert torch.equal(o, ref)
    say("[ex] 6 one-shot calls queued on a side stream: equal to the plan run")
