"""Shared helpers of the GPU parity tests: device upload of a workload, the
library's lists and outputs, and the oracle's expected values.  The oracle
and the library never see each other: both receive the same generated
arrays."""

from __future__ import annotations

import functools
import sys

import numpy as np

import workloads as W
from oracle import sift_oracle as O

BF16_TOL = 2e-2     # max-abs, bf16 path vs fp64 oracle
F32_TOL = 1e-5      # max-abs, fp32 path vs fp64 oracle


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU (run them on the MI355X box)"
    return torch.device("cuda:0")


@functools.lru_cache(maxsize=8)
def workload(name: str, dense: bool = False, **kw) -> W.Workload:
    wl = W.make(name, **kw)
    return W.all_ones(wl) if dense else wl


class DevWorkload:
    """A workload's arrays on the GPU, plus its plan."""

    def __init__(self, wl: W.Workload):
        import torch

        from paper_2606_09441_amd import Plan

        dev = device()
        dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        self.wl = wl
        self.q = torch.from_numpy(wl.q).to(dev).to(dt).contiguous()
        self.k = torch.from_numpy(wl.k).to(dev).to(dt).contiguous()
        self.v = torch.from_numpy(wl.v).to(dev).to(dt).contiguous()
        self.la = torch.from_numpy(wl.la if wl.la.size else np.zeros(1, np.uint8)).to(dev)
        self.ca = torch.from_numpy(wl.ca if wl.ca.size else np.zeros(1, np.uint8)).to(dev)
        self.plan = Plan(wl.seg_offsets, wl.prompt_seg_ptr, wl.hq, wl.hkv, wl.d, wl.tile)

    def lists(self):
        import torch
        rp, ci = self.plan.decode(self.la, self.ca)
        torch.cuda.synchronize()
        rp = rp.cpu().numpy().astype(np.int64)
        return rp, ci[: int(rp[-1])].cpu().numpy().astype(np.int64)

    def run(self, out_dtype=None):
        import torch
        out = self.plan.run(self.q, self.k, self.v, self.la, self.ca, out_dtype=out_dtype)
        torch.cuda.synchronize()
        return out

    def close(self):
        self.plan.close()


def oracle_layout(wl: W.Workload) -> O.Layout:
    return O.Layout(wl.seg_offsets, wl.prompt_seg_ptr, wl.tile, wl.hq)


def oracle_csr(wl: W.Workload):
    return O.csr_lists(oracle_layout(wl), wl.la, wl.ca)


def sample_rows(wl: W.Workload, n: int, seed: int = 0) -> np.ndarray:
    """Rows worth checking: first, last and boundary rows of every segment
    (tile edges, partial tails), all kinds of segment, plus random rows."""
    rng = np.random.default_rng(seed)
    so = wl.seg_offsets
    cand = set()
    for s in range(len(so) - 1):
        a, z = int(so[s]), int(so[s + 1])
        if z <= a:
            continue
        for r in (a, a + 1, z - 1, min(z - 1, a + wl.tile - 1), min(z - 1, a + wl.tile)):
            cand.add(r)
    cand = sorted(cand)
    if len(cand) > n // 2:
        cand = sorted(rng.choice(cand, n // 2, replace=False).tolist())
    rest = rng.choice(wl.tokens, max(0, n - len(cand)), replace=False)
    return np.array(sorted(set(cand) | set(int(x) for x in rest)), dtype=np.int64)


def max_abs(a, b) -> float:
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64)))) if np.size(a) else 0.0


def workers() -> int:
    """Threads for the oracle: the host cores this process may use, at most 16."""
    import os
    return max(1, min(16, len(os.sched_getaffinity(0))))


def page_pool(wl, k, v, extra_pages=5, seed=0):
    """Page pool [num_pages * T, Hkv, D] of a workload's K/V (device tensors
    k, v) in a random page order, with NaN in the unused pages and page
    tails, and its page table."""
    import torch
    lay = oracle_layout(wl)
    M = lay.num_tiles
    T = wl.tile
    rng = np.random.default_rng(seed)
    num_pages = M + extra_pages
    perm = rng.permutation(num_pages)[:M].astype(np.int32)
    kp = torch.full((num_pages * T, wl.hkv, wl.d), float("nan"), dtype=k.dtype, device=k.device)
    vp = torch.full_like(kp, float("nan"))
    for m in range(M):
        _, _, a, cnt = lay.tile_span(m)
        p = int(perm[m])
        kp[p * T: p * T + cnt] = k[a: a + cnt]
        vp[p * T: p * T + cnt] = v[a: a + cnt]
    return kp, vp, torch.from_numpy(perm).to(k.device)
