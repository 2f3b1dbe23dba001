"""GPU: seeded random layouts through the whole path.

Each case draws a layout (prompts of 0-6 documents of 1-300 tokens and a
query of 0-100 tokens), a tile size, head counts and bit densities, then
compares the decoded lists with the oracle's bit for bit and the outputs
with the fp64 oracle.  Small layouts take the per-head count and the
cross-list copy; the cases cover every tile size of the bf16 path (adjacent
and gathered steps) and the fp32 path.  Some of them run again with K/V in a
page pool, which must give the packed run's outputs bit for bit."""

import numpy as np
import pytest

from gpu_helpers import (BF16_TOL, F32_TOL, DevWorkload, max_abs, oracle_csr, oracle_layout,
                         page_pool, say, workers)
from oracle import sift_oracle as O
import workloads as W

pytestmark = pytest.mark.gpu


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    f32 = seed % 4 == 3
    tile = int(rng.choice([16, 32, 64] if f32 else [16, 32, 64, 128]))
    hkv = int(rng.choice([1, 2, 4]))
    hq = hkv * int(rng.choice([1, 2, 3]))
    d = int(rng.choice([64, 128])) if f32 else 128
    layout = []
    for _ in range(int(rng.integers(1, 7))):
        docs = [int(x) for x in rng.integers(1, 301, size=int(rng.integers(0, 7)))]
        layout.append(docs + [int(rng.integers(0, 101))])
    p_la, p_ca = float(rng.uniform(0.05, 0.9)), float(rng.uniform(0.05, 0.9))
    return layout, dict(tile=tile, hq=hq, hkv=hkv, d=d, dtype="f32" if f32 else "bf16",
                        seed=seed, p_la=p_la, p_ca=p_ca)


@pytest.mark.parametrize("seed", range(48))
def test_random_layout(seed):
    layout, kw = _case(seed)
    wl = W.custom(layout, **kw)
    tag = (f"seed {seed}: T={kw['tile']} {kw['hq']}/{kw['hkv']} heads D={kw['d']} {kw['dtype']} "
           f"segments={len(wl.seg_offsets) - 1} tokens={wl.tokens}")
    dw = DevWorkload(wl)
    try:
        rp, ci = dw.lists()
        out = dw.run().float().cpu().numpy()
    finally:
        dw.close()
    erp, eci = oracle_csr(wl)
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci), f"{tag}: lists differ"
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca, workers=workers())
    err = max_abs(out, ref)
    tol = F32_TOL if kw["dtype"] == "f32" else BF16_TOL
    say(f"[rand] {tag}: lists bit-exact, max-abs {err:.3e}")
    assert np.isfinite(out).all(), tag
    assert err <= tol, (tag, err)


@pytest.mark.parametrize("seed", range(0, 48, 3))
def test_random_layout_paged(seed):
    layout, kw = _case(seed)
    wl = W.custom(layout, **kw)
    dw = DevWorkload(wl)
    try:
        packed = dw.run()
        kp, vp, table = page_pool(wl, dw.k, dw.v, seed=seed)
        paged = dw.plan.run_paged(dw.q, kp, vp, table, dw.la, dw.ca)
        import torch
        torch.cuda.synchronize()
        assert torch.isfinite(paged.float()).all()
        assert torch.equal(packed, paged), f"seed {seed}: paged differs from packed"
    finally:
        dw.close()
    say(f"[rand] seed {seed} T={kw['tile']} {kw['dtype']}: paged bit-identical to packed")
