"""GPU: K/V in a page pool (sift_plan_run_paged).

The paper's key tiles are KV pages (Sections 4.2-4.3); here every tile is
one page of the pool and a page table maps tiles to pages.  The pool is
built from the same packed K/V in a random page order, with the unused
pages and the unused rows of partial pages set to NaN: the outputs must be
bit-identical to the packed run (same arithmetic on the same values) and
within tolerance of the fp64 oracle."""

import numpy as np
import pytest
import torch

from gpu_helpers import (BF16_TOL, F32_TOL, DevWorkload, max_abs, oracle_layout, page_pool, say,
                         workload)
from oracle import sift_oracle as O
import workloads as W

pytestmark = pytest.mark.gpu


def _check(wl, tol, tag, full_oracle=True):
    dw = DevWorkload(wl)
    try:
        packed = dw.run()
        kp, vp, table = page_pool(wl, dw.k, dw.v)
        paged = dw.plan.run_paged(dw.q, kp, vp, table, dw.la, dw.ca)
        torch.cuda.synchronize()
        assert torch.isfinite(paged.float()).all(), tag
        assert torch.equal(packed, paged), f"{tag}: paged differs from packed"
        if full_oracle:
            ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca)
            err = max_abs(paged.float().cpu().numpy(), ref)
            say(f"[paged] {tag}: bit-identical to packed, max-abs vs oracle {err:.3e}")
            assert err <= tol, (tag, err)
        else:
            say(f"[paged] {tag}: bit-identical to packed")
    finally:
        dw.close()


@pytest.mark.parametrize("tile", [16, 32, 64])
def test_paged_bf16_ragged_layouts(tile):
    """At T < 64 a 64-key step holds 64 / T tiles, each read from its own
    page."""
    wl = W.custom([[300, 64, 129, 75], [5], [1, 64, 0], [200, 131, 70]], tile=tile, hq=8, hkv=2,
                  d=128, dtype="bf16", seed=7, p_la=0.4, p_ca=0.3)
    _check(wl, BF16_TOL, f"bf16 ragged layouts T={tile}")


@pytest.mark.parametrize("tile,d", [(16, 64), (32, 128)])
def test_paged_fp32_layouts(tile, d):
    wl = W.custom([[70, 33, 10], [5], [64, 129, 0]], tile=tile, hq=4, hkv=2, d=d, dtype="f32",
                  seed=tile + d)
    _check(wl, F32_TOL, f"fp32 T={tile} D={d}")


def test_paged_long64k_bit_identical():
    _check(workload("long64k"), BF16_TOL, "64k rho=0.15", full_oracle=False)


def test_paged_argument_errors():
    from paper_2606_09441_amd import SiftError
    wl = W.custom([[130, 64], [70, 20]], tile=64, hq=4, hkv=2, d=128, dtype="bf16", seed=3)
    dw = DevWorkload(wl)
    try:
        kp, vp, table = page_pool(wl, dw.k, dw.v)
        with pytest.raises(SiftError) as e:   # not whole pages
            dw.plan.run_paged(dw.q, kp[:-1], vp[:-1], table, dw.la, dw.ca)
        assert e.value.status == 2
        with pytest.raises(SiftError) as e:   # pools of different heads
            dw.plan.run_paged(dw.q, kp[:, :1].contiguous(), vp, table, dw.la, dw.ca)
        assert e.value.status == 2
        with pytest.raises(SiftError) as e:   # no page table
            dw.plan.run_paged(dw.q, kp, vp, None, dw.la, dw.ca)
        assert e.value.status == 1
        # after a paged run the plan's step lists index the pool: the packed
        # attention over them is refused until the next decode
        dw.plan.run_paged(dw.q, kp, vp, table, dw.la, dw.ca)
        with pytest.raises(SiftError) as e:
            dw.plan.attention_internal(dw.q, dw.k, dw.v)
        assert e.value.status == 7
        dw.plan.decode_internal(dw.la, dw.ca)
        dw.plan.attention_internal(dw.q, dw.k, dw.v)
        torch.cuda.synchronize()
    finally:
        dw.close()


def test_paged_out_of_range_entries_stay_in_the_pool():
    """Entries outside [0, num_pages) are clamped: the call completes with
    finite values (the result for those tiles is meaningless)."""
    wl = W.custom([[130, 64], [70, 20]], tile=64, hq=4, hkv=2, d=128, dtype="bf16", seed=4)
    dw = DevWorkload(wl)
    try:
        kp, vp, table = page_pool(wl, dw.k, dw.v, extra_pages=0)
        kp = torch.nan_to_num(kp, nan=0.0)
        vp = torch.nan_to_num(vp, nan=0.0)
        bad = table.clone()
        bad[0] = -3
        bad[-1] = 10 ** 6
        out = dw.plan.run_paged(dw.q, kp, vp, bad, dw.la, dw.ca)
        torch.cuda.synchronize()
        assert torch.isfinite(out.float()).all()
    finally:
        dw.close()
