"""GPU: element-by-element parity of the 64K layer (48/8 heads, D 128, 32 x
2048-token documents + a 512-token query, T = 64), on the bits at 15% tile
density and on all-ones bits (dense causal).

Two slices of the full output are compared with the fp64 oracle:
  * all 512 query rows for all 48 heads: each query unit is long enough to
    run as several pieces whose partial results are merged;
  * every row of the first and the last query head (66,048 rows each)."""

import functools

import numpy as np
import pytest
import torch

from gpu_helpers import BF16_TOL, DevWorkload, max_abs, oracle_layout, say, workers, workload
from oracle import sift_oracle as O

pytestmark = pytest.mark.gpu

HEADS = [0, 47]


@functools.lru_cache(maxsize=2)
def _gpu_slices(dense: bool):
    """(query rows x all heads, all rows x HEADS) of the library's output."""
    wl = workload("long64k", dense=dense)
    dw = DevWorkload(wl)
    try:
        out = dw.run()
        q0 = int(wl.seg_offsets[-2])
        a = out[q0:].float().cpu().numpy()
        b = out[:, HEADS].float().cpu().numpy()
        del out
    finally:
        dw.close()
        torch.cuda.empty_cache()
    return a, b


@pytest.mark.parametrize("dense", [False, True], ids=["rho0.15", "all-ones"])
def test_long64k_query_rows_all_heads(dense):
    wl = workload("long64k", dense=dense)
    tag = f"64k {'all-ones' if dense else 'rho=0.15'} query rows"
    say(f"[64k] {tag}: running")
    got, _ = _gpu_slices(dense)
    rows = np.arange(int(wl.seg_offsets[-2]), wl.tokens)
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca, rows=rows,
                      workers=workers())
    err = max_abs(got, ref)
    say(f"[64k] {tag}: {len(rows)} rows x {wl.hq} heads, max-abs {err:.3e}")
    assert np.isfinite(got).all()
    assert err <= BF16_TOL, f"{tag}: max-abs {err}"


@pytest.mark.parametrize("dense", [False, True], ids=["rho0.15", "all-ones"])
def test_long64k_all_rows_first_last_head(dense):
    wl = workload("long64k", dense=dense)
    tag = f"64k {'all-ones' if dense else 'rho=0.15'} heads {HEADS}"
    say(f"[64k] {tag}: running")
    _, got = _gpu_slices(dense)
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca, heads=HEADS,
                      workers=workers())[:, HEADS]
    err = max_abs(got, ref)
    say(f"[64k] {tag}: {wl.tokens} rows x {len(HEADS)} heads, max-abs {err:.3e}")
    assert np.isfinite(got).all()
    assert err <= BF16_TOL, f"{tag}: max-abs {err}"
