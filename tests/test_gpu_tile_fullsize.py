"""GPU: the tile-size variants at the full sizes they are benchmarked at.

The 64K layer (48/8 heads, D 128) with bits made at T = 16, 32 and 128 (the
storage tile of Section 4.3 takes T = 16; Table 1's arithmetic implies
T = 128), and the 16K layer (32/8 heads) at rho = 0.2 with T = 32 and 16.  Lists
are compared bit for bit; outputs on sampled rows of every head and on every
query row of the first and last head, against the fp64 oracle."""

import numpy as np
import pytest
import torch

from gpu_helpers import (BF16_TOL, DevWorkload, max_abs, oracle_csr, oracle_layout, sample_rows,
                         say, workers, workload)
from oracle import sift_oracle as O

pytestmark = pytest.mark.gpu

CASES = [("long64k", {"tile": 16}), ("long64k", {"tile": 32}), ("long64k", {"tile": 128}),
         ("llama8b_16k", {"rho": 0.2, "tile": 32}), ("llama8b_16k", {"rho": 0.2, "tile": 16})]


@pytest.mark.parametrize("name,kw", CASES, ids=[f"{n}-T{kw['tile']}" for n, kw in CASES])
def test_fullsize_tile_variant(name, kw):
    wl = workload(name, **kw)
    tag = f"{wl.name}"
    say(f"[tfull] {tag}: tokens={wl.tokens} T={wl.tile}")
    q0 = int(wl.seg_offsets[-2])
    rows = sample_rows(wl, 48, seed=kw["tile"])
    heads = [0, wl.hq - 1]
    dw = DevWorkload(wl)
    try:
        rp, ci = dw.lists()
        out = dw.run()
        got_rows = out[torch.from_numpy(rows).to(out.device)].float().cpu().numpy()
        got_query = out[q0:, heads].float().cpu().numpy()
        del out
    finally:
        dw.close()
        torch.cuda.empty_cache()
    erp, eci = oracle_csr(wl)
    assert np.array_equal(rp, erp), f"{tag}: row_ptr differs"
    assert np.array_equal(ci, eci), f"{tag}: col_idx differs"
    say(f"[tfull] {tag}: nnz={ci.size} bit-exact")
    lay = oracle_layout(wl)
    ref = O.attention(lay, wl.q, wl.k, wl.v, wl.la, wl.ca, rows=rows, workers=workers())
    err1 = max_abs(got_rows, ref)
    refq = O.attention(lay, wl.q, wl.k, wl.v, wl.la, wl.ca, rows=np.arange(q0, wl.tokens),
                       heads=heads, workers=workers())[:, heads]
    err2 = max_abs(got_query, refq)
    say(f"[tfull] {tag}: {len(rows)} sampled rows x {wl.hq} heads max-abs {err1:.3e}; "
        f"{wl.tokens - q0} query rows x heads {heads} max-abs {err2:.3e}")
    assert np.isfinite(got_rows).all() and np.isfinite(got_query).all()
    assert max(err1, err2) <= BF16_TOL, f"{tag}: max-abs {err1}, {err2}"
