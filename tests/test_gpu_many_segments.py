"""GPU: layouts of more than 1024 segments.

The count pass keeps a head's segment table in LDS for layouts of up to 1024
segments; larger ones take the per-(head, segment) count and a write pass
that walks every earlier page instead of copying the head's cross list.
Lists bit for bit and outputs against the fp64 oracle, at T = 64 and at
T = 16 (steps of adjacent tiles only on that path)."""

import numpy as np
import pytest

from gpu_helpers import BF16_TOL, DevWorkload, max_abs, oracle_csr, oracle_layout, say, workers
from oracle import sift_oracle as O
import workloads as W

pytestmark = pytest.mark.gpu


def _layout(seed, prompts=212):
    """prompts x (four documents + a query) = 1060 segments."""
    rng = np.random.default_rng(seed)
    return [[int(x) for x in rng.integers(1, 90, size=4)] + [int(rng.integers(1, 40))]
            for _ in range(prompts)]


@pytest.mark.parametrize("tile", [16, 64])
def test_more_segments_than_the_count_pass_holds(tile):
    wl = W.custom(_layout(tile), tile=tile, hq=2, hkv=1, d=128, dtype="bf16", seed=tile,
                  p_la=0.4, p_ca=0.3)
    assert len(wl.seg_offsets) - 1 > 1024
    dw = DevWorkload(wl)
    try:
        rp, ci = dw.lists()
        out = dw.run().float().cpu().numpy()
    finally:
        dw.close()
    erp, eci = oracle_csr(wl)
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci)
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca, workers=workers())
    err = max_abs(out, ref)
    say(f"[segs] T={tile} segments={len(wl.seg_offsets) - 1} tokens={wl.tokens}: lists "
        f"bit-exact, max-abs {err:.3e}")
    assert np.isfinite(out).all()
    assert err <= BF16_TOL, err
