"""GPU: scores that rise far above the first tiles a row sees.

Section 5.2 keeps the online softmax of dense attention.  The bf16 kernel
forms a tile's weights against the reference max a row took from its first
tile, at whatever magnitude; when a weight, row sum or output overflows
fp32, the launch is done again with the reference following every tile's
max.  Here K rows are scaled up along each segment, so that later tiles
score up to 2^100 (finite weights) or far beyond 2^128 (overflow) times the
first one.  The outputs must still match the fp64 oracle, for every tile
variant and for split query units."""

import numpy as np
import pytest

import workloads as W
from gpu_helpers import BF16_TOL, DevWorkload, max_abs, oracle_layout, say
from oracle import sift_oracle as O

pytestmark = pytest.mark.gpu

RAGGED = [[300, 64, 129, 75], [5], [1, 64, 0], [200, 131, 70], [17, 33, 49]]


def _rising(wl: W.Workload, top: float) -> W.Workload:
    """K rows scaled from 1 at each segment's first token to `top` at its
    last, then rounded to bf16 again."""
    f = np.ones(wl.tokens, np.float64)
    so = wl.seg_offsets
    for s in range(len(so) - 1):
        a, z = int(so[s]), int(so[s + 1])
        if z > a:
            f[a:z] = 1.0 + (top - 1.0) * np.arange(z - a) / max(1, z - a - 1)
    wl.k = W.bf16_round((wl.k * f[:, None, None]).astype(np.float32))
    return wl


def _parity(wl, tag):
    dw = DevWorkload(wl)
    try:
        out = dw.run().float().cpu().numpy()
    finally:
        dw.close()
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca)
    err = max_abs(out, ref)
    say(f"[range] {tag}: max-abs {err:.3e} (tol {BF16_TOL:g})")
    assert np.isfinite(out).all(), tag
    assert err <= BF16_TOL, tag


@pytest.mark.parametrize("tile", [16, 32, 64, 128])
@pytest.mark.parametrize("top", [15.0, 30.0, 80.0])
def test_rising_scores_ragged_layouts(tile, top):
    """top 15: weights up to about 2^100 times a row's first tile, still
    finite, kept by the first pass; 30 and 80: some overflow, the exact pass
    redoes the launch."""
    wl = _rising(W.custom(RAGGED, tile=tile, hq=4, hkv=2, d=128, dtype="bf16", seed=tile + 5,
                          p_la=0.5, p_ca=0.4), top)
    _parity(wl, f"T={tile} K x1..{top:g}")


def test_rising_scores_split_query_units():
    """Eight 512-token documents and a 128-token query: the query units'
    66-step lists run as pieces, each redone on its own and then merged."""
    wl = _rising(W.custom([[512] * 8 + [128]], tile=64, hq=4, hkv=1, d=128, dtype="bf16",
                          seed=21, p_la=0.3, p_ca=0.3), 60.0)
    _parity(wl, "split query units, K x1..60")


def test_falling_and_flat_scores():
    """Scores that fall along the segment (the first reference stays the
    max) and all-equal scores (every weight is 1)."""
    wl = W.custom(RAGGED, tile=64, hq=4, hkv=2, d=128, dtype="bf16", seed=3)
    f = np.ones(wl.tokens)
    so = wl.seg_offsets
    for s in range(len(so) - 1):
        a, z = int(so[s]), int(so[s + 1])
        f[a:z] = np.linspace(40.0, 1.0, max(1, z - a))[: z - a]
    wl.k = W.bf16_round((wl.k * f[:, None, None]).astype(np.float32))
    _parity(wl, "falling scores")
    wl.k = np.zeros_like(wl.k)
    _parity(wl, "flat scores")


def test_redo_flag_is_cleared_for_the_next_launch():
    """A launch that needs the exact pass, then launches that do not, on one
    plan: each matches the oracle (a flag left set would only cost time; a
    flag lost would leave the first launch wrong)."""
    import torch
    from gpu_helpers import DevWorkload
    wl = W.custom(RAGGED, tile=64, hq=4, hkv=2, d=128, dtype="bf16", seed=8, p_la=0.5, p_ca=0.4)
    k_plain = wl.k.copy()
    rising = _rising(W.custom(RAGGED, tile=64, hq=4, hkv=2, d=128, dtype="bf16", seed=8,
                              p_la=0.5, p_ca=0.4), 80.0)
    lay = oracle_layout(wl)
    dw = DevWorkload(wl)
    try:
        for name, kk in (("rising", rising.k), ("plain", k_plain), ("plain again", k_plain)):
            dw.k.copy_(torch.from_numpy(kk).to(dw.k.device).to(dw.k.dtype))
            out = dw.run().float().cpu().numpy()
            ref = O.attention(lay, wl.q, kk, wl.v, wl.la, wl.ca)
            err = max_abs(out, ref)
            say(f"[range] one plan, {name} K: max-abs {err:.3e}")
            assert np.isfinite(out).all() and err <= BF16_TOL, name
    finally:
        dw.close()


def test_huge_values_with_rising_scores():
    """V near 2^100 with scores rising along the segment by about 2^40
    (weights within the first pass's bound): those weights times V overflow
    fp32 in O, which the kernel notices and redoes exactly.  Compared
    relative to the scale."""
    big = 2.0 ** 100
    wl = _rising(W.custom(RAGGED, tile=64, hq=4, hkv=2, d=128, dtype="bf16", seed=12,
                          p_la=0.5, p_ca=0.4), 10.0)
    wl.v = W.bf16_round((wl.v * big).astype(np.float32))
    from gpu_helpers import DevWorkload
    dw = DevWorkload(wl)
    try:
        out = dw.run(out_dtype=None).float().cpu().numpy()
    finally:
        dw.close()
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca)
    err = max_abs(out / big, ref / big)
    say(f"[range] V ~ 2^100, K x1..10: max-abs / 2^100 {err:.3e}")
    assert np.isfinite(out).all()
    assert err <= BF16_TOL


def test_large_finite_weights_need_no_second_pass():
    """Scores rising by up to about 2^80 over a row's first tile: every weight
    is finite, so the first pass keeps its result (no exact pass) and it
    matches the oracle."""
    from gpu_helpers import DevWorkload
    wl = _rising(W.custom(RAGGED, tile=64, hq=4, hkv=2, d=128, dtype="bf16", seed=14,
                          p_la=0.5, p_ca=0.4), 12.0)
    dw = DevWorkload(wl)
    try:
        before = dw.plan.exact_passes()
        out = dw.run().float().cpu().numpy()
        ran = dw.plan.exact_passes() - before
    finally:
        dw.close()
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca)
    err = max_abs(out, ref)
    say(f"[range] K x1..12: max-abs {err:.3e}, exact passes {ran}")
    assert np.isfinite(out).all() and err <= BF16_TOL
    assert ran == 0
