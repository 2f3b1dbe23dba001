"""GPU: bf16 attention at T = 16 and T = 32 (Section 4.3 takes T = 16 for
storage).

The bf16 kernel keeps 64-row blocks and 64-key steps: a step is 64 / T key
tiles with a mask of which (row tile, key tile) pairs are listed, the tiles
adjacent ones of one segment, or, over the earlier documents of a document's
rows, any CA-marked pages (gathered).  Lists stay at T and are compared bit
for bit; outputs against the fp64 oracle."""

import numpy as np
import pytest
import torch

from gpu_helpers import BF16_TOL, DevWorkload, max_abs, oracle_csr, oracle_layout, say
from oracle import sift_oracle as O
import workloads as W

pytestmark = pytest.mark.gpu

RAGGED = [[300, 64, 129, 75], [5], [1, 64, 0], [200, 131, 70], [17, 33, 49]]


def _wl(tile, seed, p_la=0.4, p_ca=0.3, layout=RAGGED, hq=8, hkv=2):
    return W.custom(layout, tile=tile, hq=hq, hkv=hkv, d=128, dtype="bf16", seed=seed, p_la=p_la,
                    p_ca=p_ca)


def _parity(wl, tag, out_dtype=None, rows=None):
    dw = DevWorkload(wl)
    try:
        out = dw.run(out_dtype=out_dtype).float().cpu().numpy()
    finally:
        dw.close()
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca, rows=rows)
    err = max_abs(out if rows is None else out[rows], ref)
    say(f"[tsmall] {tag}: max-abs {err:.3e}")
    assert np.isfinite(out).all()
    assert err <= BF16_TOL, (tag, err)


@pytest.mark.parametrize("tile", [16, 32])
def test_small_tile_lists_bitexact(tile):
    wl = _wl(tile, 31)
    dw = DevWorkload(wl)
    try:
        rp, ci = dw.lists()
    finally:
        dw.close()
    erp, eci = oracle_csr(wl)
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci)


@pytest.mark.parametrize("tile", [16, 32])
@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
def test_small_tile_ragged_attention(tile, out_dtype):
    _parity(_wl(tile, 33), f"ragged T={tile} out={out_dtype}", out_dtype=out_dtype)


@pytest.mark.parametrize("tile", [16, 32])
@pytest.mark.parametrize("p_la,p_ca", [(0.1, 0.05), (0.9, 0.8)])
def test_small_tile_sparse_and_dense_bits(tile, p_la, p_ca):
    _parity(_wl(tile, 35, p_la, p_ca), f"T={tile} p_la={p_la} p_ca={p_ca}")


@pytest.mark.parametrize("tile", [16, 32])
def test_small_tile_all_ones(tile):
    wl = W.all_ones(_wl(tile, 37, layout=[[256, 192, 100], [64, 64, 64]], hq=4, hkv=1))
    _parity(wl, f"all-ones T={tile}")


@pytest.mark.parametrize("tile", [16, 32])
def test_small_tile_split_query_units_sampled(tile):
    wl = _wl(tile, 39, 0.3, 0.2, layout=[[1024, 1024, 1024, 256]])
    rng = np.random.default_rng(0)
    rows = np.sort(np.concatenate([np.arange(3072, 3328), rng.choice(3072, 150, replace=False)]))
    _parity(wl, f"split query units T={tile}", rows=rows)


@pytest.mark.parametrize("tile", [16, 32])
def test_small_tile_given_lists(tile):
    """Caller lists make steps of adjacent tiles only (no gathering): a
    different grouping of the same keys, so compared with the oracle."""
    wl = _wl(tile, 41, 0.5, 0.4, hq=4)
    dw = DevWorkload(wl)
    try:
        a = dw.run().float().cpu().numpy()
        rp, ci = dw.plan.decode(dw.la, dw.ca)
        b = dw.plan.attention(dw.q, dw.k, dw.v, rp, ci).float().cpu().numpy()
    finally:
        dw.close()
    ref = O.attention(oracle_layout(wl), wl.q, wl.k, wl.v, wl.la, wl.ca)
    ea, eb = max_abs(a, ref), max_abs(b, ref)
    say(f"[tsmall] T={tile}: decoded lists max-abs {ea:.3e}, caller lists {eb:.3e}")
    assert np.isfinite(b).all()
    assert ea <= BF16_TOL and eb <= BF16_TOL, (ea, eb)
