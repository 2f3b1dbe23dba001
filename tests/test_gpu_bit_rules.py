"""GPU: bits that the format says carry nothing never reach the result.

Diagonal tiles are always computed, whatever their stored LA bit says, and
the bits after the last tile of an LA or CA vector only pad it to a whole
byte (Sections 4.1, 4.3).  The inputs here clear the stored diagonal bits of
every other vector, draw the others at random, and set every padding bit
(workloads.scramble_ignored_bits).  The decoded lists must still equal the
oracle's bit for bit, the outputs must stay within tolerance of the oracle,
and they must be bit-identical to the run on the unscrambled bits."""

import numpy as np
import pytest
import torch

from gpu_helpers import (BF16_TOL, F32_TOL, DevWorkload, max_abs, oracle_csr, oracle_layout,
                         say, workers, workload)
from oracle import sift_oracle as O
import workloads as W

pytestmark = pytest.mark.gpu

# page counts 1..12 and partial tiles, so that LA vectors of P(P+1)/2 bits
# and CA vectors of P bits end inside a byte; several prompts, an empty query
RAGGED = [[300, 64, 129, 75], [5], [1, 64, 0], [200, 131, 70], [17, 33, 49, 190]]


def _pair(tile, dtype, seed, d):
    wl = W.custom(RAGGED, tile=tile, hq=4, hkv=2, d=d, dtype=dtype, seed=seed, p_la=0.35,
                  p_ca=0.3)
    return wl, W.scramble_ignored_bits(wl, seed=seed + 1)


def _run(wl, out_dtype=None):
    dw = DevWorkload(wl)
    try:
        rp, ci = dw.lists()
        out = dw.run(out_dtype=out_dtype).cpu()
    finally:
        dw.close()
    return rp, ci, out


def _check(wl, ws, tol, tag):
    say(f"[bits] {tag}: tokens={wl.tokens} T={wl.tile} {wl.dtype}")
    rp_s, ci_s, out_s = _run(ws)
    erp, eci = oracle_csr(ws)
    assert np.array_equal(rp_s, erp), f"{tag}: row_ptr differs from the oracle's"
    assert np.array_equal(ci_s, eci), f"{tag}: col_idx differs from the oracle's"
    ref = O.attention(oracle_layout(ws), ws.q, ws.k, ws.v, ws.la, ws.ca, workers=workers())
    err = max_abs(out_s.float().numpy(), ref)
    assert np.isfinite(out_s.float().numpy()).all()
    assert err <= tol, f"{tag}: max-abs {err}"
    _, _, out_p = _run(wl)
    assert torch.equal(out_s, out_p), f"{tag}: output differs from the unscrambled bits' output"
    say(f"[bits] {tag}: lists bit-exact, max-abs {err:.3e}, identical to unscrambled")


@pytest.mark.parametrize("tile", [16, 32, 64, 128])
def test_ignored_bits_bf16(tile):
    wl, ws = _pair(tile, "bf16", 50 + tile, 128)
    _check(wl, ws, BF16_TOL, f"bf16 T={tile}")


@pytest.mark.parametrize("tile,d", [(16, 64), (32, 128), (64, 64)])
def test_ignored_bits_fp32(tile, d):
    wl, ws = _pair(tile, "f32", 70 + tile, d)
    _check(wl, ws, F32_TOL, f"fp32 T={tile} D={d}")


@pytest.mark.parametrize("name,kw", [("llama8b_4k", {}), ("long64k", {})])
def test_ignored_bits_full_size(name, kw):
    """Full-size inputs: lists bit-exact against the oracle, output
    bit-identical to the run on the unscrambled bits (whose own parity the
    other tests check)."""
    wl = workload(name, **kw)
    ws = W.scramble_ignored_bits(wl, seed=3)
    tag = f"{name} scrambled"
    say(f"[bits] {tag}: tokens={wl.tokens}")
    dw = DevWorkload(wl)
    try:
        out_p = dw.run()
        la_s = torch.from_numpy(ws.la).to(dw.la.device)
        ca_s = torch.from_numpy(ws.ca).to(dw.ca.device)
        rp, ci = dw.plan.decode(la_s, ca_s)
        out_s = dw.plan.run(dw.q, dw.k, dw.v, la_s, ca_s)
        torch.cuda.synchronize()
        same = torch.equal(out_s, out_p)
        rp = rp.cpu().numpy().astype(np.int64)
        ci = ci[: int(rp[-1])].cpu().numpy().astype(np.int64)
    finally:
        dw.close()
    assert same, f"{tag}: output differs from the unscrambled bits' output"
    erp, eci = oracle_csr(ws)
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci), f"{tag}: lists differ"
    say(f"[bits] {tag}: nnz={ci.size} bit-exact, output identical")
