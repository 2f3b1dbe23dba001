"""GPU: bf16 attention at T = 128 (the tile of Table 1's arithmetic).

Each 128-token tile reaches the bf16 kernel as two 64-row blocks and up to
two 64-key steps; lists stay at T = 128 and are compared bit for bit, the
outputs against the fp64 oracle."""

import numpy as np
import pytest
import torch

from gpu_helpers import BF16_TOL, DevWorkload, max_abs, oracle_csr, oracle_layout, say
from oracle import sift_oracle as O
import workloads as W

pytestmark = pytest.mark.gpu

# ragged: partial last tiles of 1..64 and 65..127 tokens, a one-token
# document, an empty query, several prompts
RAGGED = [[300, 64, 129, 75], [5], [1, 128, 0], [200, 131, 70]]


def _lists(wl, tag):
    dw = DevWorkload(wl)
    try:
        rp, ci = dw.lists()
    finally:
        dw.close()
    erp, eci = oracle_csr(wl)
    assert np.array_equal(rp, erp) and np.array_equal(ci, eci), tag
    say(f"[t128] {tag}: lists bit-exact, nnz {ci.size}")


def _parity(wl, tag, out_dtype=None, rows=None):
    dw = DevWorkload(wl)
    try:
        out = dw.run(out_dtype=out_dtype).float().cpu().numpy()
    finally:
        dw.close()
    lay = oracle_layout(wl)
    ref = O.attention(lay, wl.q, wl.k, wl.v, wl.la, wl.ca, rows=rows)
    got = out if rows is None else out[rows]
    err = max_abs(got, ref)
    say(f"[t128] {tag}: max-abs {err:.3e}")
    assert np.isfinite(out).all()
    assert err <= BF16_TOL, (tag, err)


def test_tile128_lists_bitexact():
    wl = W.custom(RAGGED, tile=128, hq=8, hkv=2, d=128, dtype="bf16", seed=21, p_la=0.4, p_ca=0.3)
    _lists(wl, "ragged T=128")


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
def test_tile128_ragged_attention(out_dtype):
    wl = W.custom(RAGGED, tile=128, hq=8, hkv=2, d=128, dtype="bf16", seed=21, p_la=0.4, p_ca=0.3)
    _parity(wl, f"ragged T=128 out={out_dtype}", out_dtype=out_dtype)


def test_tile128_dense_matches_causal():
    wl = W.all_ones(W.custom([[256, 192, 100], [128, 64, 129]], tile=128, hq=4, hkv=1, d=128,
                             dtype="bf16", seed=23))
    _parity(wl, "all-ones T=128")


def test_tile128_split_query_units_sampled():
    """Four documents of 2,048 tokens and a 256-token query: the query units'
    lists (two steps per 128-tile) are cut into pieces and merged."""
    wl = W.custom([[2048, 2048, 2048, 2048, 256]], tile=128, hq=8, hkv=2, d=128, dtype="bf16",
                  seed=25, p_la=0.3, p_ca=0.2)
    dw = DevWorkload(wl)
    try:
        info = dw.plan.info
    finally:
        dw.close()
    lists_units = 8 * (4 * 16 + 2)
    say(f"[t128] work units {info['num_work_units']} for {lists_units} list units")
    assert info["num_work_units"] > lists_units      # some units are split
    rng = np.random.default_rng(0)
    rows = np.sort(np.concatenate([np.arange(8192, 8448), rng.choice(8192, 200, replace=False)]))
    _parity(wl, "split query units T=128", rows=rows)


def test_tile128_given_lists_and_paged():
    from paper_2606_09441_amd import Plan
    wl = W.custom(RAGGED, tile=128, hq=4, hkv=2, d=128, dtype="bf16", seed=27, p_la=0.5, p_ca=0.4)
    dw = DevWorkload(wl)
    try:
        a = dw.run()
        rp, ci = dw.plan.decode(dw.la, dw.ca)
        b = dw.plan.attention(dw.q, dw.k, dw.v, rp, ci)
        torch.cuda.synchronize()
        assert torch.equal(a, b), "given lists differ from decoded lists"
        # the same K/V in a pool of 128-row pages, in a random order
        lay = oracle_layout(wl)
        M, T = lay.num_tiles, 128
        perm = np.random.default_rng(3).permutation(M + 3)[:M].astype(np.int32)
        kp = torch.full(((M + 3) * T, wl.hkv, wl.d), float("nan"), dtype=dw.k.dtype, device=dw.k.device)
        vp = torch.full_like(kp, float("nan"))
        for m in range(M):
            _, _, s, n = lay.tile_span(m)
            kp[perm[m] * T: perm[m] * T + n] = dw.k[s: s + n]
            vp[perm[m] * T: perm[m] * T + n] = dw.v[s: s + n]
        c = dw.plan.run_paged(dw.q, kp, vp, torch.from_numpy(perm).to(dw.q.device), dw.la, dw.ca)
        torch.cuda.synchronize()
        assert torch.equal(a, c), "paged differs from packed"
        say("[t128] given lists and paged K/V: bit-identical to the decoded packed run")
    finally:
        dw.close()
