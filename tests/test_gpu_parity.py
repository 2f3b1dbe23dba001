"""GPU parity: the HIP library through its C ABI against the fp64 oracle.

Lists must match bit for bit; outputs within max-abs 2e-2 (bf16 path) or
1e-5 (fp32 path), on the same seeded inputs.  Small layouts are compared on
every element; the full-size configurations on every list entry and on
sampled output rows (the oracle computes those rows one by one)."""

import numpy as np
import pytest
import torch

from gpu_helpers import (BF16_TOL, F32_TOL, DevWorkload, max_abs, oracle_csr, oracle_layout,
                         sample_rows, say, workload)
from oracle import sift_oracle as O
import workloads as W

pytestmark = pytest.mark.gpu


def _check_lists(wl, tag):
    say(f"[lists] {tag}: tokens={wl.tokens} hq={wl.hq}")
    dw = DevWorkload(wl)
    try:
        rp, ci = dw.lists()
    finally:
        dw.close()
    erp, eci = oracle_csr(wl)
    assert rp.shape == erp.shape
    bad = np.nonzero(rp != erp)[0]
    assert bad.size == 0, f"{tag}: row_ptr differs first at row {bad[0]}: {rp[bad[0]]} vs {erp[bad[0]]}"
    assert np.array_equal(ci, eci), f"{tag}: col_idx differs"
    say(f"[lists] {tag}: nnz={ci.size} bit-exact")


# ---------------------------------------------------------------------------
# decoded lists, bit-exact
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("name,kw", [
    ("tiny", {}),
    ("llama8b_4k", {}),
    ("llama8b_16k", {"rho": 0.1}),
    ("llama8b_16k", {"rho": 0.2}),
    ("llama8b_16k", {"rho": 0.4}),
    ("ragged_x8", {}),
])
def test_lists_bitexact(name, kw):
    _check_lists(workload(name, **kw), f"{name}{kw}")


def test_lists_bitexact_dense():
    _check_lists(workload("llama8b_4k", dense=True), "llama8b_4k all-ones")


def test_lists_bitexact_long64k():
    _check_lists(workload("long64k"), "long64k rho=0.15")


@pytest.mark.parametrize("seed", range(4))
def test_lists_bitexact_random_layouts(seed):
    rng = np.random.default_rng(100 + seed)
    prompts = []
    for _ in range(int(rng.integers(1, 4))):
        nd = int(rng.integers(0, 5))
        prompts.append([int(rng.integers(1, 300)) for _ in range(nd)] + [int(rng.integers(0, 200))])
    tile = int(rng.choice([16, 32, 64]))
    wl = W.custom(prompts, tile=tile, hq=4, hkv=2, d=64, dtype="f32", seed=seed,
                  p_la=float(rng.uniform(0, 1)), p_ca=float(rng.uniform(0, 1)))
    _check_lists(wl, f"random layout {prompts} T={tile}")


# ---------------------------------------------------------------------------
# attention outputs
# ---------------------------------------------------------------------------


def _full_parity(wl, tol, out_dtype=None, heads=None, tag=""):
    dw = DevWorkload(wl)
    try:
        out = dw.run(out_dtype=out_dtype).float().cpu().numpy()
    finally:
        dw.close()
    lay = oracle_layout(wl)
    ref = O.attention(lay, wl.q, wl.k, wl.v, wl.la, wl.ca, heads=heads)
    hs = list(range(wl.hq)) if heads is None else list(heads)
    err = max_abs(out[:, hs], ref[:, hs])
    say(f"[attn] {tag}: max-abs {err:.3e} (tol {tol:g})")
    assert np.isfinite(out).all()
    assert err <= tol, f"{tag}: max-abs {err}"
    return err


def _sampled_parity(wl, tol, n_rows, out_dtype=None, tag="", heads=None):
    dw = DevWorkload(wl)
    try:
        out = dw.run(out_dtype=out_dtype).float().cpu().numpy()
    finally:
        dw.close()
    rows = sample_rows(wl, n_rows)
    lay = oracle_layout(wl)
    ref = O.attention(lay, wl.q, wl.k, wl.v, wl.la, wl.ca, rows=rows, heads=heads)
    hs = list(range(wl.hq)) if heads is None else list(heads)
    err = max_abs(out[rows][:, hs], ref[:, hs])
    say(f"[attn] {tag}: {len(rows)} rows x {len(hs)} heads, max-abs {err:.3e} (tol {tol:g})")
    assert np.isfinite(out).all()
    assert err <= tol, f"{tag}: max-abs {err}"
    return err


def test_attention_tiny_fp32():
    _full_parity(workload("tiny"), F32_TOL, tag="tiny fp32")


@pytest.mark.parametrize("tile,d", [(16, 64), (32, 128), (64, 64)])
def test_attention_fp32_layouts(tile, d):
    wl = W.custom([[70, 33, 10], [5], [64, 129, 0], [1, 2, 3]], tile=tile, hq=4, hkv=2, d=d,
                  dtype="f32", seed=tile + d)
    _full_parity(wl, F32_TOL, tag=f"fp32 T={tile} D={d} ragged layout")


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
def test_attention_bf16_ragged_layouts(out_dtype):
    # several tiles, partial tails, odd page counts (unpaired M-blocks), an
    # empty query, one-token documents, several prompts in one call
    wl = W.custom([[300, 64, 129, 75], [5], [1, 64, 0], [200, 131, 70]], tile=64, hq=8, hkv=2,
                  d=128, dtype="bf16", seed=7, p_la=0.4, p_ca=0.3)
    _full_parity(wl, BF16_TOL, out_dtype=out_dtype, tag=f"bf16 ragged layouts out={out_dtype}")


def test_attention_bf16_dense_small():
    wl = W.all_ones(W.custom([[256, 192, 100], [64, 64, 64]], tile=64, hq=4, hkv=1, d=128,
                             dtype="bf16", seed=11))
    _full_parity(wl, BF16_TOL, tag="bf16 all-ones small")


def test_attention_llama4k():
    wl = workload("llama8b_4k")
    _full_parity(wl, BF16_TOL, heads=[0, 5, 18, 31], tag="llama8b_4k 4 heads all rows")
    _sampled_parity(wl, BF16_TOL, 48, tag="llama8b_4k all heads sampled rows")


@pytest.mark.parametrize("rho", [0.1, 0.2, 0.4])
def test_attention_16k_sampled(rho):
    _sampled_parity(workload("llama8b_16k", rho=rho), BF16_TOL, 40, tag=f"16k rho={rho}")


def test_attention_long64k_sampled():
    _sampled_parity(workload("long64k"), BF16_TOL, 40, tag="64k rho=0.15")


def test_attention_long64k_dense_sampled():
    _sampled_parity(workload("long64k", dense=True), BF16_TOL, 24, tag="64k all-ones")


def test_attention_ragged_sampled():
    _sampled_parity(workload("ragged_x8"), BF16_TOL, 64, tag="ragged x8")


# ---------------------------------------------------------------------------
# properties
# ---------------------------------------------------------------------------


def test_unlisted_tiles_are_never_read():
    """NaN in K and V of tiles absent from an M-block's list leaves that
    M-block's output finite and within tolerance of the oracle of the
    poisoned input (which reads allowed keys only) and of the clean run.  (The
    query rows do see those tiles and come out NaN, which sends the launch
    through the exact pass, so the two runs may differ by rounding; a read of
    a NaN tile would make the output NaN, whatever its weight.)"""
    wl = workload("llama8b_4k")
    lay = oracle_layout(wl)
    base = DevWorkload(wl)
    try:
        ref = base.run().float().cpu().numpy()
    finally:
        base.close()
    # head 0: pick M-blocks of the last document and tiles they skip
    lists = O.tile_lists(lay, wl.la, wl.ca, heads=[0])
    doc = lay.segs[-2]
    picked = []
    for i in range(doc.pages):
        m = doc.tile_base + i
        lst = set(lists[(0, m)])
        skip = [n for n in range(lay.prompt_segs(0)[0].tile_base, m) if n not in lst]
        if skip:
            picked.append((m, skip))
    assert picked
    # poison, for kv head 0, every token of a tile skipped by ALL picked M-blocks
    common = set.intersection(*[set(s) for _, s in picked])
    assert common
    k2, v2 = wl.k.copy(), wl.v.copy()
    for n in common:
        _, _, a, cnt = lay.tile_span(n)
        k2[a:a + cnt, 0] = np.nan
        v2[a:a + cnt, 0] = np.nan
    import dataclasses
    wl2 = dataclasses.replace(wl, k=k2, v=v2)
    dw = DevWorkload(wl2)
    try:
        out = dw.run().float().cpu().numpy()
    finally:
        dw.close()
    rows = np.concatenate([np.arange(lay.tile_span(m)[2], lay.tile_span(m)[2] + lay.tile_span(m)[3])
                           for m, _ in picked])
    assert np.isfinite(out[rows, 0]).all()
    # the oracle of the poisoned input reads only the allowed keys
    want = O.attention(lay, wl.q, k2, v2, wl.la, wl.ca, rows=rows, heads=[0])[:, 0]
    worst = max_abs(out[rows, 0], want)
    assert worst <= BF16_TOL, worst
    assert max_abs(out[rows, 0], ref[rows, 0]) <= BF16_TOL
    q0 = int(wl.seg_offsets[-2])
    assert np.isnan(out[q0:, 0]).any(), "the poisoned tiles did not reach the query rows"
    say(f"[nan] {len(picked)} M-blocks finite and within {worst:.2e} of the oracle, "
        f"{len(common)} poisoned tiles")


def test_run_to_run_bit_identical():
    dw = DevWorkload(workload("llama8b_16k", rho=0.2))
    try:
        a = dw.run().cpu()
        b = dw.run().cpu()
    finally:
        dw.close()
    assert torch.equal(a, b)


def test_one_shot_prefill_matches_plan_run():
    from paper_2606_09441_amd import sparse_prefill
    wl = workload("llama8b_4k")
    dw = DevWorkload(wl)
    try:
        a = dw.run()
        b = sparse_prefill(dw.q, dw.k, dw.v, wl.seg_offsets, wl.prompt_seg_ptr, dw.la, dw.ca,
                           tile=wl.tile)
        torch.cuda.synchronize()
    finally:
        dw.close()
    assert torch.equal(a, b)


def test_decode_capacity_is_checked():
    from paper_2606_09441_amd import SiftError
    wl = workload("tiny")
    dw = DevWorkload(wl)
    try:
        cap = dw.plan.info["list_capacity"]
        small = torch.empty(cap - 1, dtype=torch.int32, device=dw.q.device)
        with pytest.raises(SiftError) as e:
            dw.plan.decode(dw.la, dw.ca, col_idx=small)
        assert e.value.status == 5
    finally:
        dw.close()


def test_attention_over_given_lists_matches_plan_run():
    """sift_sparse_attention (lists given by the caller, merged on the
    device) and sift_plan_run (lists decoded from the bits) agree exactly,
    also when the given lists are padded with out-of-range entries."""
    wl = W.custom([[300, 64, 129, 75], [5], [1, 64, 0], [200, 131, 70]], tile=64, hq=8, hkv=2,
                  d=128, dtype="bf16", seed=7, p_la=0.4, p_ca=0.3)
    dw = DevWorkload(wl)
    try:
        a = dw.run()
        rp, ci = dw.plan.decode(dw.la, dw.ca)
        b = dw.plan.attention(dw.q, dw.k, dw.v, rp, ci)
        torch.cuda.synchronize()
        assert torch.equal(a, b)
        # the same lists with entries that must be skipped: a tile of another
        # prompt and a tile after the M-block, inserted in every list
        rph = rp.cpu().numpy().astype(np.int64)
        cih = ci.cpu().numpy()[: rph[-1]]
        M = dw.plan.info["num_tiles"]
        new_rp, new_ci = [0], []
        for r in range(len(rph) - 1):
            m = r % M
            lst = cih[rph[r]:rph[r + 1]].tolist()
            new_ci.extend([-5] + lst + [M + 3])
            new_rp.append(len(new_ci))
        rp2 = torch.tensor(new_rp, dtype=torch.int32, device=dw.q.device)
        ci2 = torch.tensor(new_ci, dtype=torch.int32, device=dw.q.device)
        c = dw.plan.attention(dw.q, dw.k, dw.v, rp2, ci2)
        torch.cuda.synchronize()
        assert torch.equal(a, c)
    finally:
        dw.close()


def test_attention_llama4k_fp32_output_split_units():
    """fp32 output with split query units: the pieces' partials are fp32 and
    the merge reads them as such (llama 4K: 3 pieces per query unit)."""
    _full_parity(workload("llama8b_4k"), BF16_TOL, out_dtype=torch.float32, heads=[0, 7, 31],
                 tag="llama8b_4k fp32 out")


def test_attention_over_given_lists_split_units():
    """The merge of caller-given lists fills the pieces of split query units
    (llama 4K: each query unit's 66-step list runs as 3 pieces) exactly as
    decode does."""
    dw = DevWorkload(workload("llama8b_4k"))
    try:
        a = dw.run()
        rp, ci = dw.plan.decode(dw.la, dw.ca)
        b = dw.plan.attention(dw.q, dw.k, dw.v, rp, ci)
        torch.cuda.synchronize()
        assert torch.equal(a, b)
    finally:
        dw.close()


def test_plan_decode_then_attention_matches_run():
    wl = workload("llama8b_4k")
    dw = DevWorkload(wl)
    try:
        a = dw.run()
        dw.plan.decode_internal(dw.la, dw.ca)
        b = dw.plan.attention_internal(dw.q, dw.k, dw.v)
        torch.cuda.synchronize()
    finally:
        dw.close()
    assert torch.equal(a, b)
