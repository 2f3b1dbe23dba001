"""GPU: the decoder-layer prefill slice (RMSNorm, q/k/v GEMMs, sift_rope,
sparse attention, o_proj, SwiGLU MLP) against the fp64 slice oracle, and
sift_rope alone.

The slice's GEMMs and elementwise steps round to bf16 between steps (as a
bf16 model does); the oracle keeps fp64 throughout.  The tolerance is stated
relative to the output's scale: 2% of max |output| (about 5 bf16 rounding
steps of the unit-scale activations)."""

import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import device, oracle_layout, say
from oracle import layer_oracle as LO

pytestmark = pytest.mark.gpu


def test_rope_matches_oracle():
    from paper_2606_09441_amd import rope_
    dev = device()
    rng = np.random.default_rng(0)
    n, hq, hkv, d = 300, 4, 2, 128
    q = W.bf16_round(rng.normal(size=(n, hq, d)).astype(np.float32) * 2)
    k = W.bf16_round(rng.normal(size=(n, hkv, d)).astype(np.float32) * 2)
    pos = np.sort(rng.integers(0, 70000, size=n)).astype(np.int32)    # up to a 64K prompt
    f = W.rope_inv_freq(d)
    qd = torch.from_numpy(q).to(dev).bfloat16()
    kd = torch.from_numpy(k).to(dev).bfloat16()
    rope_(qd, kd, torch.from_numpy(pos).to(dev), torch.from_numpy(f).to(dev))
    torch.cuda.synchronize()
    for got, x, tag in ((qd, q, "q"), (kd, k, "k")):
        ref = LO.rope(x, pos, f)
        err = np.abs(got.float().cpu().numpy() - ref).max()
        say(f"[layer] rope {tag}: max-abs {err:.3e} (max |x| {np.abs(ref).max():.2f})")
        assert err <= 2 ** -7 * np.abs(ref).max()       # within one bf16 ulp of the largest value


@pytest.mark.parametrize("mlp", [False, True])
@pytest.mark.parametrize("tile", [64, 128])
def test_layer_slice_matches_oracle(mlp, tile):
    from paper_2606_09441_amd import Plan
    from paper_2606_09441_amd.layer import PrefillLayer
    dev = device()
    hq, hkv, d = 4, 2, 128
    hidden, inter = hq * d, 2 * hq * d
    wl = W.custom([[300, 129, 75], [200, 70]], tile=tile, hq=hq, hkv=hkv, d=d, dtype="bf16", seed=5,
                  p_la=0.5, p_ca=0.4)
    n = wl.tokens
    w = W.layer_weights(hidden, hq, hkv, d, inter, seed=1)
    x = W.layer_input(n, hidden, seed=2)
    pos = W.prompt_positions(wl.seg_offsets, wl.prompt_seg_ptr)
    f = W.rope_inv_freq(d)
    layer = PrefillLayer({k: torch.from_numpy(v).to(dev).bfloat16() for k, v in w.items()}, hq, hkv,
                         d, torch.from_numpy(f).to(dev))
    plan = Plan(wl.seg_offsets, wl.prompt_seg_ptr, hq, hkv, d, tile)
    try:
        out = layer.forward(torch.from_numpy(x).to(dev).bfloat16(), plan,
                            torch.from_numpy(pos).to(dev), torch.from_numpy(wl.la).to(dev),
                            torch.from_numpy(wl.ca).to(dev), mlp=mlp)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy()
    finally:
        plan.close()
    ref = LO.layer_slice(oracle_layout(wl), x, w, wl.la, wl.ca, pos, f, hq, hkv, d, mlp=mlp)
    err = np.abs(got - ref).max()
    scale = np.abs(ref).max()
    say(f"[layer] slice T={tile} mlp={mlp}: max-abs {err:.3e}, max |out| {scale:.2f}")
    assert err <= 0.02 * scale
