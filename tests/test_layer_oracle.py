"""Pins of the decoder-layer slice oracle (oracle/layer_oracle.py): the
rotary embedding's defining properties with exactly representable angles,
the RMSNorm closed form, and the slice's reduction to textbook causal
attention for a single dense prompt."""

import math

import numpy as np

from oracle import layer_oracle as LO
from oracle import sift_oracle as O


def test_rope_properties():
    rng = np.random.default_rng(0)
    f = np.array([1.0, 0.5, 0.25, 0.125], dtype=np.float32)   # exact fp32 angle products
    q = rng.normal(size=(1, 1, 8))
    k = rng.normal(size=(1, 1, 8))
    assert np.allclose(LO.rope(q, np.array([0]), f), q, atol=0, rtol=0)       # position 0
    for m, n in [(5, 2), (17, 17), (3, 11)]:
        qm, kn = LO.rope(q, np.array([m]), f), LO.rope(k, np.array([n]), f)
        # pairs (i, i + D/2) keep their norms
        assert np.allclose(qm[..., :4] ** 2 + qm[..., 4:] ** 2, q[..., :4] ** 2 + q[..., 4:] ** 2)
        # scores depend on m - n only
        rel = (LO.rope(q, np.array([m - n]), f) * k).sum()
        assert abs((qm * kn).sum() - rel) < 1e-12
        # a rotation by angle a: pair 0 at m rotates by m radians
        x1, x2 = q[0, 0, 0], q[0, 0, 4]
        assert abs(qm[0, 0, 0] - (x1 * math.cos(m) - x2 * math.sin(m))) < 1e-12


def test_rms_norm_closed_form():
    x = np.full((2, 6), 3.0)
    w = np.arange(1, 7, dtype=np.float64)
    y = LO.rms_norm(x, w, eps=0.0)
    assert np.allclose(y, np.ones((2, 6)) * w)
    assert abs(LO.silu(np.array(0.0))) == 0.0 and abs(LO.silu(np.array(40.0)) - 40.0) < 1e-12


def test_slice_reduces_to_textbook_attention():
    """One prompt, one head, all-ones bits, identity-like projections: the
    slice's attention output equals plain causal softmax attention of the
    rotated q and k (numpy, computed here from the definition)."""
    rng = np.random.default_rng(1)
    L, d, T = 40, 8, 16
    hidden = 3 * d
    seg, psp = [0, 30, L], [0, 2]
    lay = O.Layout(seg, psp, T, 1)
    P = O.num_pages(30, T)
    la = np.full(O.la_num_bytes(P), 0xFF, np.uint8)
    ca = np.full(O.ca_num_bytes(P), 0xFF, np.uint8)
    x = rng.normal(size=(L, hidden))
    w = {"w_in": np.ones(hidden), "Wqkv": np.eye(3 * d, hidden), "Wo": np.eye(hidden, d)}
    pos = np.arange(L)
    f = np.array([1.0, 0.1, 0.01, 0.001], dtype=np.float32)
    out = LO.layer_slice(lay, x, w, la, ca, pos, f, 1, 1, d, mlp=False)
    h = x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + LO.EPS)
    q = LO.rope(h[:, None, :d], pos, f)[:, 0]
    k = LO.rope(h[:, None, d:2 * d], pos, f)[:, 0]
    v = h[:, 2 * d:]
    s = q @ k.T / math.sqrt(d)
    s[np.triu_indices(L, 1)] = -np.inf
    p = np.exp(s - s.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    want = x.copy()
    want[:, :d] += p @ v
    assert np.abs(out - want).max() < 1e-12
    # zero projections leave the residual stream unchanged
    w0 = {"w_in": np.ones(hidden), "Wqkv": np.zeros((3 * d, hidden)), "Wo": np.eye(hidden, d),
          "w_post": np.ones(hidden), "Wg": np.zeros((5, hidden)), "Wu": np.zeros((5, hidden)),
          "Wd": np.zeros((hidden, 5))}
    assert np.abs(LO.layer_slice(lay, x, w0, la, ca, pos, f, 1, 1, d) - x).max() == 0.0


def test_mlp_composition_hand_worked():
    """The MLP branch against a case worked by hand (golden
    layer_mlp_example.json): silu on the gate, the up projection as the
    other factor, w_post applied after the second norm, and the norm taken
    of x1 (after the attention residual).  Each wrong reading listed in the
    fixture lands far outside the tolerance."""
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "layer_mlp_example.json")
    g = json.load(open(path))
    lay = O.Layout([0, 1], [0, 1], 16, 1)          # one prompt: a 1-token query
    w = {k: np.asarray(g[k], dtype=np.float64)
         for k in ("w_in", "Wqkv", "Wo", "w_post", "Wg", "Wu", "Wd")}
    x = np.asarray(g["x"], dtype=np.float64)
    out = LO.layer_slice(lay, x, w, np.zeros(0, np.uint8), np.zeros(0, np.uint8), np.array([0]),
                         np.array([1.0], dtype=np.float32), 1, 1, 2)
    want = np.asarray(g["expected"], dtype=np.float64)
    assert np.abs(out - want).max() < 1e-12
    for wrong in g["wrong_readings"].values():
        assert abs(wrong - want[0, 0]) > 1e-2
