"""Plain fp64 CPU oracle for the decoder-layer prefill slice.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module; only the tests do.  It shares no code with the HIP library.

The slice is one pre-norm decoder layer of the Llama-3.1-8B architecture (the
model of Section 6) around SIFT's sparse attention:

    h   = rmsnorm(x) * w_in
    q, k, v = split(h @ Wqkv^T)           (GQA: Hq query heads, Hkv kv heads)
    q, k = rope(q), rope(k)                (rotate-half, per-prompt positions)
    a   = sift_attention(q, k, v, bits)    (oracle/sift_oracle.attention)
    x1  = x + a @ Wo^T
    out = x1 + (silu(g) * u) @ Wd^T,  g, u = rmsnorm(x1) * w_post @ Wg^T, Wu^T

Readings: RMSNorm epsilon 1e-5; the rotary angle of pair i at position p is
the fp32 product p * inv_freq[i] (as the usual fp32 implementations form it),
its cosine and sine are taken in fp64; positions count from 0 at each
prompt's first token.  Everything else is fp64 on the exact input values.
"""

from __future__ import annotations

import numpy as np

from oracle import sift_oracle as O

EPS = 1e-5


def rms_norm(x: np.ndarray, w: np.ndarray, eps: float = EPS) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(w, np.float64)


def rope(x: np.ndarray, positions: np.ndarray, inv_freq: np.ndarray) -> np.ndarray:
    """x [tokens, heads, D]; rotate pairs (i, i + D/2) by angle fp32(p * f_i)."""
    x = np.asarray(x, dtype=np.float64)
    half = x.shape[2] // 2
    ang = (np.asarray(positions, np.float32)[:, None] * np.asarray(inv_freq, np.float32)[None, :])
    ang = ang.astype(np.float64)                                      # [tokens, half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def layer_slice(lay: O.Layout, x, w: dict, la, ca, positions, inv_freq, hq: int, hkv: int,
                d: int, mlp: bool = True) -> np.ndarray:
    """The slice above on tokens x [tokens, hidden]; w holds w_in, Wqkv, Wo
    (and w_post, Wg, Wu, Wd when mlp)."""
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[0]
    h = rms_norm(x, w["w_in"])
    qkv = h @ np.asarray(w["Wqkv"], np.float64).T
    q = qkv[:, : hq * d].reshape(n, hq, d)
    k = qkv[:, hq * d: (hq + hkv) * d].reshape(n, hkv, d)
    v = qkv[:, (hq + hkv) * d:].reshape(n, hkv, d)
    q, k = rope(q, positions, inv_freq), rope(k, positions, inv_freq)
    a = O.attention(lay, q, k, v, la, ca)
    x1 = x + a.reshape(n, hq * d) @ np.asarray(w["Wo"], np.float64).T
    if not mlp:
        return x1
    h2 = rms_norm(x1, w["w_post"])
    g = h2 @ np.asarray(w["Wg"], np.float64).T
    u = h2 @ np.asarray(w["Wu"], np.float64).T
    return x1 + (silu(g) * u) @ np.asarray(w["Wd"], np.float64).T
