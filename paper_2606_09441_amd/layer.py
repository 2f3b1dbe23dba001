"""Decoder-layer prefill slice around the sparse attention.

One pre-norm layer of the Llama-3.1-8B architecture (the model of Section 6):
RMSNorm, the q/k/v projections, rotary embedding (libsift's `sift_rope`), the
sparse attention (libsift's plan: decode + attention over the bits), the
output projection and residual, then optionally the SwiGLU MLP.  The
projections are library GEMMs (torch.matmul -> hipBLASLt on bf16); the norm
and the MLP activation are torch elementwise ops.  It serves to measure the
per-layer prefill time of sparse against dense attention, the quantity the
paper's time-to-first-token results aggregate (Section 7).
"""

from __future__ import annotations

from ._lib import _torch, rope_


class PrefillLayer:
    """weights: dict of torch bf16 device tensors w_in, Wqkv, Wo and, for the
    MLP, w_post, Wg, Wu, Wd (shapes as in workloads.layer_weights);
    inv_freq: float32 device tensor [D/2]."""

    def __init__(self, weights: dict, hq: int, hkv: int, head_dim: int, inv_freq, eps: float = 1e-5):
        self.w = weights
        self.hq, self.hkv, self.d = hq, hkv, head_dim
        self.inv_freq = inv_freq
        self.eps = eps
        qd, kd = hq * head_dim, hkv * head_dim
        W = weights["Wqkv"]
        # row blocks of Wqkv: each projection writes a dense [tokens, heads, D]
        self.Wq, self.Wk, self.Wv = W[:qd], W[qd:qd + kd], W[qd + kd:qd + 2 * kd]

    def _norm(self, x, w):
        torch = _torch()
        xf = x.float()
        y = xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + self.eps) * w.float()
        return y.to(torch.bfloat16)

    def attention_block(self, x, plan, positions, la, ca):
        """x + o_proj(attention(rope(q), rope(k), v)) over the bits la, ca."""
        n = x.shape[0]
        h = self._norm(x, self.w["w_in"])
        q = (h @ self.Wq.T).view(n, self.hq, self.d)
        k = (h @ self.Wk.T).view(n, self.hkv, self.d)
        v = (h @ self.Wv.T).view(n, self.hkv, self.d)
        rope_(q, k, positions, self.inv_freq)
        a = plan.run(q, k, v, la, ca)
        return x + a.view(n, self.hq * self.d) @ self.w["Wo"].T

    def forward(self, x, plan, positions, la, ca, mlp: bool = True):
        torch = _torch()
        x1 = self.attention_block(x, plan, positions, la, ca)
        if not mlp:
            return x1
        h2 = self._norm(x1, self.w["w_post"])
        g = h2 @ self.w["Wg"].T
        u = h2 @ self.w["Wu"].T
        return x1 + (torch.nn.functional.silu(g) * u) @ self.w["Wd"].T
