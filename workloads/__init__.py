"""Seeded synthetic RAG-shaped inputs for SIFT sparse prefill.

This module only makes inputs.  It holds none of the hot path's arithmetic:
no bit decoding and no masked attention.  Both the HIP library's tests and the
fp64 oracle consume what it returns, and neither imports the other.

A prompt is documents followed by a user query (Section 3.1 of the paper).
Q, K and V are drawn i.i.d. N(0, 1) per token; documents get "heavy-hitter"
key positions (2% of positions per document and kv head, K row scaled by 4)
so that attention mass concentrates the way Section 3.4 describes.  The two
bit vectors per (document, query head) come from that document's standalone
causal attention, as the offline step of Section 4.4 does: the local vector
keeps the top fraction rho of lower-triangle tiles by attention mass (ties to
the lower bit index) plus the diagonal, the cross vector keeps the top
fraction rho of key pages by column mass.  These inputs stand in for the
paper's LongBench prompts, which are not used here.

Values are rounded to bf16 (round to nearest even) for the bf16 configs and
returned as float32 arrays holding those exact bf16 values.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np

__all__ = ["Workload", "make", "CONFIGS", "all_ones", "scramble_ignored_bits", "custom", "bf16_round", "pack_msb", "layer_weights",
           "layer_input", "rope_inv_freq", "prompt_positions"]


@dataclass
class Workload:
    name: str
    seg_offsets: np.ndarray      # int32 [S+1], packed token axis
    prompt_seg_ptr: np.ndarray   # int32 [B+1]; last segment of a prompt = its query
    tile: int
    hq: int
    hkv: int
    d: int
    dtype: str                   # "f32" or "bf16": the arithmetic type of the inputs
    q: np.ndarray                # float32 [L, hq, d]
    k: np.ndarray                # float32 [L, hkv, d]
    v: np.ndarray                # float32 [L, hkv, d]
    la: np.ndarray               # uint8, local-attention vectors
    ca: np.ndarray               # uint8, cross-attention vectors
    meta: dict = field(default_factory=dict)

    @property
    def tokens(self) -> int:
        return int(self.seg_offsets[-1])


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bf16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000))
    return r.view(np.float32)


def pack_msb(bits: np.ndarray) -> np.ndarray:
    """Pack 0/1 values most-significant-bit first, zero padded to a byte."""
    return np.packbits(np.asarray(bits, dtype=np.uint8), bitorder="big")


def _pages(n: int, t: int) -> int:
    return -(-n // t)


# ----------------------------------------------------------------------------
# bitmap synthesis
# ----------------------------------------------------------------------------


def _standalone_masses(qd: np.ndarray, kd: np.ndarray, tile: int, hq: int, hkv: int):
    """Tile masses of one document's standalone causal attention.

    Returns (la_mass [hq, P(P+1)/2] in lower-triangle enumeration order,
    ca_mass [hq, P]).  Computed in float32 with torch on the CPU."""
    import torch

    Ld, _, D = qd.shape
    P = _pages(Ld, tile)
    g = hq // hkv
    tri_i, tri_j = np.tril_indices(P)          # row-major: (0,0),(1,0),(1,1),...
    la_mass = np.zeros((hq, len(tri_i)), dtype=np.float64)
    ca_mass = np.zeros((hq, P), dtype=np.float64)
    qt = torch.from_numpy(np.ascontiguousarray(qd.transpose(1, 0, 2)))
    kt = torch.from_numpy(np.ascontiguousarray(kd.transpose(1, 0, 2)))
    causal = torch.ones(Ld, Ld, dtype=torch.bool).tril()
    pad = P * tile - Ld
    hc = max(1, min(hq, (1 << 28) // (Ld * Ld * 4)))
    for h0 in range(0, hq, hc):
        hs = list(range(h0, min(hq, h0 + hc)))
        qh = qt[hs]
        kh = kt[[h // g for h in hs]]
        s = torch.matmul(qh, kh.transpose(1, 2)) * (1.0 / math.sqrt(D))
        s.masked_fill_(~causal, float("-inf"))
        a = torch.softmax(s, dim=-1)
        if pad:
            a = torch.nn.functional.pad(a, (0, pad, 0, pad))
        tm = a.view(len(hs), P, tile, P, tile).sum(dim=(2, 4)).double().numpy()
        la_mass[hs] = tm[:, tri_i, tri_j]
        ca_mass[hs] = a.sum(dim=1).view(len(hs), P, tile).sum(dim=-1).double().numpy()
    return la_mass, ca_mass


def _top_bits(mass: np.ndarray, frac: float) -> np.ndarray:
    n = mass.shape[0]
    kk = min(n, max(0, math.ceil(frac * n - 1e-9)))
    order = np.argsort(-mass, kind="stable")    # ties -> lower bit index first
    bits = np.zeros(n, dtype=np.uint8)
    bits[order[:kk]] = 1
    return bits


def _doc_bitmaps(la_mass, ca_mass, P: int, rho) -> tuple[list[np.ndarray], list[np.ndarray]]:
    """Per query head: packed LA and CA vectors of one document."""
    hq = la_mass.shape[0]
    rho = np.broadcast_to(np.asarray(rho, dtype=np.float64), (hq,))
    diag = np.array([i * (i + 1) // 2 + i for i in range(P)])
    la_v, ca_v = [], []
    for h in range(hq):
        lb = _top_bits(la_mass[h], rho[h])
        lb[diag] = 1
        la_v.append(pack_msb(lb))
        ca_v.append(pack_msb(_top_bits(ca_mass[h], rho[h])))
    return la_v, ca_v


def _bernoulli_bitmaps(rng, P: int, hq: int, p: float):
    la_v, ca_v = [], []
    diag = np.array([i * (i + 1) // 2 + i for i in range(P)])
    for _ in range(hq):
        lb = (rng.random(P * (P + 1) // 2) < p).astype(np.uint8)
        lb[diag] = 1
        la_v.append(pack_msb(lb))
        ca_v.append(pack_msb((rng.random(P) < p).astype(np.uint8)))
    return la_v, ca_v


# ----------------------------------------------------------------------------
# document and prompt assembly
# ----------------------------------------------------------------------------


@dataclass
class _Doc:
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    la: list
    ca: list


def _draw_qkv(rng, n, hq, hkv, d, bf16: bool):
    q = rng.standard_normal((n, hq, d), dtype=np.float32)
    k = rng.standard_normal((n, hkv, d), dtype=np.float32)
    v = rng.standard_normal((n, hkv, d), dtype=np.float32)
    if bf16:
        q, k, v = bf16_round(q), bf16_round(k), bf16_round(v)
    return q, k, v


def _heavy_hitters(rng, k: np.ndarray, frac: float = 0.02, factor: float = 4.0):
    n, hkv, _ = k.shape
    nh = math.ceil(frac * n)
    for g in range(hkv):
        pos = rng.choice(n, size=nh, replace=False)
        k[pos, g, :] *= factor            # exact in bf16 and fp32


def _assemble(name, prompts, tile, hq, hkv, d, dtype, meta):
    """prompts: list of (docs: list[_Doc], query (q, k, v))."""
    seg_offsets = [0]
    prompt_seg_ptr = [0]
    qs, ks, vs, las, cas = [], [], [], [], []
    for docs, (qq, kq, vq) in prompts:
        for doc in docs:
            seg_offsets.append(seg_offsets[-1] + doc.q.shape[0])
            qs.append(doc.q)
            ks.append(doc.k)
            vs.append(doc.v)
            las.extend(doc.la)
            cas.extend(doc.ca)
        seg_offsets.append(seg_offsets[-1] + qq.shape[0])
        qs.append(qq)
        ks.append(kq)
        vs.append(vq)
        prompt_seg_ptr.append(prompt_seg_ptr[-1] + len(docs) + 1)
    cat = lambda xs: np.ascontiguousarray(np.concatenate(xs, axis=0))
    la = np.concatenate(las).astype(np.uint8) if las else np.zeros(0, np.uint8)
    ca = np.concatenate(cas).astype(np.uint8) if cas else np.zeros(0, np.uint8)
    return Workload(name, np.asarray(seg_offsets, np.int32), np.asarray(prompt_seg_ptr, np.int32),
                    tile, hq, hkv, d, dtype, cat(qs), cat(ks), cat(vs), la, ca, meta)


def _rag_prompt(rng, doc_lens, query_len, tile, hq, hkv, d, rho, hh=4.0):
    """Draw order: Q/K/V of every document and the query, then heavy hitters
    (K rows scaled by hh), then bitmaps."""
    raw = [_draw_qkv(rng, n, hq, hkv, d, True) for n in doc_lens]
    query = _draw_qkv(rng, query_len, hq, hkv, d, True)
    for _, k, _ in raw:
        _heavy_hitters(rng, k, factor=hh)
    docs = []
    for (q, k, v) in raw:
        la_m, ca_m = _standalone_masses(q, k, tile, hq, hkv)
        la_v, ca_v = _doc_bitmaps(la_m, ca_m, _pages(q.shape[0], tile), rho)
        docs.append(_Doc(q, k, v, la_v, ca_v))
    return docs, query


# ----------------------------------------------------------------------------
# the five configurations
# ----------------------------------------------------------------------------


def _tiny(seed=0, **_):
    rng = np.random.default_rng(seed)
    T, hq, hkv, d = 16, 2, 1, 64
    lens = [128, 128]
    raw = [_draw_qkv(rng, n, hq, hkv, d, False) for n in lens]
    query = _draw_qkv(rng, 32, hq, hkv, d, False)
    docs = []
    for (q, k, v) in raw:
        la_v, ca_v = _bernoulli_bitmaps(rng, _pages(q.shape[0], T), hq, 0.3)
        docs.append(_Doc(q, k, v, la_v, ca_v))
    return _assemble("tiny", [(docs, query)], T, hq, hkv, d, "f32",
                     {"rho": 0.3, "docs": lens, "query": 32})


def _llama(seed=0, rho=0.2, tile=64, **_):
    rng = np.random.default_rng(seed)
    docs, query = _rag_prompt(rng, [512] * 8, 128, tile, 32, 8, 128, rho)
    return _assemble("llama8b_4k" + ("" if tile == 64 else f"_t{tile}"), [(docs, query)], tile, 32,
                     8, 128, "bf16",
                     {"rho": rho, "docs": [512] * 8, "query": 128})


def _mid(seed=0, rho=0.2, tile=64, **_):
    rng = np.random.default_rng(seed)
    docs, query = _rag_prompt(rng, [1024] * 16, 256, tile, 32, 8, 128, rho)
    return _assemble(f"llama8b_16k_rho{rho:g}" + ("" if tile == 64 else f"_t{tile}"), [(docs, query)],
                     tile, 32, 8, 128, "bf16",
                     {"rho": rho, "docs": [1024] * 16, "query": 256})


def _long(seed=0, rho=0.15, hq=48, hkv=8, tile=64, hh=4.0, **_):
    rng = np.random.default_rng(seed)
    docs, query = _rag_prompt(rng, [2048] * 32, 512, tile, hq, hkv, 128, rho, hh)
    return _assemble(f"long64k_{hq}x{hkv}_rho{rho:g}" + ("" if tile == 64 else f"_t{tile}")
                     + ("" if hh == 4.0 else f"_hh{hh:g}"),
                     [(docs, query)], tile, hq, hkv, 128, "bf16",
                     {"rho": rho, "docs": [2048] * 32, "query": 512, "heavy_hitter_scale": hh})


def _ragged(seed=0, **_):
    rng = np.random.default_rng(seed)
    T, hq, hkv, d = 64, 32, 8, 128
    n_pool, n_prompts = 24, 8
    # layout first: pool lengths, prompt compositions, query lengths
    pool_lens = [int(min(2048, max(256, round(int(rng.integers(256, 2049)) / 64) * 64)))
                 for _ in range(n_pool)]
    comps = []
    for _ in range(n_prompts):
        nd = int(rng.integers(4, 13))
        comps.append([int(x) for x in rng.permutation(n_pool)[:nd]])
    qlens = [int(rng.integers(64, 513)) for _ in range(n_prompts)]
    # then Q/K/V, heavy hitters, bitmaps
    raw = [_draw_qkv(rng, n, hq, hkv, d, True) for n in pool_lens]
    queries = [_draw_qkv(rng, n, hq, hkv, d, True) for n in qlens]
    for _, k, _ in raw:
        _heavy_hitters(rng, k)
    rhos = rng.uniform(0.05, 0.5, size=(n_pool, hq))
    pool = []
    for i, (q, k, v) in enumerate(raw):
        la_m, ca_m = _standalone_masses(q, k, T, hq, hkv)
        la_v, ca_v = _doc_bitmaps(la_m, ca_m, _pages(q.shape[0], T), rhos[i])
        pool.append(_Doc(q, k, v, la_v, ca_v))
    prompts = [([pool[i] for i in comp], queries[b]) for b, comp in enumerate(comps)]
    return _assemble("ragged_x8", prompts, T, hq, hkv, d, "bf16",
                     {"pool_lens": pool_lens, "compositions": comps, "query_lens": qlens,
                      "rho_range": [0.05, 0.5]})


CONFIGS = {
    "tiny": _tiny,
    "llama8b_4k": _llama,
    "llama8b_16k": _mid,
    "long64k": _long,
    "ragged_x8": _ragged,
}


def make(name: str, seed: int = 0, **kw) -> Workload:
    """Build a named configuration.  Extra keywords: rho (density knob) and
    tile (16, 32, 64 or 128) for the RAG configs; hq/hkv and hh (the
    heavy-hitter K scale, default 4) for long64k."""
    return CONFIGS[name](seed=seed, **kw)


def all_ones(wl: Workload) -> Workload:
    """The same prompt with every tile bit set (dense causal attention)."""
    la_parts, ca_parts = [], []
    for b in range(len(wl.prompt_seg_ptr) - 1):
        s0, s1 = int(wl.prompt_seg_ptr[b]), int(wl.prompt_seg_ptr[b + 1]) - 1
        for s in range(s0, s1):
            P = _pages(int(wl.seg_offsets[s + 1] - wl.seg_offsets[s]), wl.tile)
            for _ in range(wl.hq):
                la_parts.append(pack_msb(np.ones(P * (P + 1) // 2, np.uint8)))
                ca_parts.append(pack_msb(np.ones(P, np.uint8)))
    la = np.concatenate(la_parts) if la_parts else np.zeros(0, np.uint8)
    ca = np.concatenate(ca_parts) if ca_parts else np.zeros(0, np.uint8)
    return replace(wl, name=wl.name + "_dense", la=la, ca=ca, meta={**wl.meta, "all_ones": True})


def scramble_ignored_bits(wl: Workload, seed: int = 0) -> Workload:
    """The same input with every bit the format says to ignore changed.

    Diagonal tiles are always computed, whatever their stored bit says, and
    the bits after the last tile of a vector (padding to a whole byte) carry
    nothing (Sections 4.1, 4.3).  Here the stored diagonal bits of every
    other vector (in buffer order) are cleared and those of the rest drawn
    at random, and every padding bit of every LA and CA vector is set."""
    rng = np.random.default_rng(seed)
    la = wl.la.copy()
    ca = wl.ca.copy()
    la_off = ca_off = 0
    ordinal = 0
    for b in range(len(wl.prompt_seg_ptr) - 1):
        s0, s1 = int(wl.prompt_seg_ptr[b]), int(wl.prompt_seg_ptr[b + 1]) - 1
        for s in range(s0, s1):               # documents; the last segment is the query
            P = _pages(int(wl.seg_offsets[s + 1] - wl.seg_offsets[s]), wl.tile)
            n_la, n_ca = P * (P + 1) // 2, P
            b_la, b_ca = -(-n_la // 8), -(-n_ca // 8)
            diag = np.array([i * (i + 1) // 2 + i for i in range(P)], dtype=np.int64)
            for _ in range(wl.hq):
                bits = np.unpackbits(la[la_off:la_off + b_la], bitorder="big")
                bits[diag] = 0 if ordinal % 2 == 0 else rng.integers(0, 2, size=P)
                bits[n_la:] = 1
                la[la_off:la_off + b_la] = np.packbits(bits, bitorder="big")
                cb = np.unpackbits(ca[ca_off:ca_off + b_ca], bitorder="big")
                cb[n_ca:] = 1
                ca[ca_off:ca_off + b_ca] = np.packbits(cb, bitorder="big")
                la_off += b_la
                ca_off += b_ca
                ordinal += 1
    assert la_off == la.size and ca_off == ca.size
    return replace(wl, name=wl.name + "_scrambled", la=la, ca=ca,
                   meta={**wl.meta, "ignored_bits_scrambled": seed})


def custom(seg_lens_per_prompt, tile, hq, hkv, d, dtype, seed=0, p_la=0.3, p_ca=0.3) -> Workload:
    """Small random layouts for parity tests: seg_lens_per_prompt is a list of
    prompts, each a list of document lengths followed by the query length.
    Bits are Bernoulli(p_la / p_ca) with diagonals set."""
    rng = np.random.default_rng(seed)
    prompts = []
    for lens in seg_lens_per_prompt:
        *dl, ql = lens
        docs = []
        for n in dl:
            q, k, v = _draw_qkv(rng, n, hq, hkv, d, dtype == "bf16")
            la_v, ca_v = [], []
            P = _pages(n, tile)
            diag = np.array([i * (i + 1) // 2 + i for i in range(P)])
            for _ in range(hq):
                lb = (rng.random(P * (P + 1) // 2) < p_la).astype(np.uint8)
                lb[diag] = 1
                la_v.append(pack_msb(lb))
                ca_v.append(pack_msb((rng.random(P) < p_ca).astype(np.uint8)))
            docs.append(_Doc(q, k, v, la_v, ca_v))
        query = _draw_qkv(rng, ql, hq, hkv, d, dtype == "bf16")
        prompts.append((docs, query))
    return _assemble("custom", prompts, tile, hq, hkv, d, dtype, {"p_la": p_la, "p_ca": p_ca})


# ----------------------------------------------------------------------------
# Inputs of the decoder-layer prefill slice (a Llama-3.1-8B-shaped layer)
# ----------------------------------------------------------------------------


def layer_weights(hidden: int, hq: int, hkv: int, d: int, inter: int, seed: int = 0) -> dict:
    """Random-init weights of one pre-norm decoder layer, bf16 values in
    float32 arrays: w_in, w_post [hidden]; Wqkv [(hq + 2 hkv) d, hidden];
    Wo [hidden, hq d]; Wg, Wu [inter, hidden]; Wd [hidden, inter].  Matrices
    are N(0, 1/fan_in) so that activations keep unit scale."""
    rng = np.random.default_rng(seed)

    def mat(rows, cols):
        return bf16_round((rng.standard_normal((rows, cols)) / math.sqrt(cols)).astype(np.float32))

    return {
        "w_in": bf16_round((1.0 + 0.1 * rng.standard_normal(hidden)).astype(np.float32)),
        "w_post": bf16_round((1.0 + 0.1 * rng.standard_normal(hidden)).astype(np.float32)),
        "Wqkv": mat((hq + 2 * hkv) * d, hidden),
        "Wo": mat(hidden, hq * d),
        "Wg": mat(inter, hidden),
        "Wu": mat(inter, hidden),
        "Wd": mat(hidden, inter),
    }


def layer_input(tokens: int, hidden: int, seed: int = 0) -> np.ndarray:
    """Residual-stream input x [tokens, hidden], N(0, 1), bf16 values."""
    rng = np.random.default_rng(seed + 7919)
    return bf16_round(rng.standard_normal((tokens, hidden)).astype(np.float32))


def rope_inv_freq(d: int, base: float = 500000.0) -> np.ndarray:
    """The rotary frequency table base^(-2i/d), i < d/2 (float32); 500000 is
    Llama-3.1's base (its long-context rescaling of the table is not applied)."""
    return (base ** (-np.arange(0, d, 2, dtype=np.float64) / d)).astype(np.float32)


def prompt_positions(seg_offsets, prompt_seg_ptr) -> np.ndarray:
    """Each token's index within its prompt (int32 [tokens])."""
    so = np.asarray(seg_offsets, dtype=np.int64)
    ps = np.asarray(prompt_seg_ptr, dtype=np.int64)
    pos = np.zeros(int(so[-1]), dtype=np.int32)
    for b in range(len(ps) - 1):
        a, z = int(so[ps[b]]), int(so[ps[b + 1]])
        pos[a:z] = np.arange(z - a, dtype=np.int32)
    return pos
