"""Plain fp64 CPU oracle for SIFT's offline metadata extraction.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module; only the tests and the benchmark's CPU-baseline leg do.  It shares no
code with the HIP library.

What it computes (paper: SIFT, arXiv 2606.09441, Sections 4.1, 4.2 and the
offline generation of the metadata in Section 4.4): each document is
prefilled alone, densely and causally, and its attention probabilities
A[p, k] (softmax over the keys k <= p of the same document, per query head)
decide two bit vectors:

* LA (Section 4.1): the lower triangle of A is cut into T x T tiles,
  enumerated (0,0),(1,0),(1,1),(2,0),...; a tile's bit is 1 when at least one
  of its scores exceeds alpha (0.001 in the paper).
* CA (Section 4.2): per KV page of width T, the fraction of the page's scores
  that exceed beta (0.01) is compared with gamma (10%); the page's bit is 1
  when the fraction exceeds gamma.

Readings taken where the paper is loose:

* "Attention score" is the softmax probability (the thresholds 0.001 and 0.01
  are probabilities), per query head; the kv head of query head h is
  h // (Hq / Hkv); the softmax scale is 1/sqrt(D).
* The CA fraction is taken over the page's causal score cells: all (p, k) of
  the document with k in the page and p >= k.  Section 4.2 states the rule per
  page ("fraction of tokens within that page ... greater than beta ... exceeds
  gamma"); Section 3.5 states the same concentration per key column (scores
  >= 0.01 on more than 10% of the column).  Counting the page's whole column
  block is the page-granular form of the Section 3.5 rule, and reduces to it
  for T = 1.
* Comparisons are strict (> alpha, > beta, > gamma), as both sections word
  them.
* Bits are packed MSB first, each (document, head) vector byte aligned
  (Section 4.1); the buffers concatenate, over documents in order, the query
  heads 0..Hq-1 (the document-major layout of the online path).

A threshold decision taken in floating point is only defined up to rounding:
the oracle also reports which bits are *ambiguous*, i.e. would flip if the
deciding probabilities moved by a relative `eps`.  Tests compare the other
bits exactly.

All inputs are widened to float64 exactly.
"""

from __future__ import annotations

import math

import numpy as np

ALPHA = 0.001   # Section 4.1
BETA = 0.01     # Section 4.2
GAMMA = 0.1     # Section 4.2


def num_pages(length: int, tile: int) -> int:
    """P = ceil(L / T) (Section 4.3)."""
    return -(-int(length) // int(tile))


def la_nbytes(P: int) -> int:
    """ceil(P(P+1) / 16) bytes (Section 4.3)."""
    return -(-(P * (P + 1)) // 16)


def ca_nbytes(P: int) -> int:
    """ceil(P / 8) bytes (Section 4.3)."""
    return -(-P // 8)


def pack_msb(bits: np.ndarray, nbytes: int) -> np.ndarray:
    """Bit b goes to byte b // 8, position 7 - b % 8 (MSB first, Section 4.1)."""
    out = np.zeros(nbytes, dtype=np.uint8)
    for b in np.nonzero(np.asarray(bits, dtype=bool))[0]:
        out[b >> 3] |= np.uint8(0x80 >> (b & 7))
    return out


def standalone_probs(q: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """A = causal softmax(scale * q k^T) of one document and one head, fp64.

    q: [L, D], k: [L, D].  Row p is a distribution over keys 0..p."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    L = q.shape[0]
    s = scale * (q @ k.T)
    s[np.triu_indices(L, 1)] = -np.inf
    s -= s.max(axis=1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=1, keepdims=True)


def doc_bits(A: np.ndarray, tile: int, alpha: float = ALPHA, beta: float = BETA,
             gamma: float = GAMMA, eps: float = 1e-4):
    """LA and CA bits of one (document, head) from its probabilities A [L, L].

    Returns (la, ca, la_amb, ca_amb): boolean arrays over the P(P+1)/2 LA bits
    (in enumeration order) and the P CA bits, and which of them are ambiguous
    at relative tolerance eps."""
    L = A.shape[0]
    T = int(tile)
    P = num_pages(L, T)
    causal = np.tril(np.ones((L, L), dtype=bool))
    la, la_amb = [], []
    for i in range(P):                      # tile rows, Section 4.1 order
        r0, r1 = i * T, min(L, (i + 1) * T)
        for j in range(i + 1):
            c0, c1 = j * T, min(L, (j + 1) * T)
            blk = A[r0:r1, c0:c1][causal[r0:r1, c0:c1]]
            mx = blk.max() if blk.size else 0.0
            la.append(mx > alpha)
            la_amb.append(abs(mx - alpha) <= eps * alpha)
    ca, ca_amb = [], []
    for j in range(P):                      # key pages, Section 4.2
        c0, c1 = j * T, min(L, (j + 1) * T)
        col = A[:, c0:c1][causal[:, c0:c1]]
        n = col.size
        cnt = int((col > beta).sum())
        lo = int((col > beta * (1 + eps)).sum())
        hi = int((col > beta * (1 - eps)).sum())
        ca.append(cnt > gamma * n)
        ca_amb.append((lo > gamma * n) != (hi > gamma * n))
    return (np.array(la, dtype=bool), np.array(ca, dtype=bool),
            np.array(la_amb, dtype=bool), np.array(ca_amb, dtype=bool))


def extract_bits(doc_offsets, q, k, hq: int, hkv: int, tile: int, alpha: float = ALPHA,
                 beta: float = BETA, gamma: float = GAMMA, scale: float | None = None,
                 eps: float = 1e-4):
    """Bit vectors of every document, standalone (Section 4.4).

    doc_offsets: [N+1] token offsets of the documents on the packed axis of
    q [tokens, hq, D] and k [tokens, hkv, D].  Returns (la_bytes, ca_bytes,
    la_amb_bytes, ca_amb_bytes): the packed LA and CA buffers, document-major
    with query heads inside each document, and buffers of the same layout
    whose set bits mark ambiguous decisions."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    D = q.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    g = hq // hkv
    la_parts, ca_parts, la_a, ca_a = [], [], [], []
    for d in range(len(doc_offsets) - 1):
        a, b = int(doc_offsets[d]), int(doc_offsets[d + 1])
        P = num_pages(b - a, tile)
        for h in range(hq):
            A = standalone_probs(q[a:b, h], k[a:b, h // g], scale)
            la, ca, lam, cam = doc_bits(A, tile, alpha, beta, gamma, eps)
            la_parts.append(pack_msb(la, la_nbytes(P)))
            ca_parts.append(pack_msb(ca, ca_nbytes(P)))
            la_a.append(pack_msb(lam, la_nbytes(P)))
            ca_a.append(pack_msb(cam, ca_nbytes(P)))
    cat = lambda xs: np.concatenate(xs) if xs else np.zeros(0, dtype=np.uint8)
    return cat(la_parts), cat(ca_parts), cat(la_a), cat(ca_a)


def extract_flops(doc_offsets, hq: int, head_dim: int) -> int:
    """Dense causal QK^T work of the standalone prefill, once: 2 D flop per
    causal cell (p, k), k <= p, of every document and query head."""
    cells = 0
    for d in range(len(doc_offsets) - 1):
        L = int(doc_offsets[d + 1]) - int(doc_offsets[d])
        cells += L * (L + 1) // 2
    return 2 * head_dim * cells * hq
