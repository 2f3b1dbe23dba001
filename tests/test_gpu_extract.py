"""GPU: offline metadata extraction (sift_extract_bits) against the fp64
extraction oracle (Sections 4.1, 4.2, 4.4).

The bits are compared exactly, except where the oracle marks the decision
as ambiguous: a deciding probability within a relative 1e-4 of its
threshold, where the GPU's fp32 scores and the oracle's fp64 ones may round
to different sides.  Each test also checks that such bits are rare, so the
comparison is not vacuous."""

import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import BF16_TOL, device, max_abs, say, workload
from oracle import extract_oracle as X
from oracle import sift_oracle as O

pytestmark = pytest.mark.gpu


def _draw(lens, hq, hkv, d, seed, qscale=1.0):
    rng = np.random.default_rng(seed)
    n = int(sum(lens))
    q = W.bf16_round(rng.normal(size=(n, hq, d)).astype(np.float32) * qscale)
    k = W.bf16_round(rng.normal(size=(n, hkv, d)).astype(np.float32))
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return offs, q, k


def _gpu_bits(offs, q, k, tile, alpha, beta, gamma):
    from paper_2606_09441_amd import extract_bits
    dev = device()
    qd = torch.from_numpy(q).to(dev).to(torch.bfloat16)
    kd = torch.from_numpy(k).to(dev).to(torch.bfloat16)
    la, ca = extract_bits(qd, kd, offs, tile=tile, alpha=alpha, beta=beta, gamma=gamma)
    torch.cuda.synchronize()
    return la.cpu().numpy(), ca.cpu().numpy()


def _compare(tag, got, want, amb):
    assert got.shape == want.shape, tag
    diff = np.unpackbits(got ^ want)
    ambb = np.unpackbits(amb)
    bad = int((diff & ~ambb).sum())
    flips = int((diff & ambb).sum())
    ones = int(np.unpackbits(want).sum())
    say(f"[extract] {tag}: {want.size} bytes, {ones} bits set, {int(ambb.sum())} ambiguous "
        f"({flips} differ), {bad} wrong")
    assert bad == 0, tag
    assert ambb.sum() <= max(2, diff.size // 200), tag


CASES = [
    # tile, D, document lengths, hq, hkv, q scale
    (16, 64, [130, 64, 1, 257, 45], 4, 2, 1.0),
    (32, 128, [300, 33, 96], 4, 1, 1.0),
    (64, 128, [513, 64, 200, 7], 4, 2, 1.0),
    (16, 128, [190, 128], 2, 2, 2.5),
    (64, 64, [1000], 2, 1, 2.0),
    (128, 128, [300, 129, 64, 1], 4, 2, 1.5),
    (128, 64, [700, 128], 2, 1, 1.0),
]


@pytest.mark.parametrize("tile,d,lens,hq,hkv,qs", CASES)
@pytest.mark.parametrize("thr", [(0.001, 0.01, 0.1), (0.01, 0.02, 0.05)])
def test_extract_matches_oracle(tile, d, lens, hq, hkv, qs, thr):
    offs, q, k = _draw(lens, hq, hkv, d, seed=tile + d + len(lens), qscale=qs)
    la, ca = _gpu_bits(offs, q, k, tile, *thr)
    ela, eca, ala, aca = X.extract_bits(offs, q, k, hq, hkv, tile, *thr)
    tag = f"T={tile} D={d} docs={lens} thr={thr}"
    _compare(tag + " LA", la, ela, ala)
    _compare(tag + " CA", ca, eca, aca)


@pytest.mark.parametrize("thr", [(X.ALPHA, X.BETA, X.GAMMA), (0.01, 0.005, 0.05)])
def test_extract_long64k_documents_sampled(thr):
    """The 64K layer's 32 documents of 2048 tokens, 48 query heads, T = 64:
    the whole extraction on the GPU, a sample of (document, head) vectors
    against the oracle.  With the paper's thresholds these near-uniform
    synthetic scores set every LA bit and no CA bit; the second set splits
    both."""
    wl = workload("long64k")
    docs = wl.seg_offsets[: wl.prompt_seg_ptr[1]]            # the documents' boundaries
    offs = np.asarray(docs, dtype=np.int32)
    n = int(offs[-1])
    q, k = wl.q[:n], wl.k[:n]
    la, ca = _gpu_bits(offs, q, k, 64, *thr)
    P = 32
    la_n, ca_n = X.la_nbytes(P), X.ca_nbytes(P)
    rng = np.random.default_rng(1)
    g = wl.hq // wl.hkv
    for d, h in zip(rng.choice(32, 6, replace=False), rng.choice(wl.hq, 6)):
        a, b = int(offs[d]), int(offs[d + 1])
        A = X.standalone_probs(q[a:b, h], k[a:b, h // g], 1.0 / np.sqrt(wl.d))
        lab, cab, lam, cam = X.doc_bits(A, 64, *thr)
        i_la = (d * wl.hq + h) * la_n
        i_ca = (d * wl.hq + h) * ca_n
        _compare(f"64k doc {d} head {h} LA", la[i_la:i_la + la_n], X.pack_msb(lab, la_n),
                 X.pack_msb(lam, la_n))
        _compare(f"64k doc {d} head {h} CA", ca[i_ca:i_ca + ca_n], X.pack_msb(cab, ca_n),
                 X.pack_msb(cam, ca_n))


def test_extracted_bits_drive_the_online_path():
    """Bits made by the extractor for the documents of a prompt feed the
    online path (Section 4.4: extracted offline, consumed at query time); the
    attention over them matches the oracle's attention over the same bits."""
    from paper_2606_09441_amd import Plan
    lens = [256, 192, 320]
    qlen = 100
    hq, hkv, d, T = 4, 2, 128, 64
    seg = np.array([0, 256, 448, 768, 868], dtype=np.int32)
    rng = np.random.default_rng(9)
    n = int(seg[-1])
    q = W.bf16_round(rng.normal(size=(n, hq, d)).astype(np.float32))
    k = W.bf16_round(rng.normal(size=(n, hkv, d)).astype(np.float32))
    v = W.bf16_round(rng.normal(size=(n, hkv, d)).astype(np.float32))
    docs = seg[:4]
    la, ca = _gpu_bits(docs, q[: docs[-1]], k[: docs[-1]], T, X.ALPHA, X.BETA, X.GAMMA)
    dev = device()
    lay = O.Layout(seg.tolist(), [0, 4], T, hq)
    ref = O.attention(lay, q, k, v, la, ca)
    plan = Plan(seg, np.array([0, 4], dtype=np.int32), hq, hkv, d, T)
    try:
        t = lambda x: torch.from_numpy(x).to(dev).to(torch.bfloat16)
        out = plan.run(t(q), t(k), t(v), torch.from_numpy(la).to(dev), torch.from_numpy(ca).to(dev))
        torch.cuda.synchronize()
        err = max_abs(out.float().cpu().numpy(), ref)
    finally:
        plan.close()
    say(f"[extract] prompt of {lens} + query {qlen}: extracted bits, attention max-abs {err:.3e}")
    assert err <= BF16_TOL
    assert 0 < np.unpackbits(la).sum() < np.unpackbits(la).size   # the bits select, not all or none


def test_extract_empty_and_single_token_documents():
    offs, q, k = _draw([1, 1, 2], 2, 1, 64, seed=3)
    la, ca = _gpu_bits(offs, q, k, 16, X.ALPHA, X.BETA, X.GAMMA)
    ela, eca, _, _ = X.extract_bits(offs, q, k, 2, 1, 16)
    assert np.array_equal(la, ela) and np.array_equal(ca, eca)
