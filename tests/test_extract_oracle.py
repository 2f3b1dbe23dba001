"""Pins of the extraction oracle (oracle/extract_oracle.py) against what the
paper and the mathematics fix, independent of the oracle's own code:

* a pure-Python brute force (math.exp, explicit loops, its own bit packing)
  on small random documents;
* uniform attention (q = 0): A[p, k] = 1/(p+1), so the LA and CA bits have
  closed forms;
* one-hot attention (q_p, k_k orthogonal, a large score on p = k): only
  diagonal LA tiles, CA pages decided by the page's own count;
* softmax invariance: adding one vector to every key of a document shifts
  each row's scores by a constant and changes no bit;
* limits of the thresholds and monotonicity in them;
* the storage sizes of Section 4.3, including its example (P = 8: 36 LA bits,
  8 CA bits)."""

import math

import numpy as np
import pytest

from oracle import extract_oracle as X


def _brute(doc_offsets, q, k, hq, hkv, tile, alpha, beta, gamma):
    """Everything by loops over Python floats."""
    D = len(q[0][0])
    scale = 1.0 / math.sqrt(D)
    g = hq // hkv
    la_out, ca_out = [], []
    for d in range(len(doc_offsets) - 1):
        a, b = doc_offsets[d], doc_offsets[d + 1]
        L = b - a
        P = (L + tile - 1) // tile
        for h in range(hq):
            A = [[0.0] * L for _ in range(L)]
            for p in range(L):
                s = [sum(float(q[a + p][h][x]) * float(k[a + kk][h // g][x]) for x in range(D)) * scale
                     for kk in range(p + 1)]
                m = max(s)
                e = [math.exp(v - m) for v in s]
                z = sum(e)
                for kk in range(p + 1):
                    A[p][kk] = e[kk] / z
            la_bits = []
            for i in range(P):
                for j in range(i + 1):
                    hit = False
                    for p in range(i * tile, min(L, (i + 1) * tile)):
                        for kk in range(j * tile, min(L, (j + 1) * tile)):
                            if kk <= p and A[p][kk] > alpha:
                                hit = True
                    la_bits.append(hit)
            ca_bits = []
            for j in range(P):
                cnt = n = 0
                for kk in range(j * tile, min(L, (j + 1) * tile)):
                    for p in range(kk, L):
                        n += 1
                        cnt += A[p][kk] > beta
                ca_bits.append(cnt > gamma * n)
            for bits in (la_bits, ca_bits):
                nbytes = (len(bits) + 7) // 8
                by = [0] * nbytes
                for idx, bit in enumerate(bits):
                    if bit:
                        by[idx // 8] += 2 ** (7 - idx % 8)
                (la_out if bits is la_bits else ca_out).extend(by)
    return np.array(la_out, dtype=np.uint8), np.array(ca_out, dtype=np.uint8)


@pytest.mark.parametrize("tile,lens,seed", [(2, [5, 1, 9], 0), (3, [13, 7], 1), (4, [16, 3, 11], 2)])
def test_brute_force(tile, lens, seed):
    rng = np.random.default_rng(seed)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(int)
    n = int(offs[-1])
    hq, hkv, D = 2, 1, 4
    q = rng.normal(size=(n, hq, D)) * 2.0
    k = rng.normal(size=(n, hkv, D)) * 2.0
    # thresholds near the typical probabilities of these short rows
    for alpha, beta, gamma in [(0.05, 0.2, 0.3), (0.15, 0.1, 0.5), (0.001, 0.01, 0.1)]:
        la, ca, _, _ = X.extract_bits(offs, q, k, hq, hkv, tile, alpha, beta, gamma)
        bla, bca = _brute(offs.tolist(), q.tolist(), k.tolist(), hq, hkv, tile, alpha, beta, gamma)
        assert np.array_equal(la, bla), (tile, alpha)
        assert np.array_equal(ca, bca), (tile, beta, gamma)


def _unpack(buf, nbits):
    return [(int(buf[b >> 3]) >> (7 - (b & 7))) & 1 for b in range(nbits)]


def test_uniform_attention_closed_form():
    """q = 0: every score ties, A[p, k] = 1/(p+1) for k <= p."""
    L, T, D = 40, 8, 8
    alpha, beta, gamma = 0.05, 0.04, 0.3
    q = np.zeros((L, 1, D))
    k = np.random.default_rng(3).normal(size=(L, 1, D))
    la, ca, la_amb, ca_amb = X.extract_bits([0, L], q, k, 1, 1, T, alpha, beta, gamma)
    P = L // T
    # LA: the largest score of tile (i, j) is in its first row, 1/(iT + 1)
    want_la = [int(1.0 / (i * T + 1) > alpha) for i in range(P) for _ in range(i + 1)]
    assert _unpack(la, P * (P + 1) // 2) == want_la
    assert want_la.count(1) and want_la.count(0)   # the case splits the tiles
    # CA: A[p, k] > beta iff p + 1 < 1/beta, i.e. p <= 23 here
    pmax = math.ceil(1.0 / beta) - 2
    want_ca = []
    for j in range(P):
        cnt = sum(max(0, min(pmax, L - 1) - kk + 1) for kk in range(j * T, (j + 1) * T))
        n = sum(L - kk for kk in range(j * T, (j + 1) * T))
        want_ca.append(int(cnt > gamma * n))
    assert _unpack(ca, P) == want_ca
    assert want_ca.count(1) and want_ca.count(0)
    assert not la_amb.any() and not ca_amb.any()


def test_one_hot_attention():
    """q_p = s e_p, k_k = e_k: A[p, p] = e^s / (e^s + p), the rest tiny."""
    L, T = 20, 4
    s = 30.0
    D = L
    q = np.zeros((L, 1, D))
    k = np.zeros((L, 1, D))
    for p in range(L):
        q[p, 0, p] = s * math.sqrt(D)     # undo the 1/sqrt(D) scale
        k[p, 0, p] = 1.0
    gamma = 0.06
    la, ca, _, _ = X.extract_bits([0, L], q, k, 1, 1, T, 0.001, 0.01, gamma)
    P = L // T
    want_la = [int(j == i) for i in range(P) for j in range(i + 1)]
    assert _unpack(la, P * (P + 1) // 2) == want_la
    # page j: exactly its T diagonal cells exceed beta, out of sum(L - k) cells
    want_ca = [int(T > gamma * sum(L - kk for kk in range(j * T, (j + 1) * T))) for j in range(P)]
    assert _unpack(ca, P) == want_ca
    assert want_ca.count(1) and want_ca.count(0)


def test_row_shift_invariance():
    """k_k + c for every key: scores of row p move by q_p . c, A is unchanged."""
    rng = np.random.default_rng(5)
    offs = [0, 70, 101]
    q = rng.normal(size=(101, 4, 16))
    k = rng.normal(size=(101, 2, 16))
    base = X.extract_bits(offs, q, k, 4, 2, 16, 0.01, 0.02, 0.05)
    k2 = k + rng.normal(size=(1, 2, 16)) * 3.0
    shifted = X.extract_bits(offs, q, k2, 4, 2, 16, 0.01, 0.02, 0.05)
    amb = base[2] | shifted[2]
    assert np.array_equal(base[0] & ~amb, shifted[0] & ~amb)
    amb = base[3] | shifted[3]
    assert np.array_equal(base[1] & ~amb, shifted[1] & ~amb)


def test_threshold_limits_and_monotonicity():
    rng = np.random.default_rng(6)
    offs = [0, 50, 77]
    q = rng.normal(size=(77, 2, 8))
    k = rng.normal(size=(77, 1, 8))
    P = [4, 2]                       # tile 16: 50 -> 4 pages, 27 -> 2 pages
    la_all = sum(2 * X.la_nbytes(p) for p in P)
    ca_all = sum(2 * X.ca_nbytes(p) for p in P)
    la, ca, _, _ = X.extract_bits(offs, q, k, 2, 1, 16, alpha=1.0, beta=1.0, gamma=0.0)
    assert la.size == la_all and ca.size == ca_all
    assert not la.any() and not ca.any()        # a probability never exceeds 1
    la, ca, _, _ = X.extract_bits(offs, q, k, 2, 1, 16, alpha=0.0, beta=0.0, gamma=0.0)
    for buf, nbits in ((la, [p * (p + 1) // 2 for p in P]), (ca, P)):
        pos = 0
        for nb in nbits:
            for _ in range(2):
                n = -(-nb // 8)
                assert _unpack(buf[pos:pos + n], nb) == [1] * nb
                pos += n
    lo = X.extract_bits(offs, q, k, 2, 1, 16, 0.01, 0.01, 0.05)
    hi = X.extract_bits(offs, q, k, 2, 1, 16, 0.03, 0.03, 0.15)
    assert np.array_equal(hi[0] & ~lo[0], np.zeros_like(hi[0]))   # LA(hi) subset of LA(lo)
    assert np.array_equal(hi[1] & ~lo[1], np.zeros_like(hi[1]))


def test_storage_sizes_section_4_3():
    # the example of Section 4.3: about 8 pages per document gives 36 LA bits
    # and 8 CA bits
    assert 8 * 9 // 2 == 36
    assert X.la_nbytes(8) == 5 and X.ca_nbytes(8) == 1
    assert X.num_pages(2048, 64) == 32 and X.la_nbytes(32) == 66 and X.ca_nbytes(32) == 4
    assert X.num_pages(1, 16) == 1 and X.la_nbytes(1) == 1
