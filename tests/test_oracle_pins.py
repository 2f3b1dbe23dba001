"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test ties the oracle to something other than itself: a worked example
written by hand from the paper's text, the paper's printed storage figures,
a library routine for the special cases that reduce to textbook attention,
an independent enumeration of the bit stream, or an invariant.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import sift_oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# --------------------------------------------------------------------------
# small helpers that build inputs for the pins (no oracle arithmetic here)
# --------------------------------------------------------------------------


def _pack_msb(bits):
    """Pack a 0/1 list MSB first into bytes (inputs for the pins only)."""
    out = bytearray((len(bits) + 7) // 8)
    for i, b in enumerate(bits):
        if b:
            out[i // 8] |= 0x80 >> (i % 8)
    return list(out)


def _random_case(rng, n_prompts, tile, hq, hkv, D, max_docs=3, max_len=70, query_min=0):
    seg_offsets = [0]
    prompt_seg_ptr = [0]
    for _ in range(n_prompts):
        nd = int(rng.integers(0, max_docs + 1))
        for _ in range(nd):
            seg_offsets.append(seg_offsets[-1] + int(rng.integers(1, max_len)))
        seg_offsets.append(seg_offsets[-1] + int(rng.integers(query_min, max_len)))
        prompt_seg_ptr.append(prompt_seg_ptr[-1] + nd + 1)
    lay = O.Layout(seg_offsets, prompt_seg_ptr, tile, hq)
    la = rng.integers(0, 256, size=lay.la_bytes, dtype=np.uint8)
    ca = rng.integers(0, 256, size=lay.ca_bytes, dtype=np.uint8)
    L = lay.num_tokens
    q = rng.standard_normal((L, hq, D))
    k = rng.standard_normal((L, hkv, D))
    v = rng.standard_normal((L, hkv, D))
    return lay, la, ca, q, k, v


def _sdpa_causal(q, k, v):
    """torch's textbook attention, float64 on the CPU, causal, GQA with
    consecutive grouping (torch's enable_gqa repeats each kv head Hq/Hkv
    times), default scale 1/sqrt(D).  q: [L, Hq, D], k/v: [L, Hkv, D]."""
    qt = torch.from_numpy(np.ascontiguousarray(q.transpose(1, 0, 2)))[None]
    kt = torch.from_numpy(np.ascontiguousarray(k.transpose(1, 0, 2)))[None]
    vt = torch.from_numpy(np.ascontiguousarray(v.transpose(1, 0, 2)))[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True,
                                                         enable_gqa=True)
    return o[0].numpy().transpose(1, 0, 2)


# --------------------------------------------------------------------------
# format and storage pins
# --------------------------------------------------------------------------


def test_la_bit_order_worked_example():
    """Section 4.1 enumeration, one tile at a time, against the mask."""
    g = _gold("la_bit_order.json")
    P, T = g["pages"], 2
    # one document of P pages followed by an empty query
    lay = O.Layout([0, P * T, P * T], [0, 2], T, 1)
    assert lay.la_bytes == len(g["cases"][0]["bytes"])
    for case in g["cases"]:
        i, j = case["tile"]
        la = np.array(case["bytes"], dtype=np.uint8)
        ca = np.zeros(lay.ca_bytes, dtype=np.uint8)
        assert O.read_bit(la, 0, O.la_bit_position(i, j)) == 1
        assert sum(O.read_bit(la, 0, b) for b in range(O.la_num_bits(P))) == 1
        m = O.mask_rows(lay, la, ca, 0, 0, np.arange(P * T))
        tile_m = m.reshape(P, T, P, T).any(axis=(1, 3))
        want = np.eye(P, dtype=bool)
        want[i, j] = True
        assert (tile_m == want).all(), (i, j)


def test_sizes_section_4_3():
    # "about 8 pages per document: 36 bits of LA and 8 bits of CA"
    assert O.la_num_bits(8) == 36 and O.ca_num_bits(8) == 8
    assert O.la_num_bytes(8) == 5 and O.ca_num_bytes(8) == 1
    assert O.num_pages(1024, 128) == 8 and O.num_pages(1025, 128) == 9
    for P in range(1, 200):
        assert O.la_num_bytes(P) == math.ceil(P * (P + 1) / 16)
        assert O.ca_num_bytes(P) == math.ceil(P / 8)
        assert O.la_num_bytes(P) * 8 >= O.la_num_bits(P) > (O.la_num_bytes(P) - 1) * 8


def _parse_size(s):
    val, unit = s.split()
    return float(val) * {"KB": 2 ** 10, "MB": 2 ** 20, "GB": 2 ** 30}[unit]


def _round_to_printed(x, printed):
    # agrees with the printed value to within one unit of its last digit
    # (the table rounds some cells and truncates others, e.g. 687.5 KB -> 687)
    val = printed.split()[0]
    dec = len(val.split(".")[1]) if "." in val else 0
    unit = _parse_size("1 " + printed.split()[1])
    return abs(x / unit - float(val)) < 10.0 ** -dec


def test_table1_storage():
    """Table 1 reproduces from 44 bits per (document, layer, query head)."""
    g = _gold("table1_storage.json")
    P = O.num_pages(g["doc_tokens"], g["tile"])
    bits_per_doc = O.la_num_bits(P) + O.ca_num_bits(P)
    assert bits_per_doc == 44
    for mdl in g["models"]:
        kv_tok = 2 * mdl["layers"] * mdl["kv_heads"] * mdl["head_dim"] * 2
        sift_doc = bits_per_doc * mdl["layers"] * mdl["q_heads"] / 8
        for ndocs, kv_s, sift_s in mdl["rows"]:
            assert _round_to_printed(ndocs * g["doc_tokens"] * kv_tok, kv_s), (mdl["name"], kv_s)
            assert _round_to_printed(ndocs * sift_doc, sift_s), (mdl["name"], sift_s)
        ratio = g["doc_tokens"] * kv_tok / sift_doc
        assert round(ratio) == mdl["reduction"], (mdl["name"], ratio)
        # with kv heads in place of query heads the ratio would not match
        wrong = g["doc_tokens"] * kv_tok / (bits_per_doc * mdl["layers"] * mdl["kv_heads"] / 8)
        assert round(wrong) != mdl["reduction"]


def test_wikiall_storage_byte_aligned():
    """Section 4.3's 101 GB follows from the byte-aligned vectors at T = 16."""
    g = _gold("wikiall_storage.json")
    P = O.num_pages(g["passage_tokens"], g["tile"])
    per = (O.la_num_bytes(P) + O.ca_num_bytes(P)) * g["layers"] * g["q_heads"]
    n = g["passages"] * g["fraction"]
    assert round(per * n / 2 ** 30) == g["sift_gb"]
    # "about 268 TB": 268.6 TiB
    assert abs(n * g["passage_tokens"] * g["kv_bytes_per_token"] / 2 ** 40 - g["kv_tb"]) < 1
    # without byte padding (44 bits) the figure would be 92 GB, not 101
    assert round((O.la_num_bits(P) + O.ca_num_bits(P)) / 8 * g["layers"] * g["q_heads"] * n / 2 ** 30) != g["sift_gb"]


def test_layout_offsets_and_tiles():
    # 2 prompts: [doc 100, doc 64, query 10] and [query 5]; T = 32, Hq = 3
    lay = O.Layout([0, 100, 164, 174, 179], [0, 3, 4], 32, 3)
    P = [s.pages for s in lay.segs]
    assert P == [4, 2, 1, 1]
    assert [s.tile_base for s in lay.segs] == [0, 4, 6, 7]
    assert lay.num_tiles == 8
    assert [s.la_offset for s in lay.segs[:2]] == [0, 3 * O.la_num_bytes(4)]
    assert lay.la_bytes == 3 * (O.la_num_bytes(4) + O.la_num_bytes(2))
    assert lay.ca_bytes == 3 * (O.ca_num_bytes(4) + O.ca_num_bytes(2))
    seg, i, a, n = lay.tile_span(3)
    assert (i, a, n) == (3, 96, 4)      # partial last tile of the first document
    seg, i, a, n = lay.tile_span(7)
    assert seg.prompt == 1 and (i, a, n) == (0, 174, 5)


# --------------------------------------------------------------------------
# worked example and special cases
# --------------------------------------------------------------------------


@pytest.mark.parametrize("clear_diagonal_bits", [False, True])
def test_uniform_weights_worked_example(clear_diagonal_bits):
    g = _gold("uniform_weights_example.json")
    L = g["layout"]
    lay = O.Layout(L["seg_offsets"], L["prompt_seg_ptr"], L["tile"], L["q_heads"])
    la = np.array(g["la"], dtype=np.uint8)
    if clear_diagonal_bits:
        # stored diagonal bits are ignored: clear bits (0,0) and (1,1) of both docs
        la = la & np.uint8(0b01011111)
    ca = np.array(g["ca"], dtype=np.uint8)
    n = lay.num_tokens
    q = np.zeros((n, 1, 1))
    k = np.zeros((n, 1, 1))
    v = np.array(g["v"], dtype=np.float64).reshape(n, 1, 1)
    out = O.attention(lay, q, k, v, la, ca)
    np.testing.assert_allclose(out[:, 0, 0], g["expected"], rtol=0, atol=1e-9)


def test_all_ones_is_dense_causal():
    """All-ones bitmaps give dense causal attention (full recompute)."""
    rng = np.random.default_rng(1)
    for trial in range(6):
        lay, la, ca, q, k, v = _random_case(rng, n_prompts=2, tile=8, hq=4, hkv=2, D=16,
                                             max_docs=3, max_len=30)
        la[:] = 0xFF
        ca[:] = 0xFF
        out = O.attention(lay, q, k, v, la, ca)
        for b in range(lay.num_prompts):
            p0, p1 = lay.prompt_span(b)
            if p1 == p0:
                continue
            ref = _sdpa_causal(q[p0:p1], k[p0:p1], v[p0:p1])
            np.testing.assert_allclose(out[p0:p1], ref, rtol=0, atol=1e-12)


def test_query_rows_are_dense_causal_whatever_the_bits():
    rng = np.random.default_rng(2)
    lay, la, ca, q, k, v = _random_case(rng, 1, 8, 2, 1, 8, max_docs=3, max_len=40, query_min=5)
    qs = lay.segs[-1]
    out = O.attention(lay, q, k, v, la, ca)
    ref = _sdpa_causal(q, k, v)
    sl = slice(qs.start, qs.start + qs.length)
    np.testing.assert_allclose(out[sl], ref[sl], rtol=0, atol=1e-12)


def test_no_bits_is_attention_within_the_diagonal_tile():
    """With every off-diagonal LA bit and every CA bit clear, a document row
    sees only the causal part of its own diagonal tile."""
    rng = np.random.default_rng(3)
    lay, la, ca, q, k, v = _random_case(rng, 2, 8, 2, 2, 8, max_docs=3, max_len=40)
    la[:] = 0
    ca[:] = 0
    out = O.attention(lay, q, k, v, la, ca)
    for s in lay.segs:
        if s.is_query:
            continue
        for i in range(s.pages):
            a = s.start + i * lay.tile
            z = min(a + lay.tile, s.start + s.length)
            ref = _sdpa_causal(q[a:z], k[a:z], v[a:z])
            np.testing.assert_allclose(out[a:z], ref, rtol=0, atol=1e-12)


def test_single_cross_bit_selects_one_whole_key_page():
    """One CA bit of document 0 exposes exactly that key page to every row of
    the later documents, and nothing else from document 0 (Section 3.4)."""
    T = 4
    # docs of 12, 8, 8 tokens and a 3-token query; one head
    lay = O.Layout([0, 12, 20, 28, 31], [0, 4], T, 1)
    la = np.zeros(lay.la_bytes, dtype=np.uint8)
    ca = np.zeros(lay.ca_bytes, dtype=np.uint8)
    ca[lay.segs[0].ca_offset] = 0b01000000          # page 1 of doc 0: tokens 4..7
    m = O.mask_rows(lay, la, ca, 0, 0, np.arange(lay.num_tokens))
    for r in range(12, 28):
        keys = set(np.nonzero(m[r])[0].tolist())
        own_tile = (r // T) * T
        assert keys == set(range(4, 8)) | set(range(own_tile, r + 1)), r
    # rows of doc 0 see only their diagonal tile
    for r in range(12):
        assert set(np.nonzero(m[r])[0].tolist()) == set(range((r // T) * T, r + 1))


def test_padding_bits_are_ignored():
    """Bits past the last tile of a vector change nothing."""
    rng = np.random.default_rng(4)
    lay, la, ca, q, k, v = _random_case(rng, 1, 8, 1, 1, 4, max_docs=3, max_len=60)
    la2, ca2 = la.copy(), ca.copy()
    for s in lay.segs:
        if s.is_query:
            continue
        nb = O.la_num_bits(s.pages)
        last = s.la_offset + O.la_num_bytes(s.pages) - 1
        if nb % 8:
            la2[last] ^= (0xFF >> (nb % 8))
        nb = O.ca_num_bits(s.pages)
        last = s.ca_offset + O.ca_num_bytes(s.pages) - 1
        if nb % 8:
            ca2[last] ^= (0xFF >> (nb % 8))
    a = O.mask_rows(lay, la, ca, 0, 0, np.arange(lay.num_tokens))
    b = O.mask_rows(lay, la2, ca2, 0, 0, np.arange(lay.num_tokens))
    assert (a == b).all()


# --------------------------------------------------------------------------
# brute force over the bit stream
# --------------------------------------------------------------------------


def _stream_mask(seg_offsets, prompt_seg_ptr, T, hq, la, ca, head):
    """Independent mask: walk each bit vector in storage order, consuming
    bits one at a time and assigning them to tiles in the order the paper
    enumerates them, then expand the tile grid to tokens with causality.
    Token-level, whole packed axis; cross-prompt cells stay 0."""
    L = seg_offsets[-1]
    M = np.zeros((L, L), dtype=bool)
    la_pos = 0
    ca_pos = 0

    def bits_of(buf, pos, nbytes):
        out = []
        for byte in buf[pos:pos + nbytes]:
            for sh in range(7, -1, -1):
                out.append((int(byte) >> sh) & 1)
        return out

    for b in range(len(prompt_seg_ptr) - 1):
        segs = list(range(prompt_seg_ptr[b], prompt_seg_ptr[b + 1]))
        docs = segs[:-1]
        qseg = segs[-1]
        ca_bits = {}
        la_tiles = {}
        for d in docs:
            Ld = seg_offsets[d + 1] - seg_offsets[d]
            P = -(-Ld // T)
            nla = -(-(P * (P + 1)) // 16)
            nca = -(-P // 8)
            # all heads of this document, heads in order
            for hh in range(hq):
                stream = iter(bits_of(la, la_pos, nla))
                grid = np.zeros((P, P), dtype=bool)
                for i in range(P):
                    for j in range(i + 1):
                        grid[i, j] = bool(next(stream))
                if hh == head:
                    la_tiles[d] = grid
                la_pos += nla
                cb = bits_of(ca, ca_pos, nca)[:P]
                if hh == head:
                    ca_bits[d] = cb
                ca_pos += nca
        for s in segs:
            for p in range(seg_offsets[s], seg_offsets[s + 1]):
                for k in range(seg_offsets[segs[0]], p + 1):
                    ks = next(x for x in segs if seg_offsets[x] <= k < seg_offsets[x + 1])
                    if s == qseg:
                        M[p, k] = True
                    elif ks == s:
                        i = (p - seg_offsets[s]) // T
                        j = (k - seg_offsets[s]) // T
                        M[p, k] = True if i == j else bool(la_tiles[s][i, j])
                    elif ks in docs:
                        M[p, k] = bool(ca_bits[ks][(k - seg_offsets[ks]) // T])
    return M


def test_mask_matches_bit_stream_brute_force():
    rng = np.random.default_rng(5)
    for trial in range(12):
        T = int(rng.choice([1, 2, 3, 4, 8]))
        hq = int(rng.choice([1, 2, 3]))
        lay, la, ca, *_ = _random_case(rng, int(rng.integers(1, 4)), T, hq, 1, 1,
                                       max_docs=4, max_len=14)
        for h in range(hq):
            bf = _stream_mask(lay.seg_offsets, lay.prompt_seg_ptr, T, hq, la, ca, h)
            for b in range(lay.num_prompts):
                p0, p1 = lay.prompt_span(b)
                if p1 == p0:
                    continue
                m = O.mask_rows(lay, la, ca, h, b, np.arange(p1 - p0))
                assert (m == bf[p0:p1, p0:p1]).all(), (trial, h, b)


# --------------------------------------------------------------------------
# invariants
# --------------------------------------------------------------------------


def test_rows_sum_to_one_and_vanish_outside_the_mask():
    rng = np.random.default_rng(6)
    lay, la, ca, q, k, v = _random_case(rng, 2, 8, 4, 2, 16, max_docs=3, max_len=50)
    for b in range(lay.num_prompts):
        p0, p1 = lay.prompt_span(b)
        if p1 == p0:
            continue
        rows = np.arange(p1 - p0)
        for h in range(4):
            P = O.probabilities(lay, q, k, la, ca, h, b, rows)
            msk = O.mask_rows(lay, la, ca, h, b, rows)
            np.testing.assert_allclose(P.sum(axis=1), 1.0, rtol=0, atol=1e-12)
            assert (P[~msk] == 0).all()
            assert (P[msk] > 0).all()


def test_unlisted_tile_does_not_matter():
    """NaN written into a key tile absent from an M-block's list leaves that
    M-block's output unchanged (and finite)."""
    rng = np.random.default_rng(7)
    lay, la, ca, q, k, v = _random_case(rng, 1, 8, 2, 1, 8, max_docs=4, max_len=60)
    base = O.attention(lay, q, k, v, la, ca)
    lists = O.tile_lists(lay, la, ca)
    checked = 0
    for (h, m), lst in lists.items():
        missing = [n for n in range(lay.num_tiles) if n not in lst and n < m]
        if not missing:
            continue
        n = missing[0]
        _, _, ka, kn = lay.tile_span(n)
        k2, v2 = k.copy(), v.copy()
        k2[ka:ka + kn] = np.nan
        v2[ka:ka + kn] = np.nan
        _, _, qa, qn = lay.tile_span(m)
        rows = np.arange(qa, qa + qn)
        ref = O.attention(lay, q, k, v, la, ca, heads=[h], rows=rows)
        out = O.attention(lay, q, k2, v2, la, ca, heads=[h], rows=rows)
        assert np.isfinite(out[:, h]).all()
        np.testing.assert_array_equal(out[:, h], ref[:, h])
        np.testing.assert_allclose(out[:, h], base[qa:qa + qn, h], rtol=0, atol=1e-12)
        checked += 1
        if checked >= 6:
            break
    assert checked > 0


def test_lists_last_row_equals_exhaustive():
    """The cheap list rule (last row of the M-block) equals OR over every row."""
    rng = np.random.default_rng(8)
    for trial in range(6):
        T = int(rng.choice([2, 4, 8]))
        lay, la, ca, *_ = _random_case(rng, 2, T, 2, 1, 1, max_docs=4, max_len=40)
        assert O.tile_lists(lay, la, ca) == O.tile_lists(lay, la, ca, exhaustive=True)


def test_list_lengths_closed_forms():
    rng = np.random.default_rng(9)
    lay, la, ca, *_ = _random_case(rng, 2, 4, 2, 1, 1, max_docs=4, max_len=30)
    # all bits set: every causal tile of the prompt is listed
    la[:] = 0xFF
    ca[:] = 0xFF
    for (h, m), lst in O.tile_lists(lay, la, ca).items():
        seg, i, _, _ = lay.tile_span(m)
        first = lay.prompt_segs(seg.prompt)[0].tile_base
        assert lst == list(range(first, m + 1))
    # no bits: documents list their diagonal only, the query lists all causal tiles
    la[:] = 0
    ca[:] = 0
    for (h, m), lst in O.tile_lists(lay, la, ca).items():
        seg, i, _, _ = lay.tile_span(m)
        first = lay.prompt_segs(seg.prompt)[0].tile_base
        assert lst == (list(range(first, m + 1)) if seg.is_query else [m])


def test_useful_flops_dense_closed_form():
    # one prompt: doc of 3 full tiles (T=4) and a query of 2 tokens; D = 8
    lay = O.Layout([0, 12, 14], [0, 2], 4, 1)
    la = np.full(lay.la_bytes, 0xFF, np.uint8)
    ca = np.full(lay.ca_bytes, 0xFF, np.uint8)
    lists = O.tile_lists(lay, la, ca)
    # dense causal cells: L(L+1)/2 with L = 14
    assert O.useful_flops(lay, lists, 8) == 4 * 8 * 14 * 15 // 2


def test_vectorised_bit_reader_equals_scalar_reader():
    """read_bits (used to build masks) gives read_bit's answer at every
    position, offsets included."""
    rng = np.random.default_rng(12)
    buf = rng.integers(0, 256, size=40, dtype=np.uint8)
    for off in (0, 3, 17):
        pos = np.arange((40 - off) * 8)
        want = [O.read_bit(buf, off, int(b)) for b in pos]
        assert O.read_bits(buf, off, pos).astype(int).tolist() == want
