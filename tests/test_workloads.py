"""The seeded input generator: determinism, shapes, bf16 exactness, and that
its bit vectors have the sizes and contents the oracle's reader expects."""

import hashlib

import numpy as np
import pytest

import workloads as W
from oracle import sift_oracle as O


def _digest(wl):
    h = hashlib.sha256()
    for a in (wl.seg_offsets, wl.prompt_seg_ptr, wl.q, wl.k, wl.v, wl.la, wl.ca):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def test_bf16_round_ties_to_even_and_exactness():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 3.0e38], np.float32)
    r = W.bf16_round(x)
    # 1 + 2^-8 is halfway between bf16 neighbours 1 and 1 + 2^-7: ties to even -> 1
    assert r[1] == 1.0
    assert r[2] == np.float32(1.0 + 2 ** -6)   # 1 + 3*2^-8 halfway -> even mantissa
    assert r[3] == 1.0
    assert r[4] == -2.5
    assert (r.view(np.uint32) & 0xFFFF == 0).all()
    # matches torch's RNE conversion
    import torch
    t = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(r, t)


def test_tiny_shapes_and_determinism():
    a = W.make("tiny")
    b = W.make("tiny")
    assert _digest(a) == _digest(b)
    assert a.tokens == 288 and a.q.shape == (288, 2, 64) and a.k.shape == (288, 1, 64)
    assert list(a.seg_offsets) == [0, 128, 256, 288]
    lay = O.Layout(a.seg_offsets, a.prompt_seg_ptr, a.tile, a.hq)
    assert lay.la_bytes == a.la.size and lay.ca_bytes == a.ca.size
    assert _digest(W.make("tiny", seed=1)) != _digest(a)


def test_pack_msb_matches_oracle_reader():
    rng = np.random.default_rng(0)
    bits = (rng.random(37) < 0.5).astype(np.uint8)
    buf = W.pack_msb(bits)
    assert buf.size == 5
    assert [O.read_bit(buf, 0, i) for i in range(37)] == bits.tolist()


def test_llama_bitmaps_diagonal_and_density():
    wl = W.make("llama8b_4k")
    lay = O.Layout(wl.seg_offsets, wl.prompt_seg_ptr, wl.tile, wl.hq)
    assert wl.tokens == 4224 and lay.num_tiles == 66
    assert wl.la.size == lay.la_bytes and wl.ca.size == lay.ca_bytes
    assert (wl.q.view(np.uint32) & 0xFFFF == 0).all()
    for s in lay.segs[:-1]:
        P = s.pages
        for h in range(wl.hq):
            off = s.la_offset + h * O.la_num_bytes(P)
            bits = [O.read_bit(wl.la, off, b) for b in range(O.la_num_bits(P))]
            for i in range(P):
                assert bits[O.la_bit_position(i, i)] == 1
            # top ceil(0.2 * 36) = 8 tiles, OR the 8 diagonals
            assert 8 <= sum(bits) <= 16
            coff = s.ca_offset + h * O.ca_num_bytes(P)
            assert sum(O.read_bit(wl.ca, coff, b) for b in range(P)) == 2   # ceil(0.2*8)


def test_all_ones_sets_every_bit():
    wl = W.all_ones(W.make("tiny"))
    lay = O.Layout(wl.seg_offsets, wl.prompt_seg_ptr, wl.tile, wl.hq)
    for s in lay.segs[:-1]:
        for h in range(wl.hq):
            off = s.la_offset + h * O.la_num_bytes(s.pages)
            assert all(O.read_bit(wl.la, off, b) for b in range(O.la_num_bits(s.pages)))


def test_custom_layout():
    wl = W.custom([[70, 33, 10], [5], [64, 0]], tile=16, hq=4, hkv=2, d=64, dtype="bf16", seed=3)
    assert list(wl.seg_offsets) == [0, 70, 103, 113, 118, 182, 182]
    assert list(wl.prompt_seg_ptr) == [0, 3, 4, 6]
    lay = O.Layout(wl.seg_offsets, wl.prompt_seg_ptr, 16, 4)
    assert wl.la.size == lay.la_bytes and wl.ca.size == lay.ca_bytes


@pytest.mark.slow
def test_ragged_layout():
    wl = W.make("ragged_x8")
    assert len(wl.prompt_seg_ptr) == 9
    for b in range(8):
        nd = wl.prompt_seg_ptr[b + 1] - wl.prompt_seg_ptr[b] - 1
        assert 4 <= nd <= 12
    lens = np.diff(wl.seg_offsets)
    lay = O.Layout(wl.seg_offsets, wl.prompt_seg_ptr, wl.tile, wl.hq)
    assert wl.la.size == lay.la_bytes
    for s in lay.segs:
        if not s.is_query:
            assert s.length % 64 == 0 and 256 <= s.length <= 2048
        else:
            assert 64 <= s.length <= 512


@pytest.mark.parametrize("tile", [16, 32, 64, 128])
def test_scramble_changes_only_ignored_bits(tile):
    """The scrambler clears stored diagonal bits of every other vector and
    sets every padding bit; the oracle, which ignores both (Sections 4.1,
    4.3), gives the same lists and outputs on the scrambled bits."""
    wl = W.custom([[300, 64, 129, 75], [5], [1, 64, 0], [200, 131, 70]], tile=tile, hq=4, hkv=2,
                  d=16, dtype="f32", seed=tile, p_la=0.4, p_ca=0.3)
    ws = W.scramble_ignored_bits(wl, seed=1)
    assert ws.la.shape == wl.la.shape and ws.ca.shape == wl.ca.shape
    lay = O.Layout(wl.seg_offsets, wl.prompt_seg_ptr, wl.tile, wl.hq)
    # walk the vectors: count cleared diagonals and set padding bits
    cleared = padded = 0
    for s in lay.segs:
        if s.is_query:
            continue
        P = s.pages
        for h in range(wl.hq):
            off = s.la_offset + h * O.la_num_bytes(P)
            bits = np.unpackbits(ws.la[off:off + O.la_num_bytes(P)], bitorder="big")
            diag = [O.la_bit_position(i, i) for i in range(P)]
            cleared += int((bits[diag] == 0).all())
            assert (bits[P * (P + 1) // 2:] == 1).all()
            padded += bits.size - P * (P + 1) // 2
            coff = s.ca_offset + h * O.ca_num_bytes(P)
            cb = np.unpackbits(ws.ca[coff:coff + O.ca_num_bytes(P)], bitorder="big")
            assert (cb[P:] == 1).all()
            padded += cb.size - P
    assert cleared > 0 and padded > 0
    assert O.tile_lists(lay, ws.la, ws.ca) == O.tile_lists(lay, wl.la, wl.ca)
    a = O.attention(lay, wl.q, wl.k, wl.v, wl.la, wl.ca)
    b = O.attention(lay, ws.q, ws.k, ws.v, ws.la, ws.ca)
    np.testing.assert_array_equal(a, b)
