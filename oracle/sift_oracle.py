"""Plain fp64 CPU oracle for SIFT's bitmap-driven sparse prefill attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module; only the tests, the smoke check and the benchmark's CPU-baseline leg do.
It shares no code with the HIP library: it reads the packed bit vectors with its
own bit reader, builds the token-level mask from the definition, and runs a
textbook masked softmax attention in float64 with numpy.

What the oracle computes (paper: SIFT, arXiv 2606.09441):

* A prompt is a list of RAG documents followed by the user query
  (Section 3.1, decomposition of the attention matrix).  Tokens of different
  prompts never see each other.
* Attention is causal.  Rows of the user query attend to every earlier token
  of their prompt (Section 3.1: the query sub-matrix is always recomputed;
  Section 5.1: query M-blocks count every causal N-block).
* Inside a document, key tile j of query-row tile i (j < i) is visible iff bit
  i(i+1)/2 + j of the document's local-attention (LA) vector is set
  (Section 4.1: T x T tiles of the lower triangle, enumerated row-major
  (0,0),(1,0),(1,1),(2,0),..., packed most-significant-bit first, each
  document's vector byte aligned).  Diagonal tiles (j == i) are always
  computed, whatever their stored bit says.
* Key page p of an earlier document e is visible to every row of a later
  document of the same prompt iff bit p of e's cross-attention (CA) vector is
  set (Section 4.2: one bit per KV page of width T, set = recomputed for future
  documents; Section 3.4: selection by whole key column).
* Sizes (Section 4.3): P = ceil(L/T) pages; LA = ceil(P(P+1)/16) bytes,
  CA = ceil(P/8) bytes, per (layer, head, document).
* Skipped tiles take part in neither numerator nor denominator: the result is
  the softmax over the marked locations only (Section 5.2: only the iteration
  over N-blocks changes; softmax and epilogue are those of dense attention).
* The decoded list of a (head, M-block) holds every N-block the mask touches,
  in ascending order (Section 5.1, sparse_n_indices).

Readings taken where the paper is silent: "head" means query head; the kv head of query head h is h // (Hq / Hkv); tiles are
segment local (a tile never straddles a document or the query, and the last
tile of a segment may be partial); CA bits are MSB first by page index; the
softmax scale is 1/sqrt(D); the bit-vector buffers concatenate, over prompts,
documents in prompt order and query heads 0..Hq-1, each document's vector; the
global number of tile i of segment s is the number of tiles in all earlier
segments (of all prompts) plus i; a document's rows see the CA-marked pages
of every earlier document of the prompt.

All inputs are taken at their exact values: bf16 or fp32 numbers are widened
to float64 without rounding.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# ----------------------------------------------------------------------------
# Bit-vector format (Sections 4.1-4.3)
# ----------------------------------------------------------------------------


def num_pages(length: int, tile: int) -> int:
    """P = ceil(L / T) (Section 4.3)."""
    return -(-int(length) // int(tile))


def la_num_bits(P: int) -> int:
    """Tiles in a P x P lower triangle, diagonal included (Section 4.1)."""
    return P * (P + 1) // 2


def ca_num_bits(P: int) -> int:
    """One bit per KV page (Section 4.2)."""
    return P


def la_num_bytes(P: int) -> int:
    """ceil(P(P+1) / (2*8)) bytes (Section 4.3)."""
    return -(-(P * (P + 1)) // 16)


def ca_num_bytes(P: int) -> int:
    """ceil(P / 8) bytes (Section 4.3)."""
    return -(-P // 8)


def la_bit_position(i: int, j: int) -> int:
    """Position of tile (row i, column j), j <= i, in the row-major lower
    triangle enumeration (0,0),(1,0),(1,1),(2,0),... (Section 4.1)."""
    assert 0 <= j <= i
    return i * (i + 1) // 2 + j


def read_bit(buf, byte_offset: int, b: int) -> int:
    """Bit b of the vector starting at byte_offset; the most significant bit
    of each byte comes first (Section 4.1)."""
    byte = int(buf[byte_offset + (b >> 3)])
    return (byte >> (7 - (b & 7))) & 1


def read_bits(buf, byte_offset: int, positions) -> np.ndarray:
    """read_bit at every position of an integer array (same rule, vectorised)."""
    b = np.asarray(positions, dtype=np.int64)
    byte = np.asarray(buf, dtype=np.uint8)[byte_offset + (b >> 3)].astype(np.int64)
    return ((byte >> (7 - (b & 7))) & 1).astype(bool)


# ----------------------------------------------------------------------------
# Prompt layout
# ----------------------------------------------------------------------------


@dataclass
class Segment:
    prompt: int
    is_query: bool
    start: int          # first token on the packed token axis
    length: int
    pages: int          # P = ceil(length / T)
    tile_base: int      # global number of the segment's tile 0
    la_offset: int      # byte offset of the LA vector of query head 0 (documents)
    ca_offset: int      # byte offset of the CA vector of query head 0 (documents)


class Layout:
    """Prompt b owns segments prompt_seg_ptr[b] .. prompt_seg_ptr[b+1]-1; the
    last of them is the user query, the others are its documents in order.
    Segment s covers tokens seg_offsets[s] .. seg_offsets[s+1]-1."""

    def __init__(self, seg_offsets, prompt_seg_ptr, tile: int, num_q_heads: int):
        self.seg_offsets = [int(x) for x in seg_offsets]
        self.prompt_seg_ptr = [int(x) for x in prompt_seg_ptr]
        self.tile = int(tile)
        self.hq = int(num_q_heads)
        self.segs: list[Segment] = []
        tile_base = la_off = ca_off = 0
        for b in range(len(self.prompt_seg_ptr) - 1):
            first, last = self.prompt_seg_ptr[b], self.prompt_seg_ptr[b + 1] - 1
            for s in range(first, last + 1):
                start = self.seg_offsets[s]
                length = self.seg_offsets[s + 1] - start
                P = num_pages(length, self.tile)
                self.segs.append(Segment(b, s == last, start, length, P,
                                         tile_base, la_off, ca_off))
                if s != last:
                    la_off += self.hq * la_num_bytes(P)
                    ca_off += self.hq * ca_num_bytes(P)
                tile_base += P
        self.num_tiles = tile_base
        self.la_bytes = la_off
        self.ca_bytes = ca_off
        self.num_prompts = len(self.prompt_seg_ptr) - 1
        self.num_tokens = self.seg_offsets[-1]

    def prompt_segs(self, b: int) -> list[Segment]:
        return [s for s in self.segs if s.prompt == b]

    def prompt_span(self, b: int) -> tuple[int, int]:
        ps = self.prompt_segs(b)
        return ps[0].start, ps[-1].start + ps[-1].length

    def tile_span(self, m: int) -> tuple[Segment, int, int, int]:
        """(segment, local tile i, first token, token count) of global tile m."""
        for s in self.segs:
            if s.tile_base <= m < s.tile_base + s.pages:
                i = m - s.tile_base
                a = s.start + i * self.tile
                return s, i, a, min(self.tile, s.start + s.length - a)
        raise IndexError(m)


# ----------------------------------------------------------------------------
# The mask (Sections 3.1, 4.1, 4.2)
# ----------------------------------------------------------------------------


def _page_bits(buf, off: int, n: int) -> np.ndarray:
    return read_bits(buf, off, np.arange(n))


def _tile_row(lay: Layout, la, ca, head: int, b: int, seg_index: int, i: int,
              cache: dict | None = None) -> np.ndarray:
    """Key visibility for every row of tile i of segment seg_index (prompt b),
    before the causal cut: one bool per token of the prompt.  `cache` may
    hold the part that depends only on (head, prompt, segment): the keys of
    earlier documents."""
    ps = lay.prompt_segs(b)
    p0, p1 = lay.prompt_span(b)
    me = ps[seg_index]
    key = (head, b, seg_index)
    if cache is not None and key in cache:
        row = cache[key].copy()
    else:
        row = np.zeros(p1 - p0, dtype=bool)
        for si, se in enumerate(ps[:seg_index]):
            a = se.start - p0
            if me.is_query:
                # the user query recomputes everything before it (Section 3.1)
                row[a:a + se.length] = True
            else:
                # cross attention: page p of an earlier document (Section 4.2)
                off = se.ca_offset + head * ca_num_bytes(se.pages)
                bits = _page_bits(ca, off, se.pages)
                row[a:a + se.length] = np.repeat(bits, lay.tile)[:se.length]
        if cache is not None:
            cache[key] = row.copy()
    a = me.start - p0
    if me.is_query:
        row[a:a + me.length] = True
    else:
        # local attention: tiles j <= i of the same document (Section 4.1)
        off = me.la_offset + head * la_num_bytes(me.pages)
        bits = read_bits(la, off, la_bit_position(i, 0) + np.arange(i + 1))
        bits[i] = True                      # the diagonal tile, whatever its bit
        lo, hi = a, a + min((i + 1) * lay.tile, me.length)
        row[lo:hi] = np.repeat(bits, lay.tile)[:hi - lo]
    return row


def mask_rows(lay: Layout, la, ca, head: int, b: int, rows, cache: dict | None = None) -> np.ndarray:
    """allowed[r, k] for the prompt-relative query tokens `rows` of prompt b
    against every key token of that prompt, for query head `head`."""
    ps = lay.prompt_segs(b)
    p0, p1 = lay.prompt_span(b)
    keys = np.arange(p1 - p0)
    rows = np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(rows), p1 - p0), dtype=bool)
    cache_rows: dict[tuple[int, int], np.ndarray] = {}
    for r, p in enumerate(rows):
        si = next(k for k, s in enumerate(ps) if s.start - p0 <= p < s.start - p0 + s.length)
        i = (p - (ps[si].start - p0)) // lay.tile
        if (si, i) not in cache_rows:
            cache_rows[(si, i)] = _tile_row(lay, la, ca, head, b, si, int(i), cache)
        out[r] = cache_rows[(si, i)] & (keys <= p)
    return out


# ----------------------------------------------------------------------------
# Attention (Section 5.2: dense attention restricted to the marked tiles)
# ----------------------------------------------------------------------------


def _kv_head(h: int, hq: int, hkv: int) -> int:
    return h // (hq // hkv)


def masked_softmax_rows(s: np.ndarray, allowed: np.ndarray) -> np.ndarray:
    """Row softmax of s over the allowed entries only; 0 elsewhere."""
    s = np.where(allowed, s, -np.inf)
    mx = s.max(axis=1, keepdims=True)
    e = np.exp(s - mx)
    e = np.where(allowed, e, 0.0)
    return e / e.sum(axis=1, keepdims=True)


def _probs_and_mask(lay: Layout, q, k, la, ca, head: int, b: int, rows, scale):
    hkv = k.shape[1]
    D = q.shape[2]
    scale = 1.0 / np.sqrt(D) if scale is None else float(scale)
    p0, p1 = lay.prompt_span(b)
    rows = np.asarray(rows, dtype=np.int64)
    g = _kv_head(head, lay.hq, hkv)
    qr = np.asarray(q[p0 + rows, head, :], dtype=np.float64)
    kk = np.asarray(k[p0:p1, g, :], dtype=np.float64)
    allowed = mask_rows(lay, la, ca, head, b, rows)
    s = (qr @ kk.T) * scale
    return masked_softmax_rows(s, allowed), allowed


def probabilities(lay: Layout, q, k, la, ca, head: int, b: int, rows, scale=None) -> np.ndarray:
    """P[r, key] of query head `head` for prompt-relative `rows` of prompt b."""
    return _probs_and_mask(lay, q, k, la, ca, head, b, rows, scale)[0]


def _weighted_rows(P: np.ndarray, allowed: np.ndarray, vv: np.ndarray) -> np.ndarray:
    """O[r] = sum over the allowed keys of P[r, key] * V[key].  Keys outside
    the mask are never read, so their V may hold anything, NaN included."""
    out = np.empty((P.shape[0], vv.shape[1]), dtype=np.float64)
    for r in range(P.shape[0]):
        idx = np.nonzero(allowed[r])[0]
        out[r] = P[r, idx] @ vv[idx]
    return out


def _row_groups(lay: Layout, rows: np.ndarray):
    """Split global token rows into groups of one prompt and one query tile
    (M-block): yields (prompt b, positions into `rows`, prompt-relative rows)."""
    tile_of = np.empty(len(rows), dtype=np.int64)
    prompt_of = np.empty(len(rows), dtype=np.int64)
    for s in lay.segs:
        sel = (rows >= s.start) & (rows < s.start + s.length)
        tile_of[sel] = s.tile_base + (rows[sel] - s.start) // lay.tile
        prompt_of[sel] = s.prompt
    order = np.argsort(tile_of, kind="stable")
    bounds = np.nonzero(np.diff(tile_of[order]))[0] + 1
    for grp in np.split(order, bounds):
        if grp.size:
            b = int(prompt_of[grp[0]])
            yield b, grp, rows[grp] - lay.prompt_span(b)[0]


def _attend_group(lay: Layout, q, kk, vv, la, ca, head: int, b: int, rel_rows, scale,
                  cache: dict) -> np.ndarray:
    """Output rows of one group (rows of one M-block of prompt b) for one query
    head.  kk, vv: the prompt's K and V rows of the head's kv head, float64.
    Scores are formed for the keys some row of the group may see (the union of
    the rows' masks); every other key has probability 0 for all of them."""
    p0, _ = lay.prompt_span(b)
    allowed = mask_rows(lay, la, ca, head, b, rel_rows, cache)
    keys = np.nonzero(allowed.any(axis=0))[0]
    if keys.size and keys[-1] - keys[0] + 1 == keys.size:
        ksel = slice(int(keys[0]), int(keys[-1]) + 1)      # a contiguous range: no copy
    else:
        ksel = keys
    qr = np.asarray(q[p0 + rel_rows, head, :], dtype=np.float64)
    s = (qr @ kk[ksel].T) * scale
    am = allowed[:, ksel]
    P = masked_softmax_rows(s, am)
    vs = vv[ksel]
    if np.isfinite(vs).all():
        return P @ vs                      # P is 0 outside each row's mask
    return _weighted_rows(P, am, vs)       # non-finite V: read the allowed keys only


def attention(lay: Layout, q, k, v, la, ca, scale=None, heads=None, rows=None,
              workers: int = 1) -> np.ndarray:
    """O[t, h, :] in float64.

    q: [L, Hq, D]; k, v: [L, Hkv, D]; la, ca: uint8 buffers.  With `rows`
    (global token indices) only those rows are computed and the result is
    [len(rows), Hq, D]; with `heads` only those heads are filled.  Rows are
    handled in groups that share a query tile, one (head, prompt) at a time;
    `workers` threads take (head, prompt) pairs in parallel."""
    L, hq, D = q.shape
    hkv = k.shape[1]
    heads = list(range(hq)) if heads is None else list(heads)
    sc = 1.0 / np.sqrt(D) if scale is None else float(scale)
    want = np.arange(L, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(want), hq, D), dtype=np.float64)
    groups: dict[int, list] = {}
    for b, pos, rel in _row_groups(lay, want):
        groups.setdefault(b, []).append((pos, rel))
    kv_cache: dict = {}

    def kv(b, g):
        if (b, g) not in kv_cache:
            p0, p1 = lay.prompt_span(b)
            kv_cache[(b, g)] = (np.asarray(k[p0:p1, g, :], dtype=np.float64),
                                np.asarray(v[p0:p1, g, :], dtype=np.float64))
        return kv_cache[(b, g)]

    # the float64 K/V copies are made up front, once per (prompt, kv head)
    for b in groups:
        for h in heads:
            kv(b, _kv_head(h, hq, hkv))

    def job(h, b, part):
        kk, vv = kv(b, _kv_head(h, hq, hkv))
        cache: dict = {}
        for pos, rel in part:
            out[pos, h, :] = _attend_group(lay, q, kk, vv, la, ca, h, b, rel, sc, cache)

    # jobs: (head, prompt, a run of consecutive row groups)
    per_job = 1 if workers <= 1 else 8
    jobs = [(h, b, grp[i:i + per_job] if workers > 1 else grp)
            for h in heads for b, grp in groups.items()
            for i in (range(0, len(grp), per_job) if workers > 1 else [0])]
    if workers <= 1 or len(jobs) <= 1:
        for h, b, part in jobs:
            job(h, b, part)
    else:
        # one BLAS thread per worker: the workers are the parallelism
        from concurrent.futures import ThreadPoolExecutor
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1, user_api="blas"):
            with ThreadPoolExecutor(max_workers=workers) as ex:
                for f in [ex.submit(job, *jb) for jb in jobs]:
                    f.result()
    return out


# ----------------------------------------------------------------------------
# Expected decoded lists (Section 5.1), read off the mask
# ----------------------------------------------------------------------------


def _prompt_key_tiles(lay: Layout, b: int) -> tuple[np.ndarray, np.ndarray]:
    """(prompt-relative first token, global tile number) of the prompt's tiles."""
    p0, _ = lay.prompt_span(b)
    starts, ids = [], []
    for s in lay.prompt_segs(b):
        for i in range(s.pages):
            starts.append(s.start - p0 + i * lay.tile)
            ids.append(s.tile_base + i)
    return np.asarray(starts, dtype=np.int64), np.asarray(ids, dtype=np.int64)


def _key_tile_any(lay: Layout, b: int, keyrow: np.ndarray, tiles=None) -> list[int]:
    """Global tile numbers of the prompt's key tiles that hold a True.
    `tiles` may pass _prompt_key_tiles(lay, b) computed once."""
    starts, ids = _prompt_key_tiles(lay, b) if tiles is None else tiles
    if starts.size == 0:
        return []
    hit = np.logical_or.reduceat(keyrow, starts)
    return ids[hit].tolist()


def tile_lists(lay: Layout, la, ca, heads=None, mblocks=None, exhaustive: bool = False):
    """Expected sparse_n_indices.

    Returns {(h, m): ascending list of global key tiles n such that block
    (M-block m, N-block n) of head h's mask holds a 1}.  With exhaustive=True
    every row of the M-block is materialised and OR-ed; otherwise only the
    block's last row is, which gives the same answer because inside one
    (M-block, N-block) pair the mask is the same for every row except for the
    causal cut, which only admits more keys on later rows."""
    heads = range(lay.hq) if heads is None else heads
    mblocks = range(lay.num_tiles) if mblocks is None else mblocks
    res = {}
    cache: dict = {}
    tiles: dict = {}
    for m in mblocks:
        seg, i, a, n = lay.tile_span(m)
        b = seg.prompt
        if b not in tiles:
            tiles[b] = _prompt_key_tiles(lay, b)
        p0, _ = lay.prompt_span(b)
        rows = np.arange(a - p0, a - p0 + n) if exhaustive else np.array([a - p0 + n - 1])
        for h in heads:
            msk = mask_rows(lay, la, ca, h, b, rows, cache).any(axis=0)
            res[(h, m)] = _key_tile_any(lay, b, msk, tiles[b])
    return res


def csr_lists(lay: Layout, la, ca, exhaustive: bool = False):
    """The lists in packed form: row_ptr[Hq*M+1] (row h*M + m) and col_idx."""
    lists = tile_lists(lay, la, ca, exhaustive=exhaustive)
    M = lay.num_tiles
    row_ptr = np.zeros(lay.hq * M + 1, dtype=np.int64)
    cols = []
    for h in range(lay.hq):
        for m in range(M):
            lst = lists[(h, m)]
            row_ptr[h * M + m + 1] = row_ptr[h * M + m] + len(lst)
            cols.extend(lst)
    return row_ptr, np.asarray(cols, dtype=np.int64)


def useful_flops(lay: Layout, lists: dict, head_dim: int) -> int:
    """4*D per computed (query, key) cell of the listed tiles: causal cells of
    the tiles, within segment lengths (QK^T and PV, one multiply-add each)."""
    total = 0
    for (h, m), lst in lists.items():
        _, _, qa, qn = lay.tile_span(m)
        for n in lst:
            _, _, ka, kn = lay.tile_span(n)
            if n == m:
                total += qn * (qn + 1) // 2
            else:
                total += qn * kn
    return 4 * head_dim * total
