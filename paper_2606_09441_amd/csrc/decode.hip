// Bit-vector decoding (SIFT, Section 5.1): turn the local-attention (LA) and
// cross-attention (CA) bit vectors of every (document, query head) into one
// packed, ascending int32 list of key tiles per (query head, M-block).
//
// Three kernels:
//   decode_count  one workgroup per (query head, segment): each row's number
//                 of listed tiles.  Document rows: popcount of LA bits
//                 i(i+1)/2 .. i(i+1)/2+i-1 (row i of the lower triangle,
//                 diagonal excluded) + 1 for the always-computed diagonal +
//                 the popcount of the CA vectors of the earlier documents of
//                 the prompt (one sum per workgroup).  Query rows: every
//                 tile of the prompt up to the row's own (Section 5.1: query
//                 M-blocks count all causal N-blocks), in closed form.  The
//                 counts are scanned inside the (head, segment); the last
//                 workgroup scans the (head, segment) totals: the "designated
//                 offsets" of Section 5.1 are their sum.
//   decode_write  one wavefront per attention list unit (query head, up to
//                 eight consecutive M-blocks of one segment): writes its
//                 rows' row_ptr, then the CA pages of the earlier documents
//                 in document order, then the LA tiles (diagonals included);
//                 each chunk of 64 candidate tiles becomes indices through a
//                 ballot and a lane-prefix popcount, so every output is dense
//                 and in ascending global tile order.  It writes every row's
//                 list and the unit's merged step list (the union of the
//                 rows' lists, each step flagged with the M-blocks that list
//                 it), which the attention kernel streams.
//   schedule_scatter  the launch order of the attention's work units.
// Bits are most significant first inside each byte (Section 4.1).

#include "sift_internal.h"

namespace sift {
namespace {

__device__ __forceinline__ int la_nbytes(int P) { return (P * (P + 1) + 15) >> 4; }
__device__ __forceinline__ int ca_nbytes(int P) { return (P + 7) >> 3; }

__device__ __forceinline__ int get_bit(const uint8_t* v, int b) {
  return (v[b >> 3] >> (7 - (b & 7))) & 1;
}

// Set bits among bits b0 .. b0+n-1 of v (MSB-first numbering).  The bytes
// are read four at a time, their loads issued together.
__device__ int popc_bits(const uint8_t* v, int b0, int n) {
  if (n <= 0) return 0;
  const int end = b0 + n;
  const int last = (end - 1) >> 3;
  int c = 0;
  for (int w = b0 >> 3; w <= last; w += 4) {
    unsigned byte[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) byte[q] = w + q <= last ? v[w + q] : 0u;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int lo = (w + q) * 8;  // bit number of the byte's most significant bit
      const int a = max(b0 - lo, 0), z = min(end - lo, 8);
      const unsigned m = a < z ? (0xFFu >> a) & (0xFFu << (8 - z)) : 0u;
      c += __popc(byte[q] & m);
    }
  }
  return c;
}

// Inclusive scan of v over the 256 threads of a block (wavefront scans,
// then the four wavefront totals through LDS); returns the block total.
__device__ __forceinline__ int32_t block_scan256(int32_t v, int32_t& incl, int32_t* wtot) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  int32_t x = v;
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) wtot[w] = x;
  __syncthreads();
  int32_t before = 0, total = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    before += j < w ? wtot[j] : 0;
    total += wtot[j];
  }
  __syncthreads();  // wtot is reused by the next call
  incl = before + x;
  return total;
}

// Inclusive scan of v over the 1024 threads of a block (wavefront scans,
// then the 16 wavefront totals through LDS); returns the block total.
__device__ __forceinline__ int32_t block_scan1024(int32_t v, int32_t& incl, int32_t* wtot) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  int32_t x = v;
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) wtot[w] = x;
  __syncthreads();
  int32_t before = 0, total = 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    before += j < w ? wtot[j] : 0;
    total += wtot[j];
  }
  __syncthreads();
  incl = before + x;
  return total;
}

constexpr int kCountSegs = 1024;  // segments the per-head count pass holds in LDS

// Block h: every row of query head h (layouts of at most kCountSegs
// segments).  A document row i lists the marked pages of the earlier
// documents of its prompt, the marked tiles j < i of its LA row and its
// diagonal; a query row lists every tile of its prompt up to its own
// (Section 5.1).  First each document's CA popcount for head h, then, per
// prompt, what each of its segments' rows see of the earlier documents
// (in LDS, and to seg_cross); then the rows, scanned in tile order: local[]
// gets each row's offset inside head h, head_tot[h] the head's total.  The
// write pass adds the totals of the heads before h.
// The CA-marked tiles of a prompt, in tile order, also go to the head's
// cross list (from the prompt's first tile on: there are fewer marked tiles
// than tiles): the earlier documents' part of a document row's list is a
// prefix of it, which the write pass copies instead of walking every page.
__global__ __launch_bounds__(1024) void decode_count_head(PlanTables pt, WorkTables wt,
                                                          const uint8_t* __restrict__ la,
                                                          const uint8_t* __restrict__ ca,
                                                          int32_t* __restrict__ local,
                                                          KvPages pages) {
  __shared__ int32_t cross[kCountSegs];  // CA popcount, then the pages a row of s sees
  __shared__ int32_t first[kCountSegs];  // first segment of the prompt
  __shared__ int32_t sgt[5][kCountSegs];  // first tile, pages, kind, LA and CA offsets
  __shared__ int32_t wtot[16];
  const int S = pt.num_segments;
  const int M = pt.num_tiles;
  const int h = blockIdx.x;
  const int t = threadIdx.x;
  constexpr int kQ = 4;  // rows t + 1024 q of a group, their loads issued together
  int sq[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) sq[q] = t + 1024 * q < M ? pt.tile_seg[t + 1024 * q] : 0;
  for (int s = t; s < S; s += 1024) {
    const int P = pt.seg_pages[s];
    const int kind = pt.seg_kind[s];
    const int caoff = pt.seg_ca_off[s];
    first[s] = pt.seg_first[s];
    sgt[0][s] = pt.seg_tile0[s];
    sgt[1][s] = P;
    sgt[2][s] = kind;
    sgt[3][s] = pt.seg_la_off[s];
    sgt[4][s] = caoff;
    cross[s] = kind == kQuery
                   ? 0
                   : popc_bits(ca + caoff + static_cast<int64_t>(h) * ca_nbytes(P), 0, P);
  }
  __syncthreads();
  // per prompt, in segment order: each segment's rows see the pages its
  // earlier documents mark (a query's rows are counted in closed form)
  for (int s = t; s < S; s += 1024) {
    if (first[s] != s) continue;  // one thread per prompt
    int32_t run = 0;
    for (int e = s; e < S && first[e] == s; ++e) {
      const int32_t v = cross[e];
      cross[e] = run;
      wt.seg_cross[h * S + e] = run;
      run += v;
    }
  }
  __syncthreads();
  int32_t* lrow = local + static_cast<int64_t>(h) * M;
  int32_t run = 0;
  for (int g0 = 0; g0 < M; g0 += 1024 * kQ) {
    if (g0 > 0) {
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        const int m = g0 + 1024 * q + t;
        sq[q] = m < M ? pt.tile_seg[m] : 0;
      }
    }
    int32_t cnt[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const int m = g0 + 1024 * q + t;
      cnt[q] = 0;
      if (m < M) {
        const int s = sq[q];
        const int i = m - sgt[0][s];
        if (sgt[2][s] == kQuery) {
          cnt[q] = m - sgt[0][first[s]] + 1;
        } else {
          const int P = sgt[1][s];
          const uint8_t* lav = la + sgt[3][s] + static_cast<int64_t>(h) * la_nbytes(P);
          const uint8_t* cav = ca + sgt[4][s] + static_cast<int64_t>(h) * ca_nbytes(P);
          const int32_t before = popc_bits(cav, 0, i);  // marked pages of s before i
          cnt[q] = cross[s] + 1 + popc_bits(lav, i * (i + 1) / 2, i);
          if (get_bit(cav, i)) {
            const int64_t y = static_cast<int64_t>(h) * M + sgt[0][first[s]] + cross[s] + before;
            wt.cross_col[y] = m;
            wt.cross_rows[y] = make_int2(kv_row0(pt, pages, m), pt.tile_len[m]);
          }
        }
      }
    }
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      if (g0 + 1024 * q >= M) break;  // uniform
      int32_t incl;
      const int32_t chunk = block_scan1024(cnt[q], incl, wtot);
      if (g0 + 1024 * q + t < M) lrow[g0 + 1024 * q + t] = run + incl - cnt[q];
      run += chunk;
    }
  }
  if (t == 0) wt.head_tot[h] = run;
}

// Block b = h S + s: the rows of segment s for query head h.  A document row
// i lists the marked pages of the earlier documents of its prompt, the
// marked tiles j < i of its LA row and its diagonal; a query row lists every
// tile of its prompt up to its own (Section 5.1).  Each row's count goes to
// local[] as its offset inside the (head, segment); the total to seg_base[b].
// The last block to finish turns seg_base into each (head, segment)'s first
// list entry (the rows' order is h-major, then tile order) and writes
// row_ptr[Hq M] = nnz.
__global__ __launch_bounds__(256) void decode_count(PlanTables pt, WorkTables wt,
                                                    const uint8_t* __restrict__ la,
                                                    const uint8_t* __restrict__ ca,
                                                    int32_t* __restrict__ local,
                                                    int32_t* __restrict__ row_ptr) {
  __shared__ int32_t wtot[4];
  __shared__ int last;
  const int S = pt.num_segments;
  const int b = blockIdx.x;
  const int h = b / S, s = b - h * S;
  const int t = threadIdx.x;
  const int P = pt.seg_pages[s];
  const int tile0 = pt.seg_tile0[s];
  int32_t* lrow = local + static_cast<int64_t>(h) * pt.num_tiles + tile0;
  uint8_t* mrow = wt.ca_mark + static_cast<int64_t>(h) * pt.num_tiles + tile0;
  int32_t total;
  if (pt.seg_kind[s] == kQuery) {
    // row i lists a + i tiles, a = the tiles before the segment plus one
    const int a = tile0 - pt.seg_tile0[pt.seg_first[s]] + 1;
    for (int i = t; i < P; i += 256) {
      lrow[i] = i * a + i * (i - 1) / 2;
      mrow[i] = 0;
    }
    total = P * a + P * (P - 1) / 2;
  } else {
    // marked pages of the earlier documents (the same for every row) and
    // the LA bits of each row before its diagonal: all loads issued first
    const uint8_t* lav = la + pt.seg_la_off[s] + static_cast<int64_t>(h) * la_nbytes(P);
    const uint8_t* cav = ca + pt.seg_ca_off[s] + static_cast<int64_t>(h) * ca_nbytes(P);
    for (int i = t; i < P; i += 256) mrow[i] = static_cast<uint8_t>(get_bit(cav, i));
    int32_t c = 0;
    for (int e = pt.seg_first[s] + t; e < s; e += 256) {
      const int Pe = pt.seg_pages[e];
      c += popc_bits(ca + pt.seg_ca_off[e] + static_cast<int64_t>(h) * ca_nbytes(Pe), 0, Pe);
    }
    int32_t own = t < P ? 1 + popc_bits(lav, t * (t + 1) / 2, t) : 0;  // rows 0..255
    // one pass: the CA sum and the scan of the first 256 rows together
    int32_t incl, cincl;
    const int32_t first = block_scan256(own, incl, wtot);
    const int32_t cross = block_scan256(c, cincl, wtot);
    if (t < P) lrow[t] = incl - own + t * cross;
    int32_t run = first;
    for (int i0 = 256; i0 < P; i0 += 256) {  // longer documents: more rows
      const int i = i0 + t;
      const int32_t cnt = i < P ? 1 + popc_bits(lav, i * (i + 1) / 2, i) : 0;
      const int32_t chunk = block_scan256(cnt, incl, wtot);
      if (i < P) lrow[i] = run + incl - cnt + i * cross;
      run += chunk;
    }
    total = run + P * cross;
  }
  if (t == 0) {
    wt.seg_base[b] = total;
    __threadfence();
    last = atomicAdd(wt.decode_done, 1) == static_cast<int>(gridDim.x) - 1;
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  // thread t takes the consecutive totals [t per, (t + 1) per): a serial
  // sum, one block scan of the thread sums, then each thread's offsets
  const int n = gridDim.x;
  const int per = (n + 255) / 256;
  const int a = min(n, t * per), z = min(n, a + per);
  auto load8 = [&](int i0, int32_t (&v)[8]) {  // eight loads issued together
#pragma unroll
    for (int q = 0; q < 8; ++q)
      v[q] = i0 + q < z ? __hip_atomic_load(&wt.seg_base[i0 + q], __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT)
                        : 0;
  };
  int32_t sum = 0;
  for (int i0 = a; i0 < z; i0 += 8) {
    int32_t v[8];
    load8(i0, v);
#pragma unroll
    for (int q = 0; q < 8; ++q) sum += v[q];
  }
  int32_t incl;
  const int32_t all = block_scan256(sum, incl, wtot);
  int32_t run = incl - sum;
  for (int i0 = a; i0 < z; i0 += 8) {
    int32_t v[8];
    load8(i0, v);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (i0 + q < z) wt.seg_base[i0 + q] = run;
      run += v[q];
    }
  }
  if (t == 0) {
    row_ptr[static_cast<int64_t>(pt.num_q_heads) * pt.num_tiles] = all;
    *wt.decode_done = 0;
  }
}

// Wave-cooperative emitter of one unit's outputs.  Each call handles up to 64
// candidate key tiles n (one per lane); bit k of `listed` says M-block m0 + k
// lists n.  Tiles are appended, in lane order, to the lists of the M-blocks
// that list them, and to the merged step list: at T >= 64 one or two steps
// per tile (tile_steps); at T < 64 one step per group of G = 64 / T
// consecutive tiles of a segment that any M-block lists (emit_grouped).
// kNb: most M-blocks of a list unit (128 / T, at least 2); kHalves: T = 128
// (a tile is one or two 64-key steps).
template <int kNb, bool kHalves>
struct Emitter {
  int32_t* col;
  int2* steps;
  const PlanTables* pt;
  const WorkTables* wt;
  int32_t base;  // the list unit's first step
  int32_t w0;    // its first work unit
  bool whole;    // not split: the first steps go to w0's record here
  KvPages pages;
  int32_t pos[kNb];  // next write position in each M-block's list
  int32_t ps;                   // next write position in the step list
  int32_t m0, nb;
  unsigned hrows;  // T = 128: kernel blocks of the M-block (tile_steps_at)
  unsigned long long below;
  int32_t gt, grun;  // copy_gathered: entries done, first entry of the current run
  int32_t nw, plen;  // the unit's pieces and their length (emit_grouped)

  // A step's place among the first steps of its piece (read by the attention
  // kernel's prologue from the work record).
  __device__ __forceinline__ void note_first(int32_t idx, int2 st) {
    const int32_t rel = idx - base;
    if (whole) {
      if (rel < kFirstSteps) wt->rec[w0].first[rel] = st;
    } else {
      const int32_t k = rel / plen, j = rel - k * plen;
      if (j < kFirstSteps && k < nw) wt->rec[w0 + k].first[j] = st;
    }
  }

  __device__ __forceinline__ void lists(unsigned listed, int32_t n) {
#pragma unroll
    for (int k = 0; k < kNb; ++k) {
      if (k >= nb) break;
      const bool on = (listed >> k) & 1u;
      const unsigned long long mk = __ballot(on);
      if (on) col[pos[k] + __popcll(mk & below)] = n;
      pos[k] += __popcll(mk);
    }
  }

  // The same with the tile's first K/V row and length already loaded.
  __device__ __forceinline__ void emit_at(unsigned listed, int32_t n, int32_t row0, int32_t len) {
    lists(listed, n);
    if constexpr (!kHalves) {
      // T = 64: one step per listed tile, in lane order
      const unsigned long long mu = __ballot(listed != 0u);
      if (listed != 0u) {
        const unsigned diag = (n >= m0 && n < m0 + nb) ? 1u << (n - m0) : 0u;
        const int info = len | static_cast<int>(listed << kStepListedShift) |
                         static_cast<int>(diag << kStepDiagShift);
        const int32_t idx = ps + __popcll(mu & below);
        const int2 st = make_int2(row0, info);
        steps[idx] = st;
        if (whole && idx - base < kFirstSteps) wt->rec[w0].first[idx - base] = st;
      }
      ps += __popcll(mu);
      return;
    }
    // one or two steps per listed tile, in lane order
    const TileSteps ts = tile_steps_at(*pt, n, listed, m0, nb, row0, len, hrows);
    const unsigned long long mu1 = __ballot(ts.cnt >= 1), mu2 = __ballot(ts.cnt >= 2);
    const int32_t idx = ps + __popcll(mu1 & below) + __popcll(mu2 & below);
    for (int q = 0; q < ts.cnt; ++q) {
      steps[idx + q] = ts.s[q];
      if (whole && idx + q - base < kFirstSteps) wt->rec[w0].first[idx + q - base] = ts.s[q];
    }
    ps += __popcll(mu1) + __popcll(mu2);
  }

  // One round of a document unit's earlier-document part, copied from the
  // head's cross list: the first cnt lanes hold a CA-marked tile (id c,
  // {first row, length} r), listed by every M-block; at T = 64 one step
  // each, at T = 128 one per 64 keys.
  __device__ __forceinline__ void copy_round(int32_t c, int2 r, int32_t cnt, int lane) {
    const bool valid = lane < cnt;
    const unsigned lst = kHalves ? hrows : (1u << nb) - 1u;
    const int info_or = static_cast<int>(lst << kStepListedShift);
#pragma unroll
    for (int k = 0; k < kNb; ++k) {
      if (k >= nb) break;
      if (valid) col[pos[k] + lane] = c;
      pos[k] += cnt;
    }
    if constexpr (!kHalves) {
      if (valid) {
        const int2 st = make_int2(r.x, r.y | info_or);
        steps[ps + lane] = st;
        if (whole && ps + lane - base < kFirstSteps) wt->rec[w0].first[ps + lane - base] = st;
      }
      ps += cnt;
    } else {
      const bool two = valid && r.y > 64;
      const unsigned long long m2 = __ballot(two);
      const int32_t idx = ps + lane + __popcll(m2 & below);
      if (valid) {
        const int2 s0 = make_int2(r.x, min(r.y, 64) | info_or);
        steps[idx] = s0;
        if (whole && idx - base < kFirstSteps) wt->rec[w0].first[idx - base] = s0;
        if (two) {
          const int2 s1 = make_int2(r.x + 64, (r.y - 64) | info_or);
          steps[idx + 1] = s1;
          if (whole && idx + 1 - base < kFirstSteps) wt->rec[w0].first[idx + 1 - base] = s1;
        }
      }
      ps += cnt + __popcll(m2);
    }
  }

  // T < 64: one round of a document unit's earlier-document part from the
  // head's cross list (n entries; the first cnt lanes hold entries gt ..,
  // tile id c, {first row, length} r), listed by every M-block.  A step
  // gathers G such tiles, adjacent or not, each wavefront of the kernel
  // reading its rows from its own tile (kvb); a partial tile (the last of
  // its document) ends its step, so that only a step's last tile is short.
  // Entry t starts a step when (t - first entry of its run) % G == 0, runs
  // ending after partial tiles.
  __device__ __forceinline__ void copy_gathered(int32_t c, int2 r, int32_t cnt, int32_t n,
                                                int lane) {
    const int T = pt->tile, G = pt->group;
    const bool valid = lane < cnt;
#pragma unroll
    for (int k = 0; k < kNb; ++k) {
      if (k >= nb) break;
      if (valid) col[pos[k] + lane] = c;
      pos[k] += cnt;
    }
    const bool part = valid && r.y < T;
    const unsigned long long pm = __ballot(part);
    const unsigned long long pb = pm & below;
    const int t = gt + lane;
    const int run = pb != 0ull ? gt + (63 - __clzll(pb)) + 1 : grun;
    const int q = (t - run) & (G - 1);
    const unsigned long long sm = __ballot(valid && q == 0);
    const int32_t idx = ps + __popcll(sm & (below | (1ull << lane))) - 1;
    const int32_t kv = r.x - q * T;
    int* kw = reinterpret_cast<int*>(wt->kvb);
    if (valid) kw[4 * static_cast<int64_t>(idx) + q] = kv;
    if (valid && (part || q == G - 1 || t == n - 1)) {
      // the step's last tile: the step's record, and its unused kvb words
      const unsigned lst = (2u << ((nb - 1) / G)) - 1u;
      unsigned sub = 0u;
      for (int k = 0; k < nb; ++k) sub |= ((2u << q) - 1u) << (G * k);
      const int2 st = make_int2(static_cast<int>(sub),
                                (q * T + r.y) | static_cast<int>(lst << kStepListedShift));
      steps[idx] = st;
      for (int x = q + 1; x < 4; ++x) kw[4 * static_cast<int64_t>(idx) + x] = kv;
      if (whole && idx - base < kFirstSteps) wt->rec[w0].first[idx - base] = st;
    }
    ps += __popcll(sm);
    if (pm != 0ull) grun = gt + (63 - __clzll(pm)) + 1;
    gt += cnt;
  }

  // T < 64.  The lanes hold tiles local = c0 + lane of one segment of P
  // tiles (c0 a multiple of 64, so a group never straddles two calls).  The
  // group's first lane gathers its members' bits and writes the step: the
  // group's first key row and key count, per kernel block (G M-blocks) the
  // OR of the listed bits and whether the group is the block's diagonal, and
  // the sub-tile mask.
  __device__ __forceinline__ void emit_grouped(unsigned listed, int32_t n, int32_t local, int32_t P,
                                               int lane) {
    lists(listed, n);
    const int G = pt->group;
    unsigned gl[4];
    gl[0] = listed;
#pragma unroll
    for (int q = 1; q < 4; ++q) {
      const unsigned x = __shfl_down(listed, q, 64);
      gl[q] = (q < G && lane + q < 64) ? x : 0u;
    }
    unsigned any = 0u;
#pragma unroll
    for (int q = 0; q < 4; ++q) any |= gl[q];
    const bool emits = (local & (G - 1)) == 0 && local < P && any != 0u;
    const unsigned long long mu = __ballot(emits);
    if (emits) {
      const int cnt = min(G, P - local);
      const int len = (cnt - 1) * pt->tile + pt->tile_len[n + cnt - 1];
      unsigned lst = 0u, sm = 0u;
      for (int k = 0; k < nb; ++k)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if ((gl[q] >> k) & 1u) {
            lst |= 1u << (k / G);
            sm |= 1u << (G * k + q);
          }
      unsigned diag = 0u;
#pragma unroll
      for (int b = 0; b < kUnitBlocks; ++b)
        if (n == m0 + G * b) diag |= 1u << b;
      const int32_t idx = ps + __popcll(mu & below);
      const int32_t row0 = kv_row0(*pt, pages, n);
      const int2 st = make_int2(static_cast<int>(sm), len | static_cast<int>(lst << kStepListedShift) |
                                                      static_cast<int>(diag << kStepDiagShift));
      steps[idx] = st;
      note_first(idx, st);
      // the group's tiles are adjacent in the packed K/V; a page pool places
      // each on its own
      int4 kb = make_int4(row0, row0, row0, row0);
      if (pages.table != nullptr) {
        const int T = pt->tile;
        if (cnt > 1) kb.y = kv_row0(*pt, pages, n + 1) - T;
        if (cnt > 2) kb.z = kv_row0(*pt, pages, n + 2) - 2 * T;
        if (cnt > 3) kb.w = kv_row0(*pt, pages, n + 3) - 3 * T;
      }
      wt->kvb[idx] = kb;
    }
    ps += __popcll(mu);
  }
};

// kNb: the most M-blocks of a list unit (2 at T >= 64, 4 at T = 32, 8 at
// T = 16); kGrouped: T < 64 (steps are groups of tiles); kHalves: T = 128.
// Separate instances keep the T = 64 one free of the other sizes' work.
template <int kNb, bool kGrouped, bool kHalves>
__global__ __launch_bounds__(256) void decode_write(PlanTables pt, WorkTables wt,
                                                    const uint8_t* __restrict__ la,
                                                    const uint8_t* __restrict__ ca,
                                                    const int32_t* __restrict__ local,
                                                    int32_t* __restrict__ row_ptr,
                                                    int32_t* __restrict__ col, KvPages pages) {
  const int lane = threadIdx.x & 63;
  const int slot = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  if (slot >= wt.num_urec) return;  // uniform per wavefront
  const UnitRec ur = wt.urec[slot];
  const int h = ur.head, m0 = ur.m0, nb = ur.nb, s = ur.seg;
  const int M = pt.num_tiles;
  const unsigned all = (1u << nb) - 1u;
  const int64_t r0 = static_cast<int64_t>(h) * M + m0;
  const int mlast = m0 + nb - 1;
  // Every load that depends on the record alone is issued before any result
  // is used: the rows' offsets, the first rounds of the candidate walk and
  // of the cross-list copy, then the heads' totals.
  int32_t loc[kNb];
#pragma unroll
  for (int k = 0; k < kNb; ++k) loc[k] = k < nb ? local[r0 + k] : 0;
  //   T >= 64: the candidates are the prompt's tiles lo .. mlast in order
  //   (the earlier documents' pages, then this segment's tiles), 64 per
  //   round.  Query unit: M-block m0 + k lists n when n <= m0 + k (Section
  //   5.1).  Document unit: every M-block lists the CA-marked pages of the
  //   earlier documents (copied from the head's cross list when the count
  //   pass built it), and row r = i + k its LA-marked tiles j < r and j == r.
  //   Rounds go in chunks: a chunk's loads are all issued before any of
  //   their results is used (raw bytes kept, bits taken later), so a chunk
  //   waits on memory once.
  constexpr int kChunk = 4, kCopy = 4;
  const bool query = (ur.flags & kUnitQuery) != 0;
  const int lo = ur.lo, sd0 = ur.sd0, i = m0 - sd0;
  const uint8_t* lav = query ? la : la + ur.la_off + static_cast<int64_t>(h) * la_nbytes(ur.pages);
  const uint8_t* mark = wt.ca_mark + static_cast<int64_t>(h) * M;
  const int2* rowlen = reinterpret_cast<const int2*>(pt.tile_info);  // {first row, length} at 2 n
  const bool copy = !query && wt.cross_col != nullptr;
  const int64_t ybase = static_cast<int64_t>(h) * M + lo;
  const int start = copy ? sd0 : lo;
  int32_t ncross = 0;
  int32_t yc[kCopy];
  int2 yr[kCopy];
  int2 tl[kChunk];
  unsigned raw[kChunk][2];  // CA mark, or the LA bytes of rows i and i + 1
  auto load_copy = [&](int t0) {
#pragma unroll
    for (int q = 0; q < kCopy; ++q) {
      const int t = min(t0 + 64 * q + lane, M - 1 - lo);  // inside the head's list
      yc[q] = wt.cross_col[ybase + t];
      yr[q] = wt.cross_rows[ybase + t];
    }
  };
  auto load_walk = [&](int c0) {
    const int nr = min(kChunk, (mlast - c0) / 64 + 1);
#pragma unroll
    for (int c = 0; c < kChunk; ++c) {
      if (c >= nr) break;
      const int n = min(c0 + 64 * c + lane, mlast);
      tl[c] = rowlen[2 * n];
      if (pages.table != nullptr) tl[c].x = pages.table[n];
      raw[c][0] = raw[c][1] = 0u;
      if (!query) {
        // every address valid: lav is the document's own LA vector
        const int j = n - sd0;
        const int b0 = i * (i + 1) / 2 + j, b1 = (i + 1) * (i + 2) / 2 + j;
        const uint8_t* a0 = n < sd0 ? mark + n : (j < i ? lav + (b0 >> 3) : lav);
        const uint8_t* a1 = (n >= sd0 && nb > 1 && j < i + 1) ? lav + (b1 >> 3) : lav;
        raw[c][0] = *a0;
        raw[c][1] = *a1;
      }
    }
  };
  if (copy) {
    ncross = wt.seg_cross[h * pt.num_segments + s];
    load_copy(0);
  }
  if constexpr (!kGrouped) load_walk(start);
  Emitter<kNb, kHalves> e;
  e.col = col;
  e.steps = wt.steps;
  e.pt = &pt;
  e.wt = &wt;
  e.pages = pages;
  e.base = ur.step_off;
  e.ps = e.base + ur.part_skip;
  const int32_t nw = ur.nwork, plen = ur.plen;  // pieces
  e.w0 = ur.work0;
  e.whole = nw == 1;
  e.nw = nw;
  e.plen = plen;
  e.m0 = m0;
  e.nb = nb;
  e.hrows = static_cast<unsigned>((ur.flags >> 1) & 3);
  e.below = (1ull << lane) - 1ull;
  e.gt = e.grun = 0;
  int32_t base;
  if (wt.head_tot != nullptr) {
    // local[] holds offsets inside the head: add the totals of heads 0 .. h-1
    int32_t before = 0, nnz = 0;
    for (int j0 = 0; j0 < pt.num_q_heads; j0 += 64) {
      const int j = j0 + lane;
      const int32_t v = j < pt.num_q_heads ? wt.head_tot[j] : 0;
      before += j < h ? v : 0;
      nnz += v;
    }
    for (int off = 32; off > 0; off >>= 1) {
      before += __shfl_xor(before, off, 64);
      nnz += __shfl_xor(nnz, off, 64);
    }
    base = before;
    if (slot == 0 && lane == 0) row_ptr[static_cast<int64_t>(pt.num_q_heads) * M] = nnz;
  } else {
    base = wt.seg_base[h * pt.num_segments + s];
  }
  // a part of a query unit starts after the earlier segments' tiles, which
  // every M-block lists
  const int32_t skip = kGrouped && query ? pt.seg_tile0[ur.part_d0] - lo : 0;
  const bool first_part = (ur.flags & kUnitFirstPart) != 0;
#pragma unroll
  for (int k = 0; k < kNb; ++k) {
    e.pos[k] = k < nb ? base + loc[k] : 0;
    if (k < nb && lane == 0 && first_part) row_ptr[r0 + k] = e.pos[k];
    e.pos[k] += skip;
  }
  if constexpr (!kGrouped) {
    for (int t0 = 0; t0 < ncross;) {
#pragma unroll
      for (int q = 0; q < kCopy; ++q) {
        if (t0 + 64 * q >= ncross) break;
        e.copy_round(yc[q], yr[q], min(64, ncross - t0 - 64 * q), lane);
      }
      t0 += 64 * kCopy;
      if (t0 < ncross) load_copy(t0);
    }
    for (int c0 = start;;) {
      const int nr = min(kChunk, (mlast - c0) / 64 + 1);
#pragma unroll
      for (int c = 0; c < kChunk; ++c) {
        if (c >= nr) break;
        const int n = c0 + 64 * c + lane;
        unsigned listed = 0u;
        if (n <= mlast) {
          if (query) {
            listed = n < m0 ? all : (all & ~((1u << (n - m0)) - 1u));
          } else if (n < sd0) {
            listed = raw[c][0] != 0u ? all : 0u;
          } else {
            const int j = n - sd0;
#pragma unroll
            for (int k = 0; k < 2; ++k) {
              const int r = i + k;
              if (k < nb && j < r) listed |= ((raw[c][k] >> (7 - ((r * (r + 1) / 2 + j) & 7))) & 1u) << k;
            }
            if (j >= i && j < i + nb) listed |= 1u << (j - i);  // the diagonal tile
          }
        }
        int32_t row0 = tl[c].x;
        if (pages.table != nullptr)
          row0 = (row0 < 0 ? 0 : (row0 >= pages.num_pages ? pages.num_pages - 1 : row0)) * pt.tile;
        e.emit_at(listed, n, row0, tl[c].y);
      }
      c0 += 64 * kChunk;
      if (c0 > mlast) break;
      load_walk(c0);
    }
  } else if (query) {
    // the same, segment by segment so that tile groups stay within one call
    // (this record's segments of the prompt)
    for (int d = ur.part_d0; d < ur.part_d1; ++d) {
      const int last = d < s ? pt.seg_pages[d] - 1 : mlast - pt.seg_tile0[s];
      for (int c0 = 0; c0 <= last; c0 += 64) {
        const int j = c0 + lane;
        const int n = pt.seg_tile0[d] + j;
        unsigned listed = 0u;
        if (j <= last) listed = n < m0 ? all : (all & ~((1u << (n - m0)) - 1u));
        e.emit_grouped(listed, n, j, last + 1, lane);
      }
    }
  } else {
    // T < 64, a document unit.  CA pages of every earlier document: the
    // same for all M-blocks; gathered G to a step from the cross list when
    // the count pass built it
    if (copy) {
      for (int t0 = 0; t0 < ncross;) {
#pragma unroll
        for (int q = 0; q < kCopy; ++q) {
          if (t0 + 64 * q >= ncross) break;
          e.copy_gathered(yc[q], yr[q], min(64, ncross - t0 - 64 * q), ncross, lane);
        }
        t0 += 64 * kCopy;
        if (t0 < ncross) load_copy(t0);
      }
    } else {
      for (int d = pt.seg_first[s]; d < s; ++d) {
        const int Pe = pt.seg_pages[d];
        const uint8_t* cav = ca + pt.seg_ca_off[d] + static_cast<int64_t>(h) * ca_nbytes(Pe);
        for (int c0 = 0; c0 < Pe; c0 += 64) {
          const int b = c0 + lane;
          const bool on = b < Pe && get_bit(cav, b);
          e.emit_grouped(on ? all : 0u, pt.seg_tile0[d] + b, b, Pe, lane);
        }
      }
    }
    // LA rows i .. i+nb-1 of the document's triangle, tiles j = 0 .. i+nb-1;
    // row r lists j < r when its bit is set, and its diagonal j == r
    const int i = m0 - pt.seg_tile0[s];
    const int P = pt.seg_pages[s];
    const uint8_t* lav = la + pt.seg_la_off[s] + static_cast<int64_t>(h) * la_nbytes(P);
    for (int c0 = 0; c0 < i + nb; c0 += 64) {
      const int j = c0 + lane;
      unsigned listed = 0u;
#pragma unroll
      for (int k = 0; k < kNb; ++k) {
        const int r = i + k;
        if (k < nb && j <= r && (j == r || get_bit(lav, r * (r + 1) / 2 + j))) listed |= 1u << k;
      }
      e.emit_grouped(listed, pt.seg_tile0[s] + j, j, P, lane);
    }
  }
  const int32_t cnt = e.ps - e.base;
  if (!kGrouped && !e.whole) {
    // the first steps of every piece, read back from the finished list (the
    // workgroup-scope fence waits for this wavefront's stores, which its
    // CU's loads then see)
    __threadfence_block();
    for (int q = lane; q < nw * kFirstSteps; q += 64) {
      const int32_t k = q / kFirstSteps, j = q - k * kFirstSteps;
      if (k * plen + j < cnt) wt.rec[e.w0 + k].first[j] = wt.steps[e.base + k * plen + j];
    }
  }
  if (ur.flags & kUnitLastPart) write_work_counts(wt, e.w0, nw, plen, cnt, lane, 64);
}

// Generic merge of caller-given lists (one thread per unit): the union of
// the unit's rows, ascending, entries outside [first tile of the prompt,
// M-block] skipped, at most lu_off[u+1] - lu_off[u] steps.
__global__ __launch_bounds__(256) void merge_steps(PlanTables pt, WorkTables wt,
                                                   const int32_t* __restrict__ row_ptr,
                                                   const int32_t* __restrict__ col,
                                                   int64_t cap) {
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= wt.num_units) return;
  const int h = wt.lu_head[u];
  const int m0 = wt.lu_m0[u];
  const int nb = wt.lu_nb[u];
  const int lo = pt.tile_lo[m0];
  const int G = pt.group;
  const int64_t r0 = static_cast<int64_t>(h) * pt.num_tiles + m0;
  auto clampi = [cap](int64_t x) { return min(cap, max(static_cast<int64_t>(0), x)); };
  int64_t it[kMaxListBlocks], end[kMaxListBlocks];
#pragma unroll
  for (int k = 0; k < kMaxListBlocks; ++k) {
    it[k] = 0;
    end[k] = 0;
    if (k < nb) {
      it[k] = clampi(row_ptr[r0 + k]);
      end[k] = max(it[k], clampi(row_ptr[r0 + k + 1]));
    }
  }
  const int base = wt.lu_off[u];
  const int room = wt.lu_off[u + 1] - base;
  int ns = 0;
  int pw = wt.lu_work0[u];        // work unit of the next step
  int pj = 0;                     // its place in that piece
  const int plen = wt.lu_len[u];  // piece length
  auto put = [&](int2 st, uint32_t sm) {
    if (G > 1) {
      wt.kvb[base + ns] = make_int4(st.x, st.x, st.x, st.x);  // adjacent tiles
      st.x = static_cast<int>(sm);
    }
    wt.steps[base + ns] = st;
    if (pj < kFirstSteps) wt.rec[pw].first[pj] = st;
    if (++pj == plen) {  // the next step opens the next piece
      pj = 0;
      ++pw;
    }
    ++ns;
  };
  // T < 64: the group being gathered (first tile g0, its segment's tile
  // count P, the listed bits of each member)
  int g0 = -1, gP = 0;
  unsigned gl[4] = {0u, 0u, 0u, 0u};
  auto flush = [&]() {
    if (g0 < 0 || ns >= room) return;
    const int cnt = min(G, gP - (g0 - pt.seg_tile0[pt.tile_seg[g0]]));
    const int len = (cnt - 1) * pt.tile + pt.tile_len[g0 + cnt - 1];
    unsigned lst = 0u, sm = 0u;
    for (int k = 0; k < nb; ++k)
      for (int q = 0; q < G; ++q)
        if ((gl[q] >> k) & 1u) {
          lst |= 1u << (k / G);
          sm |= 1u << (G * k + q);
        }
    unsigned diag = 0u;
    for (int b = 0; b < kUnitBlocks; ++b)
      if (g0 == m0 + G * b) diag |= 1u << b;
    put(make_int2(pt.tile_tok0[g0], len | static_cast<int>(lst << kStepListedShift) |
                                        static_cast<int>(diag << kStepDiagShift)),
        sm);
    g0 = -1;
    gl[0] = gl[1] = gl[2] = gl[3] = 0u;
  };
  while (true) {
    int head[kMaxListBlocks];
    int n = 0x7fffffff;
#pragma unroll
    for (int k = 0; k < kMaxListBlocks; ++k) {
      head[k] = 0x7fffffff;
      if (k >= nb) continue;
      while (it[k] < end[k]) {
        const int x = col[it[k]];
        if (x >= lo && x <= m0 + k) {
          head[k] = x;
          break;
        }
        ++it[k];
      }
      n = min(n, head[k]);
    }
    if (n == 0x7fffffff) break;
    unsigned listed = 0u;
#pragma unroll
    for (int k = 0; k < kMaxListBlocks; ++k)
      if (k < nb && head[k] == n) {
        listed |= 1u << k;
        ++it[k];
      }
    if (G == 1) {
      const TileSteps ts = tile_steps(pt, KvPages{nullptr, 0}, n, listed, m0, nb);
      if (ns + ts.cnt > room) break;
      for (int q = 0; q < ts.cnt; ++q) put(ts.s[q], 0u);
    } else {
      const int sg = pt.tile_seg[n];
      const int local = n - pt.seg_tile0[sg];
      const int lead = n - (local & (G - 1));
      if (lead != g0) {
        flush();
        if (ns >= room) break;
        g0 = lead;
        gP = pt.seg_pages[sg];
      }
      gl[local & (G - 1)] |= listed;
    }
  }
  if (G > 1 && ns < room) flush();
  write_work_counts(wt, wt.lu_work0[u], wt.lu_nwork[u], plen, ns, 0, 1);
}

// Schedule pass, blocks x sched_blocks .. for chunk x: each scans the
// chunk's bucket sizes (one bucket per thread) into offsets, then copies its
// share of the chunk's work units to launch[x + kNumXcd * k], k = the offset
// of the unit's bucket plus its rank in the bucket.  The chunk's last block
// to finish clears its buckets for the next decode.
__global__ __launch_bounds__(1024) void schedule_scatter(WorkTables wt) {
  __shared__ int32_t off[kSchedBuckets];
  __shared__ int32_t wsum[16];
  __shared__ int last;
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int nbk = wt.sched_blocks;
  const int x = blockIdx.x / nbk;
  const int part = blockIdx.x - x * nbk;
  int32_t* hist = wt.hist + x * kSchedBuckets;
  const int32_t own = hist[t];
  int32_t s = own;  // inclusive scan inside the wavefront
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t y = __shfl_up(s, o, 64);
    if (lane >= o) s += y;
  }
  if (lane == 63) wsum[wave] = s;
  __syncthreads();
  int32_t e = s - own;
  for (int j = 0; j < wave; ++j) e += wsum[j];
  off[t] = e;
  __syncthreads();
  const int32_t c0 = x * wt.chunk_size;
  const int32_t c1 = min(wt.num_work, c0 + wt.chunk_size);
  const int32_t per = (wt.chunk_size + nbk - 1) / nbk;
  const int32_t w_end = min(c1, c0 + (part + 1) * per);
  for (int32_t w = c0 + part * per + t; w < w_end; w += 1024) {
    const int4* src = reinterpret_cast<const int4*>(wt.rec + w);
    int4 r[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = src[q];
    // the step count is word 9 of the record (int4 2, .y), the rank word 2
    const int32_t k = off[sched_bucket(r[2].y)] + r[0].z;
    if (k >= 0 && k < wt.chunk_size) {
      int4* dst = reinterpret_cast<int4*>(wt.launch + x + kNumXcd * k);
#pragma unroll
      for (int q = 0; q < 4; ++q) dst[q] = r[q];
    }
  }
  // every block of the chunk has read the buckets once the last one is here
  if (t == 0) last = atomicAdd(&wt.sched_done[x], 1) == nbk - 1;
  __syncthreads();
  if (last) {
    hist[t] = 0;
    if (t == 0) wt.sched_done[x] = 0;
  }
}

hipError_t launch_schedule(const WorkTables& wt, hipStream_t stream) {
  if (wt.num_work == 0) return hipSuccess;
  static_assert(kSchedBuckets == 1024, "one bucket per thread of the schedule pass");
  hipLaunchKernelGGL(schedule_scatter, dim3(kNumXcd * wt.sched_blocks), dim3(1024), 0, stream,
                     wt);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const PlanTables& pt, const WorkTables& wt, const uint8_t* la,
                         const uint8_t* ca, int32_t* counts, int32_t* row_ptr, int32_t* col_idx,
                         const KvPages& pages, hipStream_t stream) {
  hipError_t e;
  WorkTables w2 = wt;
  if (pt.num_segments <= kCountSegs && wt.num_units > 0) {
    // one count block per head; the write pass adds the heads' totals and
    // writes row_ptr[Hq M]
    hipLaunchKernelGGL(decode_count_head, dim3(static_cast<unsigned>(pt.num_q_heads)), dim3(1024),
                       0, stream, pt, wt, la, ca, counts, pages);
  } else {
    // one count block per (head, segment); the last one scans the totals
    // and writes row_ptr[Hq M].  No cross lists: the write pass walks every
    // page.
    w2.head_tot = nullptr;
    w2.cross_col = nullptr;
    const int64_t blocks = static_cast<int64_t>(pt.num_q_heads) * pt.num_segments;
    hipLaunchKernelGGL(decode_count, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, pt,
                       wt, la, ca, counts, row_ptr);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (wt.num_units == 0) return hipSuccess;
  const dim3 wgrid(static_cast<unsigned>((wt.num_urec + 3) / 4));
  if (pt.group == 4)
    hipLaunchKernelGGL((decode_write<8, true, false>), wgrid, dim3(256), 0, stream, pt, w2, la, ca,
                       counts, row_ptr, col_idx, pages);
  else if (pt.group == 2)
    hipLaunchKernelGGL((decode_write<4, true, false>), wgrid, dim3(256), 0, stream, pt, w2, la, ca,
                       counts, row_ptr, col_idx, pages);
  else if (pt.halves == 2)
    hipLaunchKernelGGL((decode_write<2, false, true>), wgrid, dim3(256), 0, stream, pt, w2, la, ca,
                       counts, row_ptr, col_idx, pages);
  else
    hipLaunchKernelGGL((decode_write<2, false, false>), wgrid, dim3(256), 0, stream, pt, w2, la, ca,
                       counts, row_ptr, col_idx, pages);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_schedule(w2, stream);
}

hipError_t launch_merge_steps(const PlanTables& pt, const WorkTables& wt, const int32_t* row_ptr,
                              const int32_t* col_idx, int64_t col_capacity, hipStream_t stream) {
  if (wt.num_units == 0) return hipSuccess;
  hipLaunchKernelGGL(merge_steps, dim3(static_cast<unsigned>((wt.num_units + 255) / 256)),
                     dim3(256), 0, stream, pt, wt, row_ptr, col_idx, col_capacity);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_schedule(wt, stream);
}

}  // namespace sift
