// Bit-vector decoding (SIFT, Section 5.1): turn the local-attention (LA) and
// cross-attention (CA) bit vectors of every (document, query head) into one
// packed, ascending int32 list of key tiles per (query head, M-block).
//
// Three kernels:
//   decode_count  one thread per row (h, m): number of tiles the row lists.
//                 Document rows: popcount of LA bits i(i+1)/2 .. i(i+1)/2+i-1
//                 (row i of the lower triangle, diagonal excluded) + 1 for the
//                 always-computed diagonal + popcount of the CA vector of
//                 every earlier document of the prompt.  Query rows: every
//                 tile of the prompt up to the row's own (Section 5.1: query
//                 M-blocks count all causal N-blocks).
//   decode_scan   exclusive prefix sum of the counts -> row_ptr (one block).
//   decode_write  one wavefront per row: CA pages of the earlier documents in
//                 document order, then LA tiles j < i, then the diagonal;
//                 each chunk of 64 bits is turned into indices with a ballot
//                 and a lane-prefix popcount, so the output is dense and in
//                 ascending global tile order.
// Bits are most significant first inside each byte (Section 4.1).

#include "sift_internal.h"

namespace sift {
namespace {

__device__ __forceinline__ int la_nbytes(int P) { return (P * (P + 1) + 15) >> 4; }
__device__ __forceinline__ int ca_nbytes(int P) { return (P + 7) >> 3; }

__device__ __forceinline__ int get_bit(const uint8_t* v, int b) {
  return (v[b >> 3] >> (7 - (b & 7))) & 1;
}

// Set bits among bits b0 .. b0+n-1 of v (MSB-first numbering).
__device__ int popc_bits(const uint8_t* v, int b0, int n) {
  int c = 0;
  int b = b0;
  const int end = b0 + n;
  while (b < end) {
    const int bit = b & 7;
    const int take = min(8 - bit, end - b);
    const unsigned mask = (0xFFu >> bit) & (0xFFu << (8 - bit - take));
    c += __popc(static_cast<unsigned>(v[b >> 3]) & mask);
    b += take;
  }
  return c;
}

__global__ __launch_bounds__(256) void decode_count(PlanTables pt, const uint8_t* __restrict__ la,
                                                    const uint8_t* __restrict__ ca,
                                                    int32_t* __restrict__ counts) {
  const int64_t M = pt.num_tiles;
  const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= M * pt.num_q_heads) return;
  const int h = static_cast<int>(r / M);
  const int m = static_cast<int>(r - static_cast<int64_t>(h) * M);
  const int s = pt.tile_seg[m];
  if (pt.seg_kind[s] == kQuery) {
    counts[r] = m - pt.tile_lo[m] + 1;
    return;
  }
  const int i = m - pt.seg_tile0[s];
  const int P = pt.seg_pages[s];
  const uint8_t* lav = la + pt.seg_la_off[s] + static_cast<int64_t>(h) * la_nbytes(P);
  int c = 1 + popc_bits(lav, i * (i + 1) / 2, i);
  for (int e = pt.seg_first[s]; e < s; ++e) {
    const int Pe = pt.seg_pages[e];
    c += popc_bits(ca + pt.seg_ca_off[e] + static_cast<int64_t>(h) * ca_nbytes(Pe), 0, Pe);
  }
  counts[r] = c;
}

// Exclusive scan of n counts into row_ptr[0..n]; a single 1024-thread block.
// Thread t owns a contiguous chunk; chunk totals are scanned with wavefront
// shuffles and one LDS step across the 16 wavefronts.
__global__ __launch_bounds__(1024) void decode_scan(const int32_t* __restrict__ counts,
                                                    int32_t* __restrict__ row_ptr, int64_t n) {
  __shared__ int32_t wsum[16];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int w = t >> 6;
  const int64_t per = (n + 1023) / 1024;
  const int64_t a = min(n, static_cast<int64_t>(t) * per);
  const int64_t z = min(n, a + per);
  int32_t s = 0;
  for (int64_t i = a; i < z; ++i) s += counts[i];
  int32_t x = s;  // inclusive scan inside the wavefront
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  if (w == 0) {
    int32_t ws = lane < 16 ? wsum[lane] : 0;
    for (int off = 1; off < 16; off <<= 1) {
      const int32_t y = __shfl_up(ws, off, 64);
      if (lane >= off) ws += y;
    }
    if (lane < 16) wsum[lane] = ws;
  }
  __syncthreads();
  int32_t excl = x - s + (w > 0 ? wsum[w - 1] : 0);
  for (int64_t i = a; i < z; ++i) {
    row_ptr[i] = excl;
    excl += counts[i];
  }
  if (t == 1023) row_ptr[n] = excl;
}

// Append to col_idx[pos..] the indices base + b of the set bits among bits
// b0 .. b0+n-1 of v, in bit order; returns the new pos.  Wave-cooperative.
__device__ __forceinline__ int32_t emit_bits(const uint8_t* v, int b0, int n, int32_t base,
                                             int32_t pos, int lane, int32_t* __restrict__ col) {
  const unsigned long long below = (1ull << lane) - 1ull;
  for (int c0 = 0; c0 < n; c0 += 64) {
    const int b = c0 + lane;
    const bool on = b < n && get_bit(v, b0 + b);
    const unsigned long long mask = __ballot(on);
    if (on) col[pos + __popcll(mask & below)] = base + b;
    pos += __popcll(mask);
  }
  return pos;
}

__global__ __launch_bounds__(256) void decode_write(PlanTables pt, const uint8_t* __restrict__ la,
                                                    const uint8_t* __restrict__ ca,
                                                    const int32_t* __restrict__ row_ptr,
                                                    int32_t* __restrict__ col) {
  const int64_t M = pt.num_tiles;
  const int lane = threadIdx.x & 63;
  const int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (r >= M * pt.num_q_heads) return;  // uniform per wavefront
  const int h = static_cast<int>(r / M);
  const int m = static_cast<int>(r - static_cast<int64_t>(h) * M);
  const int s = pt.tile_seg[m];
  int32_t pos = row_ptr[r];
  if (pt.seg_kind[s] == kQuery) {
    const int n0 = pt.tile_lo[m];
    const int cnt = m - n0 + 1;
    for (int k = lane; k < cnt; k += 64) col[pos + k] = n0 + k;
    return;
  }
  for (int e = pt.seg_first[s]; e < s; ++e) {
    const int Pe = pt.seg_pages[e];
    const uint8_t* cav = ca + pt.seg_ca_off[e] + static_cast<int64_t>(h) * ca_nbytes(Pe);
    pos = emit_bits(cav, 0, Pe, pt.seg_tile0[e], pos, lane, col);
  }
  const int i = m - pt.seg_tile0[s];
  const int P = pt.seg_pages[s];
  const uint8_t* lav = la + pt.seg_la_off[s] + static_cast<int64_t>(h) * la_nbytes(P);
  pos = emit_bits(lav, i * (i + 1) / 2, i, pt.seg_tile0[s], pos, lane, col);
  if (lane == 0) col[pos] = m;
}

}  // namespace

hipError_t launch_decode(const PlanTables& pt, const uint8_t* la, const uint8_t* ca,
                         int32_t* counts, int32_t* row_ptr, int32_t* col_idx,
                         hipStream_t stream) {
  const int64_t rows = static_cast<int64_t>(pt.num_tiles) * pt.num_q_heads;
  if (rows == 0) {  // empty layout: the scan alone writes row_ptr[0] = 0
    hipLaunchKernelGGL(decode_scan, dim3(1), dim3(1024), 0, stream, counts, row_ptr, rows);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(decode_count, dim3(static_cast<unsigned>((rows + 255) / 256)), dim3(256), 0,
                     stream, pt, la, ca, counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_scan, dim3(1), dim3(1024), 0, stream, counts, row_ptr, rows);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_write, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0,
                     stream, pt, la, ca, row_ptr, col_idx);
  return hipGetLastError();
}

}  // namespace sift
