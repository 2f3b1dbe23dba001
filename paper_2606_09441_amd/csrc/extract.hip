// Offline metadata extraction on the GPU (Sections 4.1, 4.2; the metadata is
// made by a dense standalone prefill of each document, Section 4.4).
//
// For every document, query head and block of 128 query rows, one workgroup
// (4 wavefronts x 32 rows) walks the causal key blocks of 64 keys twice:
//
//   pass 1: S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (queries on lanes, as in
//           the attention kernel), running row max m and row sum l of
//           exp2(c S - m), c = scale * log2(e);
//   pass 2: the same S; probability A = exp2(c S - m) / l exceeds a threshold
//           t exactly when S > (log2 t + log2 l + m) / c, so the decisions
//           need no exponential.  LA: a tile's flag is set when any of its
//           cells passes alpha (wavefront ballots over 16-key quarters, one
//           byte store per set flag).  CA: the cells of each key page that
//           pass beta are counted (ballot popcounts, one atomic add per page
//           and wavefront).
//
// A pack pass then turns flags into LA bits and counts into CA bits (count >
// gamma * the page's causal cells), MSB first, document-major with the query
// heads inside each document: the layout the online path reads.

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "sift_internal.h"

namespace sift {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kQB = 128;  // query rows per workgroup
constexpr int kKB = 64;   // keys per block

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Key index (inside the 64-key block) of accumulator a, register j of a lane
// in half hf of the wavefront (32x32 MFMA output layout).
__device__ __forceinline__ int key_of(int a, int j, int hf) {
  return 32 * a + 8 * (j >> 2) + 4 * hf + (j & 3);
}

// Global -> LDS copy of one block of 64 key rows, 16-byte chunks, chunk
// index XOR (row & (chunks per row - 1)) so that the 32 rows read by one
// MFMA fragment spread over the banks.  Rows at or past `rows` are zero.
template <int D>
struct KLoader {
  static constexpr int kCpr = D / 8;               // chunks per row
  static constexpr int kPer = kKB * kCpr / 256;    // chunks per thread
  u32x4 r[kPer];
  __device__ __forceinline__ void fetch(const __bf16* kbase, int64_t row_stride, int rows) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = threadIdx.x + 256 * i;
      const int row = c / kCpr, ch = c % kCpr;
      r[i] = u32x4{0u, 0u, 0u, 0u};
      if (row < rows) r[i] = *reinterpret_cast<const u32x4*>(kbase + row * row_stride + ch * 8);
    }
  }
  __device__ __forceinline__ void store(__bf16* lds) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = threadIdx.x + 256 * i;
      const int row = c / kCpr, ch = c % kCpr;
      *reinterpret_cast<u32x4*>(lds + row * D + ((ch ^ (row & (kCpr - 1))) * 8)) = r[i];
    }
  }
};

// S^T for 64 keys x this wavefront's 32 queries: s[0] keys 0..31, s[1] 32..63.
template <int D>
__device__ __forceinline__ void scores(const __bf16* lds, const bf16x8 (&qf)[D / 16], int l32, int hf,
                                       f32x16 (&s)[2]) {
  constexpr int kCpr = D / 8;
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int row = 32 * a + l32;
    s[a] = f32x16{};
#pragma unroll
    for (int k = 0; k < D / 16; ++k) {
      const int ch = (2 * k + hf) ^ (row & (kCpr - 1));
      const bf16x8 frag = *reinterpret_cast<const bf16x8*>(lds + row * D + ch * 8);
      s[a] = mfma(frag, qf[k], s[a]);
    }
  }
}

template <int D, int T>
__global__ __launch_bounds__(256, 3) void extract_kernel(ExtractArgs a) {
  constexpr int kKS = D / 16;
  // two K blocks: block kb is read from slot kb & 1 while block kb + 1 is
  // written to the other, one barrier per block
  __shared__ __attribute__((aligned(16))) __bf16 lds[2][kKB * D];

  const int2 bl = a.blocks[blockIdx.x];  // {document, query block}, longest first
  const ExtractDoc dc = a.docs[bl.x];
  const int h = blockIdx.y;
  const int kvh = h / (a.hq / a.hkv);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int row0 = bl.y * kQB + wave * 32;  // first query row of this wavefront
  const int p = row0 + l32;                 // this lane's query row (in the document)
  const int L = dc.len;

  bf16x8 qf[kKS];
  {
    const __bf16* src = a.q + (static_cast<int64_t>(dc.tok0 + p) * a.hq + h) * D + 8 * hf;
#pragma unroll
    for (int k = 0; k < kKS; ++k) {
      u32x4 x = u32x4{0u, 0u, 0u, 0u};
      if (p < L) x = *reinterpret_cast<const u32x4*>(src + 16 * k);
      qf[k] = __builtin_bit_cast(bf16x8, x);
    }
  }
  const int last = min(bl.y * kQB + kQB, L) - 1;  // last query row of the block
  const int nkb = last / kKB + 1;                 // causal key blocks
  const int wave_last = min(row0 + 31, L - 1);    // this wavefront's last row (may be < row0)
  const int64_t kstride = static_cast<int64_t>(a.hkv) * D;
  const __bf16* kdoc = a.k + static_cast<int64_t>(dc.tok0) * kstride + static_cast<int64_t>(kvh) * D;
  const float c = a.c;

  // Cells outside the causal triangle or the document become -inf (their
  // exponential is 0 and they pass no threshold).  A block is full for a
  // wavefront when all its keys precede the wavefront's first row and all
  // its rows are in the document: then nothing is masked.
  auto mask = [&](f32x16 (&s)[2], int kb) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int kg = kb * kKB + key_of(t, j, hf);
        if (!(kg <= p && p < L)) s[t][j] = -INFINITY;
      }
  };
  auto full = [&](int kb) { return kb * kKB + kKB - 1 <= row0 && row0 + 31 < L; };

  // ---- pass 1: row max and row sum (log2 domain)
  float m = -INFINITY, l = 0.f;
  KLoader<D> ld;
  ld.fetch(kdoc, kstride, min(kKB, L));
  ld.store(lds[0]);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const bool more = kb + 1 < nkb;
    if (more) ld.fetch(kdoc + static_cast<int64_t>(kb + 1) * kKB * kstride, kstride,
                       min(kKB, L - (kb + 1) * kKB));
    if (kb * kKB <= wave_last) {  // else no causal cell for this wavefront
      f32x16 s[2];
      scores<D>(lds[kb & 1], qf, l32, hf, s);
      if (!full(kb)) mask(s, kb);
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[t][j]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mn = fmaxf(m, mx * c);
      // mn == -inf: no key yet (lanes past the document's end)
      const float mb = mn == -INFINITY ? 0.f : mn;
      float sum = 0.f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < 16; ++j) sum += __builtin_amdgcn_exp2f(s[t][j] * c - mb);
      sum += __shfl_xor(sum, 32, 64);
      l = l * __builtin_amdgcn_exp2f(m - mb) + sum;
      m = mn;
    }
    if (more) ld.store(lds[(kb + 1) & 1]);
    __syncthreads();
  }

  // ---- pass 2: decisions.  A > t  <=>  S > (log2 t + log2 l + m) / c
  const float ll = l > 0.f ? log2f(l) : 0.f;
  const float thr_a = (a.log2_alpha + ll + m) / c;
  const float thr_b = (a.log2_beta + ll + m) / c;
  const int nt = dc.P * (dc.P + 1) / 2;
  uint8_t* flags = a.flags + dc.flag_off + static_cast<int64_t>(h) * nt;
  int32_t* counts = a.counts + dc.cnt_off + static_cast<int64_t>(h) * dc.P;
  ld.fetch(kdoc, kstride, min(kKB, L));
  ld.store(lds[0]);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const bool more = kb + 1 < nkb;
    if (more) ld.fetch(kdoc + static_cast<int64_t>(kb + 1) * kKB * kstride, kstride,
                       min(kKB, L - (kb + 1) * kKB));
    if (kb * kKB <= wave_last) {
      f32x16 s[2];
      scores<D>(lds[kb & 1], qf, l32, hf, s);
      if (!full(kb)) mask(s, kb);
      // per 16-key quarter: the lanes with a cell above alpha (a ballot per
      // register, OR-ed); per page: the cells above beta (ballot popcounts;
      // both halves of the wavefront hold keys of the same page)
      unsigned long long qa[4] = {0ull, 0ull, 0ull, 0ull};
      int cnt[4] = {0, 0, 0, 0};
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          qa[2 * t + (j >> 3)] |= __ballot(s[t][j] > thr_a);
          cnt[T == 16 ? 2 * t + (j >> 3) : (T == 32 ? t : 0)] += __popcll(__ballot(s[t][j] > thr_b));
        }
      // LA flags: fold the two halves of each quarter's ballot onto 32 queries
      uint32_t f[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) f[q] = static_cast<uint32_t>(qa[q]) | static_cast<uint32_t>(qa[q] >> 32);
      if (lane == 0) {
        if constexpr (T == 16) {
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            const int ti = row0 / 16 + r;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int tj = kb * 4 + q;
              if (((f[q] >> (16 * r)) & 0xffffu) && tj <= ti) flags[ti * (ti + 1) / 2 + tj] = 1;
            }
          }
        } else if constexpr (T == 32) {
          const int ti = row0 / 32;
          for (int q = 0; q < 2; ++q) {
            const int tj = kb * 2 + q;
            if ((f[2 * q] | f[2 * q + 1]) && tj <= ti) flags[ti * (ti + 1) / 2 + tj] = 1;
          }
        } else if constexpr (T == 64) {
          const int ti = row0 / 64;
          if ((f[0] | f[1] | f[2] | f[3]) && kb <= ti) flags[ti * (ti + 1) / 2 + kb] = 1;
        } else {  // T = 128: the tile spans the workgroup's rows and two key blocks
          const int ti = row0 / 128, tj = kb / 2;
          if ((f[0] | f[1] | f[2] | f[3]) && tj <= ti) flags[ti * (ti + 1) / 2 + tj] = 1;
        }
        if constexpr (T <= kKB) {
          constexpr int kPages = kKB / T;
#pragma unroll
          for (int q = 0; q < kPages; ++q)
            if (cnt[q] > 0) atomicAdd(&counts[kb * kPages + q], cnt[q]);
        } else {
          if (cnt[0] > 0) atomicAdd(&counts[kb / 2], cnt[0]);
        }
      }
    }
    if (more) ld.store(lds[(kb + 1) & 1]);
    __syncthreads();
  }
}

// One workgroup per (document, head): flags -> LA bytes, counts -> CA bytes.
__global__ __launch_bounds__(256) void extract_pack(ExtractArgs a, uint8_t* __restrict__ la,
                                                    uint8_t* __restrict__ ca, int tile) {
  const ExtractDoc dc = a.docs[blockIdx.x];
  const int h = blockIdx.y;
  const int P = dc.P, L = dc.len;
  const int nt = P * (P + 1) / 2;
  const int la_n = (nt + 7) / 8, ca_n = (P + 7) / 8;
  const uint8_t* flags = a.flags + dc.flag_off + static_cast<int64_t>(h) * nt;
  const int32_t* counts = a.counts + dc.cnt_off + static_cast<int64_t>(h) * P;
  uint8_t* la_v = la + dc.la_off + static_cast<int64_t>(h) * la_n;
  uint8_t* ca_v = ca + dc.ca_off + static_cast<int64_t>(h) * ca_n;
  for (int b = threadIdx.x; b < la_n; b += 256) {
    unsigned v = 0;
    for (int i = 0; i < 8; ++i) {
      const int idx = 8 * b + i;
      if (idx < nt && flags[idx]) v |= 0x80u >> i;
    }
    la_v[b] = static_cast<uint8_t>(v);
  }
  for (int b = threadIdx.x; b < ca_n; b += 256) {
    unsigned v = 0;
    for (int i = 0; i < 8; ++i) {
      const int j = 8 * b + i;
      if (j >= P) break;
      // causal cells of page j: sum over its keys k of (L - k)
      const int64_t k0 = static_cast<int64_t>(j) * tile;
      const int64_t k1 = min(static_cast<int64_t>(L), k0 + tile);
      const int64_t n = k1 - k0;
      const int64_t cells = n * L - (k0 + k1 - 1) * n / 2;
      if (static_cast<double>(counts[j]) > a.gamma * static_cast<double>(cells)) v |= 0x80u >> i;
    }
    ca_v[b] = static_cast<uint8_t>(v);
  }
}

__global__ __launch_bounds__(256) void zero_words(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += static_cast<int64_t>(gridDim.x) * 256)
    p[i] = 0u;
}

template <int D, int T>
void launch_extract_dt(const ExtractArgs& a, int nblocks, hipStream_t stream) {
  hipLaunchKernelGGL((extract_kernel<D, T>), dim3(nblocks, a.hq), dim3(256), 0, stream, a);
}

}  // namespace

hipError_t launch_extract(const ExtractArgs& a, int32_t num_docs, int32_t num_blocks,
                          int32_t head_dim, int32_t tile, uint32_t* zero_base, int64_t zero_words_n,
                          uint8_t* la, uint8_t* ca, hipStream_t stream) {
  if (zero_words_n > 0) {
    const int64_t g = std::min<int64_t>((zero_words_n + 255) / 256, 4096);
    hipLaunchKernelGGL(zero_words, dim3(static_cast<unsigned>(g)), dim3(256), 0, stream, zero_base,
                       zero_words_n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (num_blocks > 0) {
    if (head_dim == 128) {
      if (tile == 16) launch_extract_dt<128, 16>(a, num_blocks, stream);
      else if (tile == 32) launch_extract_dt<128, 32>(a, num_blocks, stream);
      else if (tile == 64) launch_extract_dt<128, 64>(a, num_blocks, stream);
      else launch_extract_dt<128, 128>(a, num_blocks, stream);
    } else {
      if (tile == 16) launch_extract_dt<64, 16>(a, num_blocks, stream);
      else if (tile == 32) launch_extract_dt<64, 32>(a, num_blocks, stream);
      else if (tile == 64) launch_extract_dt<64, 64>(a, num_blocks, stream);
      else launch_extract_dt<64, 128>(a, num_blocks, stream);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (num_docs > 0)
    hipLaunchKernelGGL(extract_pack, dim3(num_docs, a.hq), dim3(256), 0, stream, a, la, ca, tile);
  return hipGetLastError();
}

}  // namespace sift
