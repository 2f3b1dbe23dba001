// Sparse attention over decoded tile lists, fp32 inputs (SIFT, Section 5.2).
//
// The fp32 path serves full-precision inputs at any supported tile size
// (T = 16, 32, 64) and head size (D = 64, 128).  There is no fp32 dense
// contraction worth an MFMA tiling at these sizes, so it runs on the vector
// ALUs: one workgroup per (query head, M-block), K and V tiles of each listed
// N-block staged in LDS, one wavefront per query row at a time, lane j owning
// key j of the tile for the scores and lanes owning head-dim columns for the
// P.V accumulation.  Online softmax in the log2 domain (running max and sum,
// output rescaled when the max grows), normalised once at the end.

#include "sift_internal.h"

namespace sift {
namespace {

__device__ __forceinline__ float wave_max(float x) {
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

template <int T, int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(PlanTables pt, AttnArgs a) {
  constexpr int R = T / 4;      // query rows per wavefront
  constexpr int C = D / 64;     // head-dim columns per lane
  constexpr int KP = D + 1;     // padded K row: lane j reads row j without bank conflicts
  __shared__ float Qs[T * D];
  __shared__ float Ks[T * KP];
  __shared__ float Vs[T * D];
  __shared__ __attribute__((aligned(16))) float Ps[4][T];  // a wavefront's weights of one row

  const int64_t M = pt.num_tiles;
  const int64_t row = blockIdx.x;
  const int h = static_cast<int>(row / M);
  const int m = static_cast<int>(row - static_cast<int64_t>(h) * M);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int kvh = h / (a.hq / a.hkv);
  const int qtok0 = pt.tile_tok0[m];
  const int qlen = pt.tile_len[m];
  const int lo = pt.tile_lo[m];
  const float* __restrict__ q = static_cast<const float*>(a.q);
  const float* __restrict__ k = static_cast<const float*>(a.k);
  const float* __restrict__ v = static_cast<const float*>(a.v);

  for (int e = tid; e < T * D; e += 256) {
    const int r = e / D, d = e - (e / D) * D;
    Qs[e] = r < qlen ? q[(static_cast<int64_t>(qtok0 + r) * a.hq + h) * D + d] : 0.f;
  }

  float mrun[R], lrun[R], o[R][C];
#pragma unroll
  for (int rr = 0; rr < R; ++rr) {
    mrun[rr] = -INFINITY;
    lrun[rr] = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) o[rr][c] = 0.f;
  }

  const int64_t cap = a.col_capacity;
  const int64_t beg = min(cap, max(static_cast<int64_t>(0), static_cast<int64_t>(a.row_ptr[row])));
  const int64_t end = min(cap, max(beg, static_cast<int64_t>(a.row_ptr[row + 1])));
  for (int64_t idx = beg; idx < end; ++idx) {
    const int n = a.col_idx[idx];
    if (n < lo || n > m) continue;  // outside the prompt or after the M-block
    const int ktok0 = kv_row0(pt, a.pages, n);
    const int klen = pt.tile_len[n];
    __syncthreads();  // previous tile fully consumed (and Qs written)
    for (int e = tid; e < T * D; e += 256) {
      const int r = e / D, d = e - (e / D) * D;
      const int64_t g = (static_cast<int64_t>(ktok0 + r) * a.hkv + kvh) * D + d;
      Ks[r * KP + d] = r < klen ? k[g] : 0.f;
      Vs[e] = r < klen ? v[g] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < R; ++rr) {
      // rows one after another: interleaved by the scheduler, the unrolled
      // rows' reads would all be held in registers at once
      asm volatile("" ::: "memory");
      const int qr = w + 4 * rr;  // query row inside the M-block
      float s = -INFINITY;
      const bool ok = lane < T && lane < klen && (n != m || lane <= qr);
      if (ok) {
        float acc = 0.f;
#pragma unroll 8
        for (int d = 0; d < D; ++d) acc = fmaf(Qs[qr * D + d], Ks[lane * KP + d], acc);
        s = acc * a.scale_log2;
      }
      const float mx = wave_max(s);
      const float mnew = fmaxf(mrun[rr], mx);
      const float base = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = exp2f(mrun[rr] - base);
      const float p = ok ? exp2f(s - base) : 0.f;
      lrun[rr] = lrun[rr] * alpha + wave_sum(p);
      mrun[rr] = mnew;
#pragma unroll
      for (int c = 0; c < C; ++c) o[rr][c] *= alpha;
      // the weights go through LDS (one wavefront writes and reads its own
      // row, in order) and come back four at a time to every lane
      if (lane < T) Ps[w][lane] = p;
#pragma unroll 4
      for (int j = 0; j < T; j += 4) {
        const float4 p4 = *reinterpret_cast<const float4*>(&Ps[w][j]);
#pragma unroll
        for (int c = 0; c < C; ++c) {
          float acc = o[rr][c];
          acc = fmaf(p4.x, Vs[j * D + lane + 64 * c], acc);
          acc = fmaf(p4.y, Vs[(j + 1) * D + lane + 64 * c], acc);
          acc = fmaf(p4.z, Vs[(j + 2) * D + lane + 64 * c], acc);
          acc = fmaf(p4.w, Vs[(j + 3) * D + lane + 64 * c], acc);
          o[rr][c] = acc;
        }
      }
    }
  }

  float* __restrict__ out = static_cast<float*>(a.out);
#pragma unroll
  for (int rr = 0; rr < R; ++rr) {
    const int qr = w + 4 * rr;
    if (qr >= qlen) continue;
    const float inv = lrun[rr] > 0.f ? 1.f / lrun[rr] : 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c)
      out[(static_cast<int64_t>(qtok0 + qr) * a.hq + h) * D + lane + 64 * c] = o[rr][c] * inv;
  }
}

template <int T, int D>
hipError_t launch_t(const PlanTables& pt, const AttnArgs& a, hipStream_t stream) {
  const int64_t rows = static_cast<int64_t>(pt.num_tiles) * pt.num_q_heads;
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL((attn_f32_kernel<T, D>), dim3(static_cast<unsigned>(rows)), dim3(256), 0,
                     stream, pt, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_f32(const PlanTables& pt, const AttnArgs& a, hipStream_t stream) {
  if (a.head_dim == 64) {
    if (a.tile == 16) return launch_t<16, 64>(pt, a, stream);
    if (a.tile == 32) return launch_t<32, 64>(pt, a, stream);
    if (a.tile == 64) return launch_t<64, 64>(pt, a, stream);
  } else if (a.head_dim == 128) {
    if (a.tile == 16) return launch_t<16, 128>(pt, a, stream);
    if (a.tile == 32) return launch_t<32, 128>(pt, a, stream);
    if (a.tile == 64) return launch_t<64, 128>(pt, a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace sift
