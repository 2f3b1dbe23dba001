// Rotary position embedding of q and k, in place, for the decoder-layer
// prefill slice at the Llama-3.1-8B shape (the model of Section 6).  Rotate-
// half form: for i < D/2, with angle a = pos * inv_freq[i] (an fp32 product),
//   x[i]       <- x[i] cos a - x[i + D/2] sin a
//   x[i + D/2] <- x[i + D/2] cos a + x[i] sin a
// inv_freq is given by the caller, so any frequency schedule (plain base^-2i/D
// or a rescaled one) is one table.  One thread per (token, head, pair i);
// bf16 in and out, fp32 arithmetic.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>

#include "sift_internal.h"

namespace sift {
namespace {

__device__ __forceinline__ float bf2f(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

__device__ __forceinline__ uint16_t f2bf(float f) {  // round to nearest even
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

__global__ __launch_bounds__(256) void rope_kernel(uint16_t* __restrict__ x, int64_t rows, int heads,
                                                   int half, const int32_t* __restrict__ pos,
                                                   const float* __restrict__ inv_freq) {
  const int64_t n = rows * heads * half;
  for (int64_t t = blockIdx.x * 256 + threadIdx.x; t < n; t += static_cast<int64_t>(gridDim.x) * 256) {
    const int i = static_cast<int>(t % half);
    const int64_t rh = t / half;              // token * heads + head
    const int64_t tok = rh / heads;
    const float a = static_cast<float>(pos[tok]) * inv_freq[i];
    float s, c;
    sincosf(a, &s, &c);
    uint16_t* p = x + rh * (2 * half);
    const float x1 = bf2f(p[i]), x2 = bf2f(p[i + half]);
    p[i] = f2bf(x1 * c - x2 * s);
    p[i + half] = f2bf(x2 * c + x1 * s);
  }
}

}  // namespace

hipError_t launch_rope(void* q, int64_t tokens, int hq, void* k, int hkv, int head_dim,
                       const int32_t* positions, const float* inv_freq, hipStream_t stream) {
  const int half = head_dim / 2;
  for (int pass = 0; pass < 2; ++pass) {
    void* x = pass == 0 ? q : k;
    const int heads = pass == 0 ? hq : hkv;
    const int64_t n = tokens * heads * half;
    if (n == 0) continue;
    const int64_t g = std::min<int64_t>((n + 255) / 256, 65536);
    hipLaunchKernelGGL(rope_kernel, dim3(static_cast<unsigned>(g)), dim3(256), 0, stream,
                       static_cast<uint16_t*>(x), tokens, heads, half, positions, inv_freq);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sift
