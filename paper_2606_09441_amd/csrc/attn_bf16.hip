// Sparse flash attention over decoded tile lists on bf16 MFMA (gfx950).
// SIFT, Section 5.2: a dense flash-attention main loop whose N-block
// iteration reads the next key tile from the decoded list instead of
// counting down; softmax and epilogue are those of dense attention.
//
// Design for CDNA4 (T = 64 keys per tile, D = 128):
//  * Work unit = (query head h, two consecutive M-blocks m0, m1 of one
//    segment): 128 query rows, 4 wavefronts of 32 rows.  Wavefronts 0-1 own
//    m0, 2-3 own m1.  The two lists are merged on the fly (both ascending);
//    every listed tile is staged once in LDS and each wavefront computes it
//    only if its own M-block lists it.  Two M-blocks of one document share
//    the whole cross-attention part of their lists (it depends on the key
//    document only), so the pair halves K/V traffic per row.
//  * S^T = K Q^T on v_mfma_f32_32x32x16_bf16: keys on the M side, queries on
//    the N side, so each lane holds one query's scores for 32 of the 64 keys
//    and row max / row sum are in-lane plus one exchange with lane ^ 32.
//  * The S^T accumulator, rounded to bf16, is already the B operand of
//    O^T += V^T P^T (same MFMA): the 16 keys of a k-step are permuted inside
//    the step, and V^T is written to LDS in that permuted key order.
//  * K rows are staged row-major (padded pitch), V transposed on the way in
//    (registers -> LDS), double buffered: the global loads of tile t+1 are in
//    flight while tile t is computed; one barrier per tile.
//  * Online softmax in the log2 domain; P is rounded to bf16 and the row sum
//    adds exactly those rounded values (v_dot2_f32_bf16 against 1.0), so
//    normalisation matches the weights the MFMA used.
//  * Workgroup -> unit mapping comes from the plan's schedule: units are
//    grouped per XCD (workgroups go round-robin over the 8 XCDs) so that the
//    query heads sharing a kv head, and the M-blocks sharing key pages, run
//    on one L2; longest lists first.

#include "sift_internal.h"

namespace sift {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kT = 64;
constexpr int kD = 128;
constexpr int kKPitch = kD + 8;            // bf16 per K row in LDS (272 B)
constexpr int kVPitch = kT + 8;            // bf16 per V^T row in LDS (144 B)
constexpr int kKElems = kT * kKPitch;
constexpr int kVElems = kD * kVPitch;
constexpr int kStage = kKElems + kVElems;  // one buffer: 35840 B
constexpr int kNone = 0x7fffffff;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

// Cursor over one ascending list, skipping entries outside [lo, hi].
struct ListCursor {
  const int32_t* col;
  int64_t i, e;
  int lo, hi;
  __device__ __forceinline__ int head() {
    while (i < e) {
      const int n = col[i];
      if (n >= lo && n <= hi) return n;
      ++i;
    }
    return kNone;
  }
};

struct Step {
  int n;      // key tile, kNone when done
  bool in0;   // listed by m0
  bool in1;   // listed by m1
};

__device__ __forceinline__ Step next_step(ListCursor& a, ListCursor& b) {
  const int na = a.head();
  const int nb = b.head();
  Step s;
  s.n = min(na, nb);
  s.in0 = na == s.n && na != kNone;
  s.in1 = nb == s.n && nb != kNone;
  if (s.in0) ++a.i;
  if (s.in1) ++b.i;
  return s;
}

// Global -> register staging of one K/V tile (256 threads).
//   K: thread t loads rows it*16 + t/16 (it = 0..3), 16 B chunk t%16.
//   V: thread t loads, for key group G = t/32 and head-dim quad dq = t%32,
//      the 8 keys base(G) + {0,1,2,3,8,9,10,11} at dims 4dq..4dq+3, with
//      base(G) = 32(G>>2) + 16((G>>1)&1) + 4(G&1).
struct TileRegs {
  u32x4 k[4];
  u32x2 v[8];
};

__device__ __forceinline__ void load_tile(TileRegs& r, const __bf16* __restrict__ kp,
                                          const __bf16* __restrict__ vp, int tok0, int len,
                                          int hkv, int kvh, int tid) {
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int row = it * 16 + (tid >> 4);
    const int ch = tid & 15;
    if (row < len) {
      const __bf16* src = kp + (static_cast<int64_t>(tok0 + row) * hkv + kvh) * kD + ch * 8;
      r.k[it] = *reinterpret_cast<const u32x4*>(src);
    } else {
      r.k[it] = u32x4{0u, 0u, 0u, 0u};
    }
  }
  const int G = tid >> 5;
  const int dq = tid & 31;
  const int base = 32 * (G >> 2) + 16 * ((G >> 1) & 1) + 4 * (G & 1);
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const int key = base + (t < 4 ? t : t + 4);
    if (key < len) {
      const __bf16* src = vp + (static_cast<int64_t>(tok0 + key) * hkv + kvh) * kD + dq * 4;
      r.v[t] = *reinterpret_cast<const u32x2*>(src);
    } else {
      r.v[t] = u32x2{0u, 0u};
    }
  }
}

// Register -> LDS: K row-major; V transposed to V^T[d][pos] with the key at
// pos = key with bits 2 and 3 swapped (the permutation the P^T operand uses).
__device__ __forceinline__ void store_tile(const TileRegs& r, __bf16* stage, int tid) {
  __bf16* Ks = stage;
  __bf16* Vt = stage + kKElems;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int row = it * 16 + (tid >> 4);
    const int ch = tid & 15;
    *reinterpret_cast<u32x4*>(Ks + row * kKPitch + ch * 8) = r.k[it];
  }
  const int G = tid >> 5;
  const int dq = tid & 31;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    // element e (dim 4dq+e) of each of the 8 loaded keys, packed in key order
    const int w = e >> 1;
    u32x4 o;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const unsigned lo = r.v[2 * p][w];
      const unsigned hi = r.v[2 * p + 1][w];
      o[p] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    *reinterpret_cast<u32x4*>(Vt + (4 * dq + e) * kVPitch + G * 8) = o;
  }
}

template <bool kOutF32>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(PlanTables pt, WorkTables wt,
                                                           AttnArgs a) {
  __shared__ __attribute__((aligned(16))) __bf16 lds[2 * kStage];

  const int unit = wt.sched[blockIdx.x];
  if (unit < 0) return;
  const int h = wt.unit_head[unit];
  const int m0 = wt.unit_m0[unit];
  const int m1 = wt.unit_m1[unit];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int hq = a.hq;
  const int hkv = a.hkv;
  const int kvh = h / (hq / hkv);
  const int lo = pt.tile_lo[m0];
  const int mine = wave < 2 ? m0 : m1;     // this wavefront's M-block (-1: none)
  const int qrow = (wave & 1) * 32 + l32;  // query row inside that M-block
  const __bf16* __restrict__ qp = static_cast<const __bf16*>(a.q);
  const __bf16* __restrict__ kp = static_cast<const __bf16*>(a.k);
  const __bf16* __restrict__ vp = static_cast<const __bf16*>(a.v);

  // Q^T fragments (B operand of S^T = K Q^T): lane holds query row qrow,
  // dims 16s + 8hf .. +7 for k-step s.
  int qtok0 = 0, qlen = 0;
  if (mine >= 0) {
    qtok0 = pt.tile_tok0[mine];
    qlen = pt.tile_len[mine];
  }
  bf16x8 qf[8];
  {
    const bool live = qrow < qlen;
    const __bf16* src = qp + (static_cast<int64_t>(qtok0 + qrow) * hq + h) * kD + 8 * hf;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      u32x4 x = u32x4{0u, 0u, 0u, 0u};
      if (live) x = *reinterpret_cast<const u32x4*>(src + 16 * s);
      qf[s] = as_bf16x8(x);
    }
  }

  // the two lists, clamped to the list buffer
  const int64_t M = pt.num_tiles;
  const int64_t cap = a.col_capacity;
  auto clampi = [cap](int64_t x) { return min(cap, max(static_cast<int64_t>(0), x)); };
  ListCursor la{a.col_idx, 0, 0, lo, m0};
  ListCursor lb{a.col_idx, 0, 0, lo, m1};
  {
    const int64_t r0 = static_cast<int64_t>(h) * M + m0;
    la.i = clampi(a.row_ptr[r0]);
    la.e = max(la.i, clampi(a.row_ptr[r0 + 1]));
    if (m1 >= 0) {
      const int64_t r1 = static_cast<int64_t>(h) * M + m1;
      lb.i = clampi(a.row_ptr[r1]);
      lb.e = max(lb.i, clampi(a.row_ptr[r1 + 1]));
    }
  }

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  float mrun = -INFINITY;
  float lrun = 0.f;
  const float c = a.scale_log2;

  TileRegs regs;
  Step cur = next_step(la, lb);
  if (cur.n != kNone) {
    load_tile(regs, kp, vp, pt.tile_tok0[cur.n], pt.tile_len[cur.n], hkv, kvh, tid);
    store_tile(regs, lds, tid);
  }
  __syncthreads();
  int buf = 0;
  while (cur.n != kNone) {
    const Step nxt = next_step(la, lb);
    if (nxt.n != kNone)
      load_tile(regs, kp, vp, pt.tile_tok0[nxt.n], pt.tile_len[nxt.n], hkv, kvh, tid);

    const bool part = wave < 2 ? cur.in0 : cur.in1;
    if (part) {
      const __bf16* Ks = lds + buf * kStage;
      const __bf16* Vt = Ks + kKElems;
      // ---- S^T = K Q^T: two 32-key blocks
      f32x16 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[kb][v] = 0.f;
        const __bf16* krow = Ks + (32 * kb + l32) * kKPitch + 8 * hf;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4*>(krow + 16 * s));
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[kb], 0, 0, 0);
        }
      }
      // ---- causal mask on the diagonal tile, length mask on a partial tile
      const int klen = pt.tile_len[cur.n];
      if (cur.n == mine || klen < kT) {
        const bool diag = cur.n == mine;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = 32 * kb + 8 * (v >> 2) + 4 * hf + (v & 3);
            if (key >= klen || (diag && key > qrow)) sacc[kb][v] = -INFINITY;
          }
      }
      // ---- online softmax (log2 domain)
      float mx = sacc[0][0];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[kb][v]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(mrun, mx);
      const float mc = mnew == -INFINITY ? 0.f : mnew * c;
      const float alpha = __builtin_amdgcn_exp2f(mrun * c - mc);
      mrun = mnew;
      bf16x8 pb[4];
      float psum = 0.f;
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const int kb = st >> 1;
        const int v0 = 8 * (st & 1);
#pragma unroll
        for (int t = 0; t < 8; t += 2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[kb][v0 + t], c, -mc));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[kb][v0 + t + 1], c, -mc));
          const bf16x2 pp = bf16x2{static_cast<__bf16>(p0), static_cast<__bf16>(p1)};
          pb[st][t] = pp[0];
          pb[st][t + 1] = pp[1];
          psum = __builtin_amdgcn_fdot2_f32_bf16(pp, bf16x2{static_cast<__bf16>(1.f),
                                                            static_cast<__bf16>(1.f)},
                                                 psum, false);
        }
      }
      lrun = lrun * alpha + psum;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
      // ---- O^T += V^T P^T
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const __bf16* vrow = Vt + (32 * db + l32) * kVPitch + 8 * hf;
#pragma unroll
        for (int st = 0; st < 4; ++st) {
          const bf16x8 vf = as_bf16x8(*reinterpret_cast<const u32x4*>(vrow + 16 * st));
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[st], o[db], 0, 0, 0);
        }
      }
    }

    if (nxt.n != kNone) store_tile(regs, lds + (buf ^ 1) * kStage, tid);
    __syncthreads();
    buf ^= 1;
    cur = nxt;
  }

  // ---- epilogue: O = O^T / l, lane writes dims 32db + 8i + 4hf .. +3 of its row
  if (mine < 0 || qrow >= qlen) return;
  const float lt = lrun + __shfl_xor(lrun, 32, 64);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  const int64_t obase = (static_cast<int64_t>(qtok0 + qrow) * hq + h) * kD + 4 * hf;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = 32 * db + 8 * i;
      f32x4 x = f32x4{o[db][4 * i] * inv, o[db][4 * i + 1] * inv, o[db][4 * i + 2] * inv,
                      o[db][4 * i + 3] * inv};
      if constexpr (kOutF32) {
        *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + obase + d) = x;
      } else {
        const bf16x2 y0 = bf16x2{static_cast<__bf16>(x[0]), static_cast<__bf16>(x[1])};
        const bf16x2 y1 = bf16x2{static_cast<__bf16>(x[2]), static_cast<__bf16>(x[3])};
        u32x2 w;
        w[0] = __builtin_bit_cast(unsigned, y0);
        w[1] = __builtin_bit_cast(unsigned, y1);
        *reinterpret_cast<u32x2*>(static_cast<__bf16*>(a.out) + obase + d) = w;
      }
    }
}

}  // namespace

hipError_t launch_attn_bf16(const PlanTables& pt, const WorkTables& wt, const AttnArgs& a,
                            hipStream_t stream) {
  if (a.tile != kT || a.head_dim != kD) return hipErrorInvalidValue;
  if (wt.grid == 0) return hipSuccess;
  if (a.out_f32)
    hipLaunchKernelGGL(attn_bf16_kernel<true>, dim3(wt.grid), dim3(256), 0, stream, pt, wt, a);
  else
    hipLaunchKernelGGL(attn_bf16_kernel<false>, dim3(wt.grid), dim3(256), 0, stream, pt, wt, a);
  return hipGetLastError();
}

}  // namespace sift
