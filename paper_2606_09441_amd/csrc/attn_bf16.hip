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
//    the step (lane half hf holds keys 4hf..4hf+3 and 8+4hf..8+4hf+3), and
//    the V^T A operand is read in that order from row-major V with gfx950's
//    LDS transpose read (ds_read_b64_tr_b16: in a 16-lane group, lane i gets
//    element i%4 of the 64-bit chunk addressed by lane 4j + i/4, j = 0..3,
//    i.e. column i of a 4-row block when lane 4j+q addresses row j, columns
//    4q..4q+3).
//  * K and V tiles are staged row-major in LDS with padded pitches (K: 272 B,
//    conflict-free 16 B row reads; V: 320 B, so the 4 rows x 64 B that two
//    16-lane groups of a transpose read touch fall on disjoint banks), double
//    buffered: the global loads of tile t+1 are in
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
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kT = 64;
constexpr int kD = 128;
constexpr int kKPitch = kD + 8;            // bf16 per K row in LDS (272 B)
constexpr int kVPitch = kD + 32;           // bf16 per V row in LDS (320 B)
constexpr int kKElems = kT * kKPitch;
constexpr int kVElems = kT * kVPitch;
constexpr int kStage = kKElems + kVElems;  // one buffer: 37888 B
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

// Global -> register staging of one K/V tile (256 threads): thread t loads
// rows it*16 + t/16 (it = 0..3), 16 B chunk t%16, of K and of V.
// Loads are buffer loads through a per-tile resource whose base is the
// tile's first token and whose range ends with the tile's last valid row:
// rows past the end of a partial tile read as zero, with no branch.  The
// per-thread byte offset is fixed for the whole kernel; the row block is a
// scalar offset.
struct TileRegs {
  u32x4 k[4];
  u32x4 v[4];
};

constexpr int kBufferWord3 = 0x00020000;  // gfx9-family raw buffer resource word 3

__device__ __forceinline__ void load_tile(TileRegs& r, const __bf16* __restrict__ kp,
                                          const __bf16* __restrict__ vp, int64_t tile_base,
                                          int len, int kstride, int off) {
  const int row_bytes = kstride * 2;
  const int valid = (len - 1) * row_bytes + kD * 2;  // through the last valid row
  const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<__bf16*>(kp + tile_base), 0, valid, kBufferWord3);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<__bf16*>(vp + tile_base), 0, valid, kBufferWord3);
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    r.k[it] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(kr, off, it * 16 * row_bytes, 0));
    r.v[it] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(vr, off, it * 16 * row_bytes, 0));
  }
}

// Register -> LDS, both row-major (16 consecutive lanes write one 256 B row).
__device__ __forceinline__ void store_tile(const TileRegs& r, __bf16* stage, int tid) {
  __bf16* Ks = stage;
  __bf16* Vs = stage + kKElems;
  const int row = tid >> 4;
  const int ch = (tid & 15) * 8;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    *reinterpret_cast<u32x4*>(Ks + (it * 16 + row) * kKPitch + ch) = r.k[it];
    *reinterpret_cast<u32x4*>(Vs + (it * 16 + row) * kVPitch + ch) = r.v[it];
  }
}

// A operand of O^T += V^T P^T for head-dim block db and key step st: lane l
// (l32 = l & 31, hf = l >> 5) needs V[key][32db + l32] for the 8 keys
// 16st + 4hf + {0,1,2,3} and 16st + 8 + 4hf + {0,1,2,3}: two transpose reads
// of 4-row blocks.  vaddr is this lane's source address for db = st = 0 and
// the first block: row ((l & 15) >> 2) + 4hf, columns 16((l >> 4) & 1) + 4(l & 3).
__device__ __forceinline__ bf16x8 v_operand(const __bf16* vaddr, int db, int st) {
  const __bf16* p0 = vaddr + (16 * st) * kVPitch + 32 * db;
  const __bf16* p1 = p0 + 8 * kVPitch;
  const bf16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4*)((__attribute__((address_space(3))) __bf16*)p0));
  const bf16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4*)((__attribute__((address_space(3))) __bf16*)p1));
  return bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
}

// Scores are compared against the running reference max only in steps of
// kLazy (log2 units): the reference moves, and O and l are rescaled, only
// when a tile's max exceeds it by more than kLazy.  exp2 arguments stay
// <= kLazy, so P <= 2^kLazy: no overflow, and the same bf16 relative precision.
constexpr float kLazy = 8.0f;

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
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int hq = a.hq;
  const int hkv = a.hkv;
  const int kvh = h / (hq / hkv);
  const int kstride = hkv * kD;
  const int lo = pt.tile_lo[m0];
  const int mine = wave < 2 ? m0 : m1;     // this wavefront's M-block (-1: none)
  const int qrow = (wave & 1) * 32 + l32;  // query row inside that M-block
  const __bf16* __restrict__ qp = static_cast<const __bf16*>(a.q);
  const __bf16* __restrict__ kp = static_cast<const __bf16*>(a.k);
  const __bf16* __restrict__ vp = static_cast<const __bf16*>(a.v);

  const int off = ((tid >> 4) * kstride + (tid & 15) * 8) * 2;  // bytes

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
    la.i = clampi(__builtin_amdgcn_readfirstlane(a.row_ptr[r0]));
    la.e = max(la.i, clampi(__builtin_amdgcn_readfirstlane(a.row_ptr[r0 + 1])));
    if (m1 >= 0) {
      const int64_t r1 = static_cast<int64_t>(h) * M + m1;
      lb.i = clampi(__builtin_amdgcn_readfirstlane(a.row_ptr[r1]));
      lb.e = max(lb.i, clampi(__builtin_amdgcn_readfirstlane(a.row_ptr[r1 + 1])));
    }
  }

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  float mref = -INFINITY;  // reference max, already multiplied by c
  float lrun = 0.f;        // this lane's share of the row sum (its 32 keys per tile)
  const float c = a.scale_log2;

  TileRegs regs;
  Step cur = next_step(la, lb);
  if (cur.n != kNone) {
    load_tile(regs, kp, vp, (static_cast<int64_t>(pt.tile_tok0[cur.n]) * hkv + kvh) * kD,
              pt.tile_len[cur.n], kstride, off);
    store_tile(regs, lds, tid);
  }
  __syncthreads();
  int buf = 0;
  while (cur.n != kNone) {
    const Step nxt = next_step(la, lb);
    // Prefetch the next tile (on the last step: the current one again, so
    // that loads and LDS stores are unconditional and no wait for them is
    // placed before this step's compute).
    const int pf = nxt.n != kNone ? nxt.n : cur.n;
    load_tile(regs, kp, vp, (static_cast<int64_t>(pt.tile_tok0[pf]) * hkv + kvh) * kD,
              pt.tile_len[pf], kstride, off);

    const bool part = wave < 2 ? cur.in0 : cur.in1;
    if (part) {
      const __bf16* Ks = lds + buf * kStage;
      const __bf16* vaddr = Ks + kKElems + (((lane & 15) >> 2) + 4 * hf) * kVPitch +
                            16 * ((lane >> 4) & 1) + 4 * (lane & 3);
      // ---- S^T = K Q^T: two independent 32-key chains, interleaved
      f32x16 s0, s1;
      {
        const __bf16* k0 = Ks + l32 * kKPitch + 8 * hf;
        const __bf16* k1 = k0 + 32 * kKPitch;
        bf16x8 a0 = as_bf16x8(*reinterpret_cast<const u32x4*>(k0));
        bf16x8 a1 = as_bf16x8(*reinterpret_cast<const u32x4*>(k1));
        s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[0], f32x16{}, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[0], f32x16{}, 0, 0, 0);
#pragma unroll
        for (int s = 1; s < 8; ++s) {
          a0 = as_bf16x8(*reinterpret_cast<const u32x4*>(k0 + 16 * s));
          a1 = as_bf16x8(*reinterpret_cast<const u32x4*>(k1 + 16 * s));
          s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[s], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[s], s1, 0, 0, 0);
        }
      }
      // ---- causal mask on the diagonal tile, length mask on a partial tile.
      // Key of value v of block kb: 32kb + 8(v>>2) + 4hf + (v&3); the
      // constant part is compared against limits shifted by 4hf.
      const int klen = pt.tile_len[cur.n];
      if (cur.n == mine || klen < kT) {
        const int klim = klen - 4 * hf;
        const int qlim = cur.n == mine ? qrow - 4 * hf : 1 << 20;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int kc = 8 * (v >> 2) + (v & 3);
          if (kc >= klim || kc > qlim) s0[v] = -INFINITY;
          if (kc + 32 >= klim || kc + 32 > qlim) s1[v] = -INFINITY;
        }
      }
      // ---- online softmax in the log2 domain, lazy reference max
      float mx = fmaxf(s0[0], s1[0]);
#pragma unroll
      for (int v = 1; v < 16; ++v) mx = fmaxf(mx, fmaxf(s0[v], s1[v]));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mxs = mx * c;
      const bool grow = mxs > mref + kLazy;
      if (__builtin_amdgcn_ballot_w64(grow)) {
        const float mnew = grow ? mxs : mref;
        const float alpha = __builtin_amdgcn_exp2f(mref - mnew);
        mref = mnew;
        lrun *= alpha;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
      }
      const float base = mref == -INFINITY ? 0.f : mref;
      bf16x8 pb[4];
      float psum = 0.f;
      const bf16x2 ones = bf16x2{static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const int v0 = 8 * (st & 1);
#pragma unroll
        for (int t = 0; t < 8; t += 2) {
          const float x0 = (st < 2) ? s0[v0 + t] : s1[v0 + t];
          const float x1 = (st < 2) ? s0[v0 + t + 1] : s1[v0 + t + 1];
          const float p0 = __builtin_amdgcn_exp2f(fmaf(x0, c, -base));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(x1, c, -base));
          const bf16x2 pp = bf16x2{static_cast<__bf16>(p0), static_cast<__bf16>(p1)};
          pb[st][t] = pp[0];
          pb[st][t + 1] = pp[1];
          psum = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, psum, false);
        }
      }
      lrun += psum;
      // ---- O^T += V^T P^T: four independent chains over the head dim
#pragma unroll
      for (int st = 0; st < 4; ++st) {
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const bf16x8 vf = v_operand(vaddr, db, st);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[st], o[db], 0, 0, 0);
        }
      }
    }

    store_tile(regs, lds + (buf ^ 1) * kStage, tid);
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
