// Sparse flash attention over decoded tile lists on bf16 MFMA (gfx950).
// SIFT, Section 5.2: a dense flash-attention main loop whose N-block
// iteration reads the next key tile from the decoded list instead of
// counting down; softmax and epilogue are those of dense attention.
//
// Design for CDNA4 (T = 64 keys per tile, D = 128):
//  * Work unit = (query head h, two consecutive M-blocks m0, m1 of one
//    segment): 128 query rows, 4 wavefronts of 32 rows.  Wavefronts 0-1 own
//    m0, 2-3 own m1.  The unit walks the merged step list the decode pass
//    wrote (the union of the two lists, each step flagged with the M-blocks
//    that list it); every listed tile is staged once in LDS and each
//    wavefront computes it only if its own M-block lists it.  Two M-blocks of one document share the
//    whole cross-attention part of their lists (it depends on the key
//    document only), so the pair halves K/V traffic per query row.
//  * S^T = K Q^T on v_mfma_f32_32x32x16_bf16: keys on the M side, queries on
//    the N side, so each lane holds one query's scores for 32 of the 64 keys;
//    row max and row sum are in-lane plus one v_permlane32_swap exchange.
//  * The S^T accumulator, rounded to bf16, is already the B operand of
//    O^T += V^T P^T (same MFMA): the 16 keys of a k-step are permuted inside
//    the step (lane half hf holds keys 4hf..4hf+3 and 8+4hf..8+4hf+3), and
//    the V^T A operand is read in that order from row-major V with the LDS
//    transpose read ds_read_b64_tr_b16 (in a 16-lane group, lane i gets
//    element i%4 of the 64-bit chunk addressed by lane 4j + i/4, j = 0..3:
//    column i of a 4-row block when lane 4j+q addresses row j, columns
//    4q..4q+3).
//  * K and V tiles are staged in LDS as unpadded 256 B rows with an XOR
//    swizzle of the 16-byte chunks (K: chunk ^ (row & 15), V: chunk ^
//    4(row & 3)) so that the MFMA operand reads are free of bank conflicts;
//    16 consecutive lanes store one row.  Global loads are buffer loads
//    through a per-tile resource that ends at the tile's last valid row:
//    rows past the end of a partial tile arrive as zeros.
//  * Double-buffered staging, one barrier per tile: the loads of step t+1's
//    K and V are issued into registers at the start of step t, step t is
//    computed from LDS, and the registers are stored into the other buffer
//    at its end.  Two workgroups per CU (2 wavefronts per SIMD) let one
//    wavefront's MFMAs overlap the other's softmax.
//  * Online softmax in the log2 domain with a lazy reference max (rescale
//    only when a tile's max exceeds it by more than kLazy); P is rounded to
//    bf16 and the row sum adds exactly those rounded values
//    (v_dot2_f32_bf16 against 1.0), so normalisation matches the weights
//    the MFMA used.
//  * Workgroup -> unit mapping comes from the plan's schedule: units are
//    grouped per XCD (workgroups go round-robin over the 8 XCDs) so that the
//    query heads sharing a kv head, and the M-blocks sharing key pages, run
//    on one L2; longest lists first.

#include "sift_internal.h"

namespace sift {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) __bf16 lds_bf16;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

constexpr int kT = 64;
constexpr int kD = 128;
constexpr int kTile = kT * kD;     // bf16 per staged K or V tile (16 KB)
constexpr int kNone = 0x7fffffff;
constexpr int kBufferWord3 = 0x00020000;  // gfx9-family raw buffer resource word 3

// Scores are compared against the running reference max only in steps of
// kLazy (log2 units): the reference moves, and O and l are rescaled, only
// when a tile's max exceeds it by more than kLazy.  exp2 arguments stay
// <= kLazy, so P <= 2^kLazy: no overflow, and the same bf16 relative precision.
constexpr float kLazy = 8.0f;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// One step of a unit's merged list (see WorkTables), wave-uniform.
struct Step {
  int tok0;  // first token of the key tile
  int info;  // len | in0 | in1 | diag0 | diag1
  bool valid;
  __device__ __forceinline__ int len() const { return info & kStepLenMask; }
  __device__ __forceinline__ bool in(int w) const {
    return (info & (w < 2 ? kStepIn0 : kStepIn1)) != 0;
  }
  __device__ __forceinline__ bool diag(int w) const {
    return (info & (w < 2 ? kStepDiag0 : kStepDiag1)) != 0;
  }
};

__device__ __forceinline__ Step make_step(int2 x, bool valid) {
  Step s;
  s.tok0 = __builtin_amdgcn_readfirstlane(x.x);
  s.info = __builtin_amdgcn_readfirstlane(x.y);
  s.valid = valid;
  if (!valid) s.info = kT;  // a full-length dummy for unconditional reloads
  return s;
}

// Global -> registers: thread t loads, for it = 0..3, row 16*(t/64) + 4it +
// (t%64)/16 of the tile, logical 16-byte chunk (t%16) ^ swizzle(row), which
// it later stores at physical chunk t%16 of that row (koff/voff are the
// per-thread byte offsets of those chunks).
__device__ __forceinline__ void load_tile(u32x4 (&r)[4], const __bf16* __restrict__ base, int len,
                                          int row_bytes, const int (&off)[4]) {
  const int valid = (len - 1) * row_bytes + kD * 2;  // through the last valid row
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<__bf16*>(base), 0, valid, kBufferWord3);
#pragma unroll
  for (int it = 0; it < 4; ++it)
    r[it] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off[it], 0, 0));
}

// Registers -> LDS: 16 consecutive lanes write one 256 B row.
__device__ __forceinline__ void store_tile(const u32x4 (&r)[4], lds_bf16* dst) {
#pragma unroll
  for (int it = 0; it < 4; ++it)
    *reinterpret_cast<__attribute__((address_space(3))) u32x4*>(dst + it * 4 * kD) = r[it];
}

// A operand of S^T = K Q^T: lane (l32, hf) reads row 32kb + l32, logical
// 16-byte chunk 2s + hf, stored at chunk (2s + hf) ^ (row & 15).
struct QkArgs {
  const lds_bf16* ks;
  int row0;  // l32 * kD
  int sw;    // l32 & 15 (== row & 15 for both 32-row blocks)
  int hf;
};

__device__ __forceinline__ bf16x8 k_frag(const QkArgs& q, int kb, int s) {
  const int chunk = (2 * s + q.hf) ^ q.sw;
  const lds_bf16* p = q.ks + q.row0 + kb * 32 * kD + chunk * 8;
  return as_bf16x8(*reinterpret_cast<const lds_u32x4*>(p));
}

// V^T operand of O^T += V^T P^T for head-dim block db and key step st: lane
// l (l32, hf) needs V[key][32db + l32] for the keys 16st + 4hf + {0..3} and
// 16st + 8 + 4hf + {0..3}: two transpose reads of 4-row blocks.  Lane l is
// the source lane of row (l & 15) >> 2 of each block, columns 32db +
// 16((l >> 4) & 1) + 4(l & 3) .. +3; the V swizzle XORs the 16-byte chunk
// with 4 * (row & 3) = 4 * ((l & 15) >> 2), constant per lane.
struct PvArgs {
  const lds_bf16* vs;
  int row0;   // (((l & 15) >> 2) + 4hf) * kD
  int cbase;  // 16((l >> 4) & 1) + 4(l & 3)
  int sw;     // 4 * ((l & 15) >> 2)
};

__device__ __forceinline__ bf16x8 v_frag(const PvArgs& v, int db, int st) {
  const int col = 32 * db + v.cbase;                    // logical column of the 8 B piece
  const int pc = ((col >> 3) ^ v.sw) * 8 + (col & 7);   // swizzled element column
  const lds_bf16* p0 = v.vs + v.row0 + 16 * st * kD + pc;
  const lds_bf16* p1 = p0 + 8 * kD;  // keys + 8: row & 3 unchanged, same swizzle
  const bf16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p0);
  const bf16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p1);
  return bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
}

__device__ __forceinline__ void qk_tile(const QkArgs& q, const bf16x8 (&qf)[8], f32x16& s0,
                                        f32x16& s1) {
  bf16x8 a0 = k_frag(q, 0, 0), a1 = k_frag(q, 1, 0);
  s0 = mfma(a0, qf[0], f32x16{});
  s1 = mfma(a1, qf[0], f32x16{});
#pragma unroll
  for (int s = 1; s < 8; ++s) {
    a0 = k_frag(q, 0, s);
    a1 = k_frag(q, 1, s);
    s0 = mfma(a0, qf[s], s0);
    s1 = mfma(a1, qf[s], s1);
  }
}

// x from lane l ^ 32: v_permlane32_swap exchanges the upper half of one
// register with the lower half of another; with both holding x, the pair
// (a, b) has a = x(l) and b = x(l ^ 32) on the lower half and the reverse on
// the upper half.  Issued as inline asm: the builtin's two results were
// folded into one by the compiler when both inputs are the same value.
__device__ __forceinline__ void swap_halves(float x, float& a, float& b) {
  a = x;
  b = x;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}

__device__ __forceinline__ float swap_max(float x) {
  float a, b;
  swap_halves(x, a, b);
  return fmaxf(a, b);
}

__device__ __forceinline__ float swap_sum(float x) {
  float a, b;
  swap_halves(x, a, b);
  return a + b;
}

// Row state of one wavefront: 32 query rows; lanes l and l^32 share row l32.
struct RowState {
  f32x16 o[4];  // O^T, head-dim blocks of 32
  float mref;   // reference max (times c)
  float lsum;   // this lane's share of the row sum
};

// Mask (diagonal / partial tile) and lazy-rescale step of the softmax for
// scores s0/s1 of a tile this wavefront computes.  Returns the exp base.
__device__ __forceinline__ float softmax_prepare(f32x16& s0, f32x16& s1, RowState& st,
                                                 const Step& cur, int wave, int qrow, int hf,
                                                 float c) {
  const bool diag = cur.diag(wave);
  if (diag || cur.len() < kT) {
    // key of value v of block kb: 32kb + 8(v>>2) + 4hf + (v&3)
    const int klim = cur.len() - 4 * hf;
    const int qlim = diag ? qrow - 4 * hf : 1 << 20;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int kc = 8 * (v >> 2) + (v & 3);
      if (kc >= klim || kc > qlim) s0[v] = -INFINITY;
      if (kc + 32 >= klim || kc + 32 > qlim) s1[v] = -INFINITY;
    }
  }
  float mx = fmaxf(s0[0], s1[0]);
#pragma unroll
  for (int v = 1; v < 16; ++v) mx = fmaxf(mx, fmaxf(s0[v], s1[v]));
  mx = swap_max(mx);
  const float mxs = mx * c;
  const bool grow = mxs > st.mref + kLazy;
  if (__builtin_amdgcn_ballot_w64(grow)) {
    const float mnew = grow ? mxs : st.mref;
    const float alpha = __builtin_amdgcn_exp2f(st.mref - mnew);
    st.mref = mnew;
    st.lsum *= alpha;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) st.o[db][v] *= alpha;
  }
  return st.mref == -INFINITY ? 0.f : st.mref;
}

// P = exp2(s*c - base) rounded to bf16, packed as the four B operands of
// O^T += V^T P^T; the row sum adds the rounded values.
__device__ __forceinline__ void softmax_exp(const f32x16& s0, const f32x16& s1, float c,
                                            float base, bf16x8 (&pb)[4], float& lsum) {
  const bf16x2 ones = bf16x2{static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
  float psum = 0.f;
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
  lsum += psum;
}

__device__ __forceinline__ void pv_tile(const PvArgs& v, const bf16x8 (&pb)[4], RowState& st) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int db = 0; db < 4; ++db) st.o[db] = mfma(v_frag(v, db, s), pb[s], st.o[db]);
}

template <bool kOutF32>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(PlanTables pt, WorkTables wt,
                                                           AttnArgs a) {
  // K slot 0, K slot 1, V slot 0, V slot 1 (16 KB each)
  __shared__ __attribute__((aligned(1024))) __bf16 smem[4 * kTile];

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
  const int row_bytes = kstride * 2;
  const int mine = wave < 2 ? m0 : m1;     // this wavefront's M-block (-1: none)
  const int qrow = (wave & 1) * 32 + l32;  // query row inside that M-block
  const float c = a.scale_log2;
  const __bf16* __restrict__ qp = static_cast<const __bf16*>(a.q);
  const __bf16* __restrict__ kp = static_cast<const __bf16*>(a.k);
  const __bf16* __restrict__ vp = static_cast<const __bf16*>(a.v);
  lds_bf16* lds = (lds_bf16*)smem;
  lds_bf16* const kslot[2] = {lds, lds + kTile};
  lds_bf16* const vslot[2] = {lds + 2 * kTile, lds + 3 * kTile};

  // global byte offsets: row 16w + 4it + l/16, logical chunk (l%16) ^
  // swizzle(row); this thread stores at element 16w*kD + it*4*kD + 8l.
  int koff[4], voff[4];
  {
    const int rsub = lane >> 4;
    const int pc = lane & 15;
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int row = 16 * wave + 4 * it + rsub;
      koff[it] = row * row_bytes + ((pc ^ (row & 15)) * 16);
      voff[it] = row * row_bytes + ((pc ^ (4 * (row & 3))) * 16);
    }
  }
  const int st_off = 16 * wave * kD + 8 * lane;

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

  // the unit's merged steps
  const int2* __restrict__ steps = wt.steps + wt.step_off[unit];
  const int nsteps = wt.step_cnt[unit];
  const int64_t kv_head_off = static_cast<int64_t>(kvh) * kD;
  auto tile_ptr = [&](const __bf16* base, const Step& s) {
    return base + static_cast<int64_t>(s.tok0) * kstride + kv_head_off;
  };
  auto fetch = [&](int i) { return steps[i < nsteps ? i : 0]; };

  RowState rs;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) rs.o[db][v] = 0.f;
  rs.mref = -INFINITY;
  rs.lsum = 0.f;

  QkArgs qa;
  qa.row0 = l32 * kD;
  qa.sw = l32 & 15;
  qa.hf = hf;
  PvArgs pva;
  pva.row0 = (((lane & 15) >> 2) + 4 * hf) * kD;
  pva.cbase = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  pva.sw = 4 * ((lane & 15) >> 2);

  // ---- prologue: stage step 0
  // (an empty list leaves O = 0 and l = 0: the epilogue writes zeros)
  u32x4 kr[4], vr[4];
  Step cur = make_step(fetch(0), nsteps > 0);
  int2 raw1 = fetch(1);
  if (cur.valid) {
    load_tile(kr, tile_ptr(kp, cur), cur.len(), row_bytes, koff);
    load_tile(vr, tile_ptr(vp, cur), cur.len(), row_bytes, voff);
    store_tile(kr, kslot[0] + st_off);
    store_tile(vr, vslot[0] + st_off);
  }
  __syncthreads();

  int par = 0;
  for (int t = 0; t < nsteps; ++t) {
    // Step t+1's tiles go into registers now and into the other buffer
    // after step t (past the end of the list: step t's tiles again, into a
    // buffer nobody reads, so loads and stores stay unconditional).  The
    // step after next is fetched here and decoded at the end of the step.
    const Step nx = make_step(raw1, t + 1 < nsteps);
    raw1 = fetch(t + 2);
    const Step& ld = nx.valid ? nx : cur;
    load_tile(kr, tile_ptr(kp, ld), ld.len(), row_bytes, koff);
    load_tile(vr, tile_ptr(vp, ld), ld.len(), row_bytes, voff);

    if (cur.in(wave)) {
      qa.ks = kslot[par];
      pva.vs = vslot[par];
      f32x16 s0, s1;
      qk_tile(qa, qf, s0, s1);
      const float base = softmax_prepare(s0, s1, rs, cur, wave, qrow, hf, c);
      bf16x8 pb[4];
      softmax_exp(s0, s1, c, base, pb, rs.lsum);
      pv_tile(pva, pb, rs);
    }
    store_tile(kr, kslot[par ^ 1] + st_off);
    store_tile(vr, vslot[par ^ 1] + st_off);
    __syncthreads();
    cur = nx;
    par ^= 1;
  }

  // ---- epilogue: O = O^T / l, lane writes dims 32db + 8i + 4hf .. +3 of its row
  if (mine < 0 || qrow >= qlen) return;
  const float lt = swap_sum(rs.lsum);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  const int64_t obase = (static_cast<int64_t>(qtok0 + qrow) * hq + h) * kD + 4 * hf;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = 32 * db + 8 * i;
      f32x4 x = f32x4{rs.o[db][4 * i] * inv, rs.o[db][4 * i + 1] * inv,
                      rs.o[db][4 * i + 2] * inv, rs.o[db][4 * i + 3] * inv};
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
