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
//    4(row & 3)) so that the MFMA operand reads are free of bank conflicts.
//    They are copied by the LDS DMA form of the buffer load (each lane's 16
//    bytes land at M0 + 16 * lane, so the swizzle is applied to the global
//    address), through a per-tile resource that ends at the tile's last
//    valid row: rows past the end of a partial tile arrive as zeros.  No
//    registers hold staged data.  The DMA is issued as inline assembly and
//    waited for explicitly before the step's barrier: the compiler, which
//    cannot tell the DMA target from the buffers being read, would otherwise
//    wait for it before every LDS read.
//  * Software pipeline, one barrier per step.  During step t a wavefront
//    computes S(t+1) = K(t+1) Q^T on the MFMA pipe while the VALU turns S(t)
//    into P(t) (exp2, bf16 rounding, row sum), then O += V(t)^T P(t).
//    Meanwhile the DMA brings K(t+2) and V(t+1): K runs one tile ahead of
//    V, each with two LDS slots (a slot is refilled only after the barrier
//    that follows its last read).  Two workgroups per CU (2 wavefronts per
//    SIMD) cover the remaining stalls.
//  * Online softmax in the log2 domain, in two launches.  On gfx950 plain
//    VALU work does not overlap the MFMAs (the exponentials do), so every
//    VALU instruction per step counts.  The first launch takes no row max
//    per tile: a row's reference is the max of the first tile it sees, and
//    later tiles' weights are formed against it at whatever magnitude.  If
//    an output or row sum comes out non-finite (a weight overflowed), the
//    launch raises a flag and the second launch does every unit again with
//    a lazy running max (kLazy); otherwise the second launch only merges
//    the pieces of split units.  P is rounded
//    to bf16 and the row sum adds exactly those rounded values
//    (v_dot2_f32_bf16 against 1.0), so normalisation matches the weights
//    the MFMA used.
//  * Workgroup -> unit mapping comes from the plan's schedule: units are
//    grouped per XCD (workgroups go round-robin over the 8 XCDs) so that the
//    query heads sharing a kv head, and the M-blocks sharing key pages, run
//    on one L2; longest lists first.

#include <type_traits>

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
typedef int i32x4 __attribute__((ext_vector_type(4)));
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

// The pass over all units does not take a tile's row max at all.  A row's
// reference max is the max of the first tile that gives it a key (that key's
// weight is 1); later tiles' weights P = 2^(s c - mref) are formed against
// it.  P rounded to bf16 keeps its relative precision at any magnitude
// (bf16 has fp32's exponent range), and l and O accumulate in fp32, so the
// result does not depend on the reference as long as nothing overflows:
// weights far below the reference are negligible next to the reference's
// own weight 1 in any case.  A weight, row sum or output beyond fp32's range
// (scores more than about 120 log2 units above the row's first tile, |v|
// large enough with such weights, or non-finite inputs) ends up infinite or
// NaN in the row sum or the output, which the epilogue tests; the launch is
// then flagged and a second launch does every unit again with the lazy
// reference above (kLazy), whose weights are <= 2^kLazy.
// Workgroups of the launch that does the units again (it returns at once
// when the first launch raised no flag).
constexpr int kRedoGrid = 512;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// One step of a unit's merged list (see WorkTables), wave-uniform.
// Wavefronts 0-1 own the unit's first M-block, 2-3 its second.
struct Step {
  unsigned sub;  // T < 64: the sub-tile mask of the step (bit G k + s: M-block k lists key tile s)
  int kvt;   // T < 64: this wavefront's K/V row base (see WorkTables::kvb)
  int tok0;  // T >= 64: first token of the key tile; T < 64: the sub-tile mask
  int info;  // len | listed << 8 | diagonal << 12
  bool valid;
  __device__ __forceinline__ int len() const { return info & kStepLenMask; }
  __device__ __forceinline__ bool in(int w) const {
    return (info >> (kStepListedShift + (w >> 1))) & 1;
  }
  __device__ __forceinline__ bool diag(int w) const {
    return (info >> (kStepDiagShift + (w >> 1))) & 1;
  }
};

__device__ __forceinline__ Step make_step(int2 x, bool valid) {
  Step s;
  s.tok0 = __builtin_amdgcn_readfirstlane(x.x);
  s.info = __builtin_amdgcn_readfirstlane(x.y);
  // decoded here, not where first used: sunk into the next step, the wait
  // for x would also wait for that step's DMA
  asm volatile("" : "+s"(s.tok0), "+s"(s.info));
  s.valid = valid;
  s.sub = static_cast<unsigned>(s.tok0);
  s.kvt = 0;  // set by the caller at T < 64
  if (!valid) s.info = kT;  // a full-length dummy for unconditional reloads
  return s;
}

// Buffer resource of one key tile of one kv head: base = its first row,
// num_records = bytes through the last valid row (loads past it return 0).
// At T < 64 the base is an address: a wavefront's rows may start further
// into the step than into their own tile, so the base can precede the tensor.
__device__ __forceinline__ i32x4 tile_rsrc(unsigned long long a, int len, int row_bytes) {
  const int valid = (len - 1) * row_bytes + kD * 2;
  return i32x4{static_cast<int>(static_cast<unsigned>(a)), static_cast<int>((a >> 32) & 0xffff),
               valid, kBufferWord3};
}

// Global -> LDS, 16 bytes per lane from byte voff of the resource, landing
// at m0 + 16 * lane.
__device__ __forceinline__ void dma_b128(int m0, int voff, const i32x4& rs) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(m0), "v"(voff), "s"(rs)
               : "memory", "m0");
}

// One wavefront's quarter of a tile: rows 16w + 4it + lane/16 (it = 0..3),
// physical chunk lane % 16 of each.  off0 is the lane's global byte offset
// for it = 0; rows 4it further down sit it * rstep bytes further, and their
// logical chunk differs by an XOR of the chunk index with xsw(it) (bits 6-7
// of the byte offset; the row part is a multiple of 256).  row0 = LDS byte
// address of row 16w.
template <bool kXor>
__device__ __forceinline__ void dma_tile(int row0, int off0, int rstep, const i32x4& rs) {
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int off = (kXor ? (off0 ^ (it << 6)) : off0) + it * rstep;
    dma_b128(row0 + it * 4 * kD * 2, off, rs);
  }
}

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// A operand of S^T = K Q^T: lane (l32, hf) reads row 32kb + l32, logical
// 16-byte chunk 2s + hf, stored at chunk (2s + hf) ^ (row & 15).  With x =
// (l32 & 15) >> 1 the byte offset inside the row is 32(s ^ x) + 16(hf ^
// (l32 & 1)): the lane's address for s = 0 XORed with 32s (bits 5-7 of an
// address whose row part is a multiple of 256).
struct QkArgs {
  int addr;  // LDS byte address of k-step 0, block 0, in K slot 0
};

__device__ __forceinline__ bf16x8 k_frag(const QkArgs& q, int slot_off, int kb, int s) {
  const int a = (q.addr ^ (s << 5)) + slot_off + kb * 32 * kD * 2;
  return as_bf16x8(*reinterpret_cast<const lds_u32x4*>(static_cast<size_t>(a)));
}

// V^T operand of O^T += V^T P^T for head-dim block db and key step st: lane
// l (l32, hf) needs V[key][32db + l32] for the keys 16st + 4hf + {0..3} and
// 16st + 8 + 4hf + {0..3}: two transpose reads of 4-row blocks.  Lane l is
// the source lane of row (l & 15) >> 2 of each block, columns 32db +
// 16((l >> 4) & 1) + 4(l & 3) .. +3; the V swizzle XORs the 16-byte chunk
// with 4 * (row & 3) = 4 * ((l & 15) >> 2), constant per lane.  In bytes the
// column part is 64(db ^ ((l & 15) >> 2)) + 32((l >> 4) & 1) + 8(l & 3), so
// the address for db is the lane's address for db = 0 XORed with 64db.
struct PvArgs {
  int addr;  // LDS byte address of db = 0, st = 0, first block, in V slot 0
};

__device__ __forceinline__ bf16x8 v_frag(const PvArgs& v, int slot_off, int db, int st) {
  const int a = (v.addr ^ (db << 6)) + slot_off + 16 * st * kD * 2;
  const bf16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      reinterpret_cast<lds_bf16x4*>(static_cast<size_t>(a)));
  // keys + 8: row & 3 unchanged, same swizzle
  const bf16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      reinterpret_cast<lds_bf16x4*>(static_cast<size_t>(a + 8 * kD * 2)));
  return bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
}

__device__ __forceinline__ void qk_tile(const QkArgs& q, int slot_off, const bf16x8 (&qf)[8],
                                        f32x16& s0, f32x16& s1) {
  bf16x8 a0 = k_frag(q, slot_off, 0, 0), a1 = k_frag(q, slot_off, 1, 0);
  s0 = mfma(a0, qf[0], f32x16{});
  s1 = mfma(a1, qf[0], f32x16{});
#pragma unroll
  for (int s = 1; s < 8; ++s) {
    a0 = k_frag(q, slot_off, 0, s);
    a1 = k_frag(q, slot_off, 1, s);
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
  asm("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
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

// Scores of keys past the end of a partial tile, or after the query on the
// diagonal tile, become -inf.  Value v of block kb holds key 32kb + 8(v>>2)
// + 4hf + (v&3).
__device__ __forceinline__ void mask_tile(f32x16& s0, f32x16& s1, const Step& st, int wave,
                                          int qrow, int hf, bool all = false) {
  const int klim = all ? -64 : st.len() - 4 * hf;
  const int qlim = st.diag(wave) ? qrow - 4 * hf : 1 << 20;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int kc = 8 * (v >> 2) + (v & 3);
    if (kc >= klim || kc > qlim) s0[v] = -INFINITY;
    if (kc + 32 >= klim || kc + 32 > qlim) s1[v] = -INFINITY;
  }
}

__device__ __forceinline__ bool needs_mask(const Step& st, int wave) {
  return st.diag(wave) || st.len() < kT;
}

// T = 64 / kG < 64: a 64-key step holds kG key tiles and a wavefront's 32
// rows kG / 2 row tiles (T = 32: one, T = 16: two, lanes l32 < 16 and >= 16).
// Cells of (row tile, key tile) pairs the step's sub-tile mask leaves out
// become -inf.  Register v of s0 holds key 8 (v / 4) + 4 hf + v % 4, of s1
// the same + 32: key tile (of 16) 2 a + v / 8, (of 32) a.
template <int kG>
__device__ __forceinline__ bool sub_partial(const Step& st, int wave) {
  if constexpr (kG == 1) return false;
  constexpr unsigned kRow = (1u << (kG * kG / 2)) - 1u;  // a wavefront's bits
  return ((st.sub >> (wave * kG * kG / 2)) & kRow) != kRow;
}

template <int kG>
__device__ __forceinline__ void mask_sub(f32x16& s0, f32x16& s1, const Step& st, int wave, int l32) {
  if constexpr (kG == 2) {
    const unsigned m = (st.sub >> (2 * wave)) & 3u;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      if (!(m & 1u)) s0[v] = -INFINITY;
      if (!(m & 2u)) s1[v] = -INFINITY;
    }
  } else if constexpr (kG == 4) {
    const unsigned m = (st.sub >> (4 * (2 * wave + (l32 >> 4)))) & 15u;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      if (!((m >> (v >> 3)) & 1u)) s0[v] = -INFINITY;
      if (!((m >> (2 + (v >> 3))) & 1u)) s1[v] = -INFINITY;
    }
  }
}

// Row max of a score tile (both lane halves of the row agree).
__device__ __forceinline__ float tile_max(const f32x16& s0, const f32x16& s1) {
  float m0 = fmaxf(s0[0], s1[0]);
  float m1 = fmaxf(s0[1], s1[1]);
#pragma unroll
  for (int v = 2; v < 16; v += 2) {
    m0 = __builtin_fmaxf(m0, __builtin_fmaxf(s0[v], s1[v]));
    m1 = __builtin_fmaxf(m1, __builtin_fmaxf(s0[v + 1], s1[v + 1]));
  }
  return swap_max(fmaxf(m0, m1));
}

// Move the reference max (and rescale O and l) when the tile's scaled max
// mxs exceeds it by more than kMargin: kLazy in the exact pass; 0 when a
// row takes its first reference.
// kG > 1: rows of one wavefront see different sub-tiles, so a lane can
// still hold mref = -inf (no key yet) when another grows: its factor is 1,
// not 2^(-inf - -inf).  At T >= 64 every row of a wavefront sees the same
// tiles and has a key from its first step on.
template <int kG = 1, bool kLazyRule = true>
__device__ __forceinline__ void rescale(RowState& st, float mxs) {
  const bool grow = kLazyRule ? mxs > st.mref + kLazy : mxs > st.mref;
  if (__builtin_amdgcn_ballot_w64(grow)) {
    const float mnew = grow ? mxs : st.mref;
    float alpha = __builtin_amdgcn_exp2f(st.mref - mnew);
    if constexpr (kG > 1) alpha = grow ? alpha : 1.f;
    st.mref = mnew;
    st.lsum *= alpha;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) st.o[db][v] *= alpha;
  }
}

__device__ __forceinline__ float exp_base(const RowState& st) {
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

// Rows without a reference take the row max of the next tile (scores s0,
// s1) before its weights are formed.  Such a row has seen no key, so its O
// and l are still 0 and nothing needs rescaling; rows that have a reference
// keep it.
template <int kG>
__device__ __forceinline__ void first_ref(RowState& rs, const f32x16& s0, const f32x16& s1,
                                          float c) {
  if (__builtin_amdgcn_ballot_w64(rs.mref == -INFINITY)) {
    const float mx = tile_max(s0, s1) * c;
    rs.mref = rs.mref == -INFINITY ? mx : rs.mref;
  }
}

__device__ __forceinline__ void pv_tile(const PvArgs& v, int slot_off, const bf16x8 (&pb)[4],
                                        RowState& st) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int db = 0; db < 4; ++db) st.o[db] = mfma(v_frag(v, slot_off, db, s), pb[s], st.o[db]);
}

// QK^T of the next tile and the softmax weights of the current one, by hand:
// k-step s issues its two MFMAs, the exponentials of four of the current
// tile's sixteen score pairs, and the K fragment reads of k-step s + 3, then
// a scheduling barrier keeps that order (three fragment pairs in flight).
__device__ __forceinline__ void qk_exp_pipelined(const QkArgs& q, int slot_off,
                                                 const bf16x8 (&qf)[8], f32x16& s0, f32x16& s1,
                                                 const f32x16& c0, const f32x16& c1, float c,
                                                 float base, bf16x8 (&pb)[4], float& lsum) {
  const bf16x2 ones = bf16x2{static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
  bf16x8 a0 = k_frag(q, slot_off, 0, 0), a1 = k_frag(q, slot_off, 1, 0);
  bf16x8 b0 = k_frag(q, slot_off, 0, 1), b1 = k_frag(q, slot_off, 1, 1);
  bf16x8 d0 = k_frag(q, slot_off, 0, 2), d1 = k_frag(q, slot_off, 1, 2);
  float psum = 0.f;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    s0 = mfma(a0, qf[s], s == 0 ? f32x16{} : s0);
    s1 = mfma(a1, qf[s], s == 0 ? f32x16{} : s1);
    const int st = s >> 1, e0 = (s & 1) * 4, v0 = 8 * (st & 1);
#pragma unroll
    for (int u = 0; u < 4; u += 2) {
      const float x0 = (st < 2) ? c0[v0 + e0 + u] : c1[v0 + e0 + u];
      const float x1 = (st < 2) ? c0[v0 + e0 + u + 1] : c1[v0 + e0 + u + 1];
      const float p0 = __builtin_amdgcn_exp2f(fmaf(x0, c, -base));
      const float p1 = __builtin_amdgcn_exp2f(fmaf(x1, c, -base));
      const bf16x2 pp = bf16x2{static_cast<__bf16>(p0), static_cast<__bf16>(p1)};
      pb[st][e0 + u] = pp[0];
      pb[st][e0 + u + 1] = pp[1];
      psum = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, psum, false);
    }
    a0 = b0;
    a1 = b1;
    b0 = d0;
    b1 = d1;
    if (s + 3 < 8) {
      d0 = k_frag(q, slot_off, 0, s + 3);
      d1 = k_frag(q, slot_off, 1, s + 3);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  lsum += psum;
}

// QK^T alone, the same way.
__device__ __forceinline__ void qk_pipelined(const QkArgs& q, int slot_off, const bf16x8 (&qf)[8],
                                             f32x16& s0, f32x16& s1) {
  bf16x8 a0 = k_frag(q, slot_off, 0, 0), a1 = k_frag(q, slot_off, 1, 0);
  bf16x8 b0 = k_frag(q, slot_off, 0, 1), b1 = k_frag(q, slot_off, 1, 1);
  bf16x8 d0 = k_frag(q, slot_off, 0, 2), d1 = k_frag(q, slot_off, 1, 2);
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    s0 = mfma(a0, qf[s], s == 0 ? f32x16{} : s0);
    s1 = mfma(a1, qf[s], s == 0 ? f32x16{} : s1);
    a0 = b0;
    a1 = b1;
    b0 = d0;
    b1 = d1;
    if (s + 3 < 8) {
      d0 = k_frag(q, slot_off, 0, s + 3);
      d1 = k_frag(q, slot_off, 1, s + 3);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Interleave QK^T of the next tile (16 LDS reads, 16 MFMAs) with the
// softmax exponentials of the current one, and PV of the current tile (32
// transpose reads, 16 MFMAs) with the row max of the next one.
__device__ __forceinline__ void interleave_qk_exp() {
  __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i < 14) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x402, 6, 0);
  }
}

__device__ __forceinline__ void interleave_pv_max() {
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i < 14) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x402, 2, 0);
  }
}

// PV with nothing to interleave: the transpose reads kept ahead.
__device__ __forceinline__ void pace_pv() {
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i < 14) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
}

// The same with nothing to interleave: keep the fragment reads two MFMAs
// ahead (an unconstrained schedule issues all of them first and runs out of
// registers).
__device__ __forceinline__ void pace_qk() {
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i < 12) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
}

// The attention kernel's arguments as one aggregate, so that their place in
// the kernel argument segment is fixed (the epilogue reads some of them from
// there again).
struct KernArgs {
  PlanTables pt;
  WorkTables wt;
  AttnArgs a;
};

// Merge the pieces of the split units.  Piece p left its normalised
// output O_p (fp32 output: fp32; bf16 output: a bf16 and the bf16 of its
// rounding error, 16 significant bits together), its reference max m_p
// (log2 domain) and its row sum l_p, relative to 2^m_p.  With M the largest
// m_p among pieces that saw keys and w_p = l_p 2^(m_p - M), a row's output
// is sum w_p O_p / sum w_p, rounded once to the output's type.  Block (s, y)
// takes rows 32y .. 32y + 31 of split unit s; thread t owns row 32y + t/8
// and head dims 16 (t%8) .. + 15.  Job j = 4 s + y.
template <bool kOutF32>
__device__ __forceinline__ void combine_job(const WorkTables& wt, const AttnArgs& a, int job) {
  using OutT = typename std::conditional<kOutF32, float, __bf16>::type;
  constexpr int kDims = 16;                         // per thread
  constexpr int kVec = 16 / sizeof(OutT);           // elements per 16-byte load
  const int4 sp = wt.splits[job >> 2];  // {record of the first piece, first slot, slots}
  const WorkRec* __restrict__ rp = wt.rec + sp.x;
  const int row = (job & 3) * 32 + (threadIdx.x >> 3);
  const int d0 = (threadIdx.x & 7) * kDims;
  const int blk = row >> 6;
  const int r = row & 63;
  if (r >= (blk == 0 ? rp->len[0] : rp->len[1])) return;
  const int tok = (blk == 0 ? rp->tok0[0] : rp->tok0[1]) + r;
  const int prow = tok & (kUnitRows - 1);  // the row's place in a slot
  const float2* ml = wt.part_ml + static_cast<int64_t>(sp.y) * kUnitRows + prow;
  float mx = -INFINITY;
#pragma unroll 4
  for (int p = 0; p < sp.z; ++p) {
    const float2 x = ml[static_cast<int64_t>(p) * kUnitRows];
    if (x.y > 0.f) mx = fmaxf(mx, x.x);
  }
  float acc[kDims];
#pragma unroll
  for (int j = 0; j < kDims; ++j) acc[j] = 0.f;
  float wsum = 0.f;
  const int64_t pbase = (static_cast<int64_t>(sp.y) * kUnitRows + prow) * kD + d0;
  const OutT* po = static_cast<const OutT*>(wt.part_o) + pbase;
  const __bf16* plo = static_cast<const __bf16*>(wt.part_lo) + pbase;  // bf16 output only
#pragma unroll 2
  for (int p = 0; p < sp.z; ++p) {
    const float2 x = ml[static_cast<int64_t>(p) * kUnitRows];
    const float w = x.y > 0.f ? x.y * __builtin_amdgcn_exp2f(x.x - mx) : 0.f;
    wsum += w;
    const OutT* src = po + static_cast<int64_t>(p) * kUnitRows * kD;
#pragma unroll
    for (int c = 0; c < kDims / kVec; ++c) {
      // (the elements of a loaded vector are read as themselves or by shifts:
      // a bit_cast of a vector element compiled to loads of element 0 only)
      if constexpr (kOutF32) {
        const f32x4 val = *reinterpret_cast<const f32x4*>(src + c * kVec);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[4 * c + e] += w * val[e];
      } else {
        const u32x4 raw = *reinterpret_cast<const u32x4*>(src + c * kVec);
        const u32x4 rlo = *reinterpret_cast<const u32x4*>(plo + static_cast<int64_t>(p) *
                                                                      kUnitRows * kD + c * kVec);
#pragma unroll
        for (int e = 0; e < 4; ++e) {  // bf16 -> f32 is exact: the high half of the word
          const unsigned u = raw[e], l = rlo[e];
          acc[8 * c + 2 * e] += w * (__builtin_bit_cast(float, u << 16) +
                                     __builtin_bit_cast(float, l << 16));
          acc[8 * c + 2 * e + 1] += w * (__builtin_bit_cast(float, u & 0xffff0000u) +
                                         __builtin_bit_cast(float, l & 0xffff0000u));
        }
      }
    }
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  OutT* dst = static_cast<OutT*>(a.out) + (static_cast<int64_t>(tok) * a.hq + rp->head) * kD + d0;
#pragma unroll
  for (int c = 0; c < kDims / kVec; ++c) {
    if constexpr (kOutF32) {
      *reinterpret_cast<f32x4*>(dst + c * kVec) =
          f32x4{acc[4 * c] * inv, acc[4 * c + 1] * inv, acc[4 * c + 2] * inv, acc[4 * c + 3] * inv};
    } else {
      u32x4 raw;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 y = bf16x2{static_cast<__bf16>(acc[8 * c + 2 * e] * inv),
                                static_cast<__bf16>(acc[8 * c + 2 * e + 1] * inv)};
        raw[e] = __builtin_bit_cast(unsigned, y);
      }
      *reinterpret_cast<u32x4*>(dst + c * kVec) = raw;
    }
  }
}

// kRedo = false: the first pass; workgroup b takes the unit of launch slot
// b and flags the launch (wt.redo[0]) if a weight check fails.  kRedo =
// true: the exact pass; when the flag is set, kRedoGrid workgroups do every
// unit again, then the last one to finish clears the flag for the next
// launch; otherwise they return at once.
template <bool kOutF32, int kG, bool kRedo>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(KernArgs ka) {
  const PlanTables& pt = ka.pt;
  const WorkTables& wt = ka.wt;
  const AttnArgs& a = ka.a;
  // K slot 0, K slot 1, V slot 0, V slot 1 (16 KB each)
  __shared__ __attribute__((aligned(1024))) __bf16 smem[4 * kTile];
  // the unit's partial-result slot, parked in LDS for the epilogue so that
  // no register is held across the main loop (every wavefront writes the
  // same value and reads back its own write)
  __shared__ int slot_park;

  if constexpr (!kRedo) {
    const int4* __restrict__ rp = reinterpret_cast<const int4*>(wt.launch + blockIdx.x);
#include "attn_bf16_unit.inc"
  } else {
    constexpr int kJobs = kUnitRows / 32;  // merge jobs per split unit
    const int jobs = wt.num_splits * kJobs;
    if (__hip_atomic_load(&wt.redo[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
      // the first pass stands: merge the pieces of the split units
      for (int j = blockIdx.x; j < jobs; j += gridDim.x) combine_job<kOutF32>(wt, a, j);
      return;
    }
    for (int u = blockIdx.x; u < wt.grid; u += gridDim.x) {
      auto unit = [&](const int4* __restrict__ rp) {
#include "attn_bf16_unit.inc"
      };
      unit(reinterpret_cast<const int4*>(wt.launch + u));
      __syncthreads();  // LDS (slots, slot_park) is reused by the next unit
    }
    if (threadIdx.x == 0) {
      __threadfence();
      slot_park = atomicAdd(&wt.redo[1], 1) == static_cast<int>(gridDim.x) - 1;
    }
    __syncthreads();
    if (slot_park) {
      // the last workgroup: every piece is written; merge them all, then
      // clear the flag for the next launch
      __threadfence();
      for (int j = 0; j < jobs; ++j) combine_job<kOutF32>(wt, a, j);
      if (threadIdx.x == 0) {
        atomicExch(&wt.redo[0], 0);
        atomicExch(&wt.redo[1], 0);
        atomicAdd(&wt.redo[2], 1);  // launches whose exact pass ran
      }
    }
  }
}

}  // namespace

hipError_t launch_attn_bf16(const PlanTables& pt, const WorkTables& wt, const AttnArgs& a,
                            hipStream_t stream) {
  // T = 128 tiles reach the kernel as 64-row blocks and 64-key steps, T = 16
  // and 32 tiles as groups of 4 and 2
  if ((a.tile != 16 && a.tile != 32 && a.tile != kT && a.tile != 2 * kT) || a.head_dim != kD)
    return hipErrorInvalidValue;
  if (wt.grid == 0) return hipSuccess;
  const int g = a.tile < kT ? kT / a.tile : 1;  // key tiles per 64-key step
  // the first pass over every unit, then the exact pass (which returns at
  // once unless the first raised its flag)
  auto launch = [&](auto out_f32, auto group) {
    constexpr bool kF = decltype(out_f32)::value;
    constexpr int kGr = decltype(group)::value;
    const KernArgs ka{pt, wt, a};
    hipLaunchKernelGGL((attn_bf16_kernel<kF, kGr, false>), dim3(wt.grid), dim3(256), 0, stream, ka);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_bf16_kernel<kF, kGr, true>), dim3(kRedoGrid), dim3(256), 0, stream,
                       ka);
    return hipGetLastError();
  };
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I4 = std::integral_constant<int, 4>;
  hipError_t e;
  if (a.out_f32)
    e = g == 4 ? launch(std::true_type{}, I4{})
               : g == 2 ? launch(std::true_type{}, I2{}) : launch(std::true_type{}, I1{});
  else
    e = g == 4 ? launch(std::false_type{}, I4{})
               : g == 2 ? launch(std::false_type{}, I2{}) : launch(std::false_type{}, I1{});
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace sift
