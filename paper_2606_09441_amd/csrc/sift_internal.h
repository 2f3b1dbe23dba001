// Internal interfaces between the host planner (sift_api.cpp) and the HIP
// kernels (decode.hip, attn_bf16.hip, attn_f32.hip).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sift {

enum SegKind : int32_t { kDocument = 0, kQuery = 1 };

// Device views of the plan tables (all int32, device memory).
struct PlanTables {
  // per segment s
  const int32_t* seg_tile0;   // global number of the segment's tile 0
  const int32_t* seg_pages;   // P_s
  const int32_t* seg_kind;    // SegKind
  const int32_t* seg_first;   // first segment of the segment's prompt
  const int32_t* seg_la_off;  // byte offset of the LA vector of query head 0
  const int32_t* seg_ca_off;  // byte offset of the CA vector of query head 0
  // per tile m
  const int32_t* tile_seg;    // segment of tile m
  const int32_t* tile_tok0;   // first token of tile m on the packed axis
  const int32_t* tile_len;    // tokens in tile m (T, or less for a last tile)
  const int32_t* tile_lo;     // first tile of m's prompt
  int32_t num_tiles;          // M
  int32_t num_q_heads;        // Hq
  int32_t tile;               // T
};

// Where the K/V rows of a key tile live.  Packed (table == nullptr): tile m
// starts at token row tile_tok0[m] of k and v.  Paged: k and v are a pool of
// num_pages pages of T rows each, and tile m is pool page table[m] (entries
// outside [0, num_pages) are clamped into the pool, so no access leaves it).
// Both layouts have the same row stride (Hkv * D elements).
struct KvPages {
  const int32_t* table;
  int32_t num_pages;
};

__device__ __forceinline__ int32_t kv_row0(const PlanTables& pt, const KvPages& pg, int32_t m) {
  if (pg.table == nullptr) return pt.tile_tok0[m];
  const int32_t p = pg.table[m];
  return (p < 0 ? 0 : (p >= pg.num_pages ? pg.num_pages - 1 : p)) * pt.tile;
}

// Attention work: a list unit = (query head, up to kUnitBlocks consecutive
// M-blocks of one segment).  The decode pass writes each list unit's merged
// step list (the union of its M-blocks' lists, in ascending key-tile order)
// at steps[lu_off[u] ..]; lu_off[u+1] - lu_off[u] bounds its length.
// Step = {first K/V row of the key tile, len | listed << 8 | diagonal << 12},
// where bit k of `listed` says M-block m0 + k lists the tile and bit k of
// `diagonal` says the tile is m0 + k itself.
//
// A workgroup runs one work unit: a list unit's whole step list, or one piece
// of it.  The query units, whose lists are long and of known length, are cut
// into pieces of at most a few dozen steps; a piece writes its partial result
// (O normalised by its own row sum, in the output's type; reference max; row
// sum) to a slot of the partial scratch, and a combine pass merges the pieces
// of every split unit into the output.
// List unit u owns work units lu_work0[u] .. + lu_nwork[u] - 1, piece k
// covering its steps [k * lu_len[u], (k + 1) * lu_len[u]); decode writes
// their step counts.
constexpr int kUnitBlocks = 2;
constexpr int kUnitRows = 64 * kUnitBlocks;  // query rows of a unit

struct WorkTables {
  // work units (attention)
  const int32_t* sched;       // [grid] work unit of each workgroup, or -1
  const int32_t* unit_head;   // [W]
  const int32_t* unit_m0;     // [W] first M-block
  const int32_t* unit_nb;     // [W] M-blocks, 1 .. kUnitBlocks
  const int32_t* step_off;    // [W] first step in steps
  int32_t* step_cnt;          // [W] steps (device scratch, written by decode)
  const int32_t* unit_slot;   // [W] partial slot, or -1: write the output
  // list units (decode)
  const int32_t* lu_head;     // [U]
  const int32_t* lu_m0;       // [U]
  const int32_t* lu_nb;       // [U]
  const int32_t* lu_off;      // [U + 1]
  const int32_t* lu_work0;    // [U]
  const int32_t* lu_nwork;    // [U]
  const int32_t* lu_len;      // [U] piece length (a bound of the list when not split)
  int2* steps;                // [lu_off[U]] (device scratch)
  const int4* splits;         // [NS] {first work unit, first slot, slots, 0}
  void* part_o;               // [slots][kUnitRows][head_dim], output type (device scratch)
  float2* part_ml;            // [slots][kUnitRows] {reference max, row sum}
  int32_t num_units;          // U
  int32_t num_work;           // W
  int32_t num_splits;         // NS
  int32_t grid;
};

// Step counts of a list unit's work units, from the length of its list.
__device__ __forceinline__ void write_work_counts(const WorkTables& wt, int32_t u, int32_t cnt) {
  const int32_t w0 = wt.lu_work0[u], nw = wt.lu_nwork[u], len = wt.lu_len[u];
  for (int32_t k = 0; k < nw; ++k) {
    const int32_t rest = cnt - k * len;
    wt.step_cnt[w0 + k] = rest < 0 ? 0 : (rest > len ? len : rest);
  }
}

constexpr int kStepLenMask = 0xff;
constexpr int kStepListedShift = 8;
constexpr int kStepDiagShift = 12;

// Decode (Section 5.1): count, scan, write.  The write pass runs per unit and
// emits its M-blocks' lists and the unit's merged step list.
hipError_t launch_decode(const PlanTables& pt, const WorkTables& wt, const uint8_t* la,
                         const uint8_t* ca, int32_t* counts, int32_t* row_ptr, int32_t* col_idx,
                         const KvPages& pages, hipStream_t stream);

// Merged step lists from caller-given per-M-block lists (entries outside
// [first tile of the prompt, M-block] skipped; lists ascending).
hipError_t launch_merge_steps(const PlanTables& pt, const WorkTables& wt, const int32_t* row_ptr,
                              const int32_t* col_idx, int64_t col_capacity, hipStream_t stream);

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  const int32_t* row_ptr;
  const int32_t* col_idx;
  int64_t col_capacity;
  int32_t hq, hkv, head_dim, tile;
  float scale_log2;           // softmax scale * log2(e)
  int32_t out_f32;            // 1: fp32 output, 0: bf16 output
  KvPages pages;              // K/V layout (table == nullptr: packed)
};

// bf16 attention reads the merged step lists of wt (not row_ptr/col_idx).
hipError_t launch_attn_bf16(const PlanTables& pt, const WorkTables& wt, const AttnArgs& a,
                            hipStream_t stream);
hipError_t launch_attn_f32(const PlanTables& pt, const AttnArgs& a, hipStream_t stream);

}  // namespace sift
