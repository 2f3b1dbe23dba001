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
};

// Attention work: one unit = (query head, a pair of consecutive M-blocks of
// one segment).  sched[g] is the unit run by workgroup g, or -1 for none.
struct WorkTables {
  const int32_t* sched;       // [grid]
  const int32_t* unit_head;   // [U]
  const int32_t* unit_m0;     // [U] first M-block
  const int32_t* unit_m1;     // [U] second M-block, or -1
  int32_t grid;
};

// Decode (Section 5.1): count, scan, write.
hipError_t launch_decode(const PlanTables& pt, const uint8_t* la, const uint8_t* ca,
                         int32_t* counts, int32_t* row_ptr, int32_t* col_idx,
                         hipStream_t stream);

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
};

hipError_t launch_attn_bf16(const PlanTables& pt, const WorkTables& wt, const AttnArgs& a,
                            hipStream_t stream);
hipError_t launch_attn_f32(const PlanTables& pt, const AttnArgs& a, hipStream_t stream);

}  // namespace sift
