// Internal interfaces between the host planner (sift_api.cpp) and the HIP
// kernels (decode.hip, attn_bf16.hip, attn_f32.hip).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
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
  const int4* tile_info;      // {tok0, len, byte offset of query head 0's CA byte holding the
                              // tile's bit (-1: a query tile), CA bytes per head << 3 | bit
                              // position in the byte}: what decode reads per candidate tile
  int32_t num_tiles;          // M
  int32_t num_segments;       // S
  int32_t num_q_heads;        // Hq
  int32_t tile;               // T
  int32_t halves;             // T = 128: 2 (each tile is two 64-row/64-key halves); else 1
  int32_t group;              // T < 64: 64 / T tiles per 64-row block and per step; else 1
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
// step list (the union of its M-blocks' lists) at steps[lu_off[u] ..];
// lu_off[u+1] - lu_off[u] bounds its length.
// Step = {first K/V row of the key tile, len | listed << 8 | diagonal << 12},
// where bit k of `listed` says M-block m0 + k lists the tile and bit k of
// `diagonal` says the tile is m0 + k itself.  At T < 64 a step is 64 keys of
// G = 64 / T tiles, bit b of `listed` / `diagonal` refers to kernel block b
// (M-blocks G b ..), the first word is the sub-tile mask (bit G k + s: M-block
// k lists the step's tile s) and kvb holds the tiles' K/V rows.  Steps run in
// ascending key order, except that a document unit's steps over the earlier
// documents gather G marked pages each, adjacent or not.
//
// A workgroup runs one work unit: a list unit's whole step list, or one piece
// of it.  The query units, whose lists are long and of known length, are cut
// into pieces of at most a few dozen steps; a piece writes its partial result
// (O normalised by its own row sum, in the output's type; reference max; row
// sum) to a slot of the partial scratch, and a combine pass merges the pieces
// of every split unit into the output.
// List unit u owns work units lu_work0[u] .. + lu_nwork[u] - 1, piece k
// covering its steps [k * lu_len[u], (k + 1) * lu_len[u]).
//
// Every work unit has a 64-byte record that holds all a workgroup needs
// before its first K/V fetch, so the kernel's start is one scalar load deep.
// rec[w] (work units in locality order) is the planner's static part plus
// the step count and first kFirstSteps steps, written by decode (for a split
// unit, once its whole list is written).
//
// Launch order.  Workgroups are dealt round-robin over the kNumXcd XCDs, so
// workgroup x + kNumXcd * k runs on XCD x.  The locality order is cut into
// kNumXcd chunks of chunk_size work units (w / chunk_size), chunk x for XCD
// x, so that the query heads sharing key tiles share an L2.  Inside a chunk
// the work units run in order of decreasing step count: the long ones start
// first and the short ones fill the end.  Decode ends with a schedule pass
// that copies each record to launch[x + kNumXcd * k], k its place in that
// order (launch slots past a chunk's end hold an empty record: one M-block
// of no rows, no steps).  The order is a counting sort: decode counts the
// work units of each (chunk, step count) bucket in hist[], keeping each
// unit's place in its bucket (rank); the schedule pass, sched_blocks blocks
// per chunk, scans the chunk's buckets and copies every work unit to its
// bucket's offset plus its rank; the chunk's last block clears the buckets.
constexpr int kNumXcd = 8;  // MI355X
constexpr int kUnitBlocks = 2;                 // 64-row kernel blocks of a unit
constexpr int kUnitRows = 64 * kUnitBlocks;  // query rows of a unit
constexpr int kMaxListBlocks = 8;            // M-blocks of a list unit: 128 / T, at most 8 (T = 16)
constexpr int kFirstSteps = 3;
constexpr int kSchedBuckets = 1024;          // step counts >= 1023 share bucket 0
constexpr int kSchedPerBlock = 1024;         // work units per schedule block (at most 8
                                             // blocks per chunk)

// Bucket of a step count: decreasing counts in increasing bucket order.
__device__ __forceinline__ int32_t sched_bucket(int32_t cnt) {
  return cnt >= kSchedBuckets - 1 ? 0 : kSchedBuckets - 1 - cnt;
}

struct alignas(64) WorkRec {
  int32_t head;      // query head
  int32_t kv_head;   // its K/V head
  int32_t rank;      // place among the work units of its (chunk, step-count bucket), in
                     // the order decode counted them (written by decode)
  int32_t slot;      // partial slot, or -1: write the output
  int32_t tok0[kUnitBlocks];  // first token of each M-block (0 when absent)
  int32_t len[kUnitBlocks];   // tokens of each M-block (0 when absent)
  int32_t step_off;  // first step in steps
  int32_t step_cnt;  // steps (written by decode)
  int2 first[kFirstSteps];    // steps 0 .. kFirstSteps - 1 (written by decode; those past
                              // step_cnt are stale)
};
static_assert(sizeof(WorkRec) == 64, "one record per 64 bytes");
static_assert(offsetof(WorkRec, step_cnt) == 36, "the step count is word 9 (read as int4 2, .y)");
static_assert(offsetof(WorkRec, rank) == 8, "the rank is word 2 (read as int4 0, .z)");

// A list unit, or a part of one, as the decode write pass reads it (one
// record, built with the plan): the pass takes them in record order, longest
// walk first.  At T < 64 a query unit's walk over its prompt is cut into
// parts of whole segments: its lists are every tile of the prompt up to the
// M-block, so where a part's entries and steps start is known in advance.
struct alignas(64) UnitRec {
  int32_t head, m0, nb, seg;  // query head, first M-block, M-blocks, their segment
  int32_t lo;                 // first tile of the prompt
  int32_t sd0;                // first tile of the segment
  int32_t pages;              // the segment's pages
  int32_t la_off;             // its LA vectors' byte offset (head 0)
  int32_t step_off;           // first step of the unit's merged list (lu_off)
  int32_t work0, nwork, plen;  // its work units: nwork pieces of plen steps from work0
  int32_t flags;              // kUnitQuery | hrows << 1 (T = 128: kernel blocks of the
                              // M-block, 3 or 1) | kUnitFirstPart | kUnitLastPart
  int32_t part_d0, part_d1;   // T < 64 query unit: the part's segments [d0, d1)
  int32_t part_skip;          // steps of the unit before the part
};
static_assert(sizeof(UnitRec) == 64, "one record per 64 bytes");
constexpr int32_t kUnitQuery = 1;
constexpr int32_t kUnitFirstPart = 8;  // writes the rows' row_ptr
constexpr int32_t kUnitLastPart = 16;  // writes the work units' step counts

struct WorkTables {
  WorkRec* rec;               // [W] locality order (device memory)
  WorkRec* launch;            // [grid] launch order (device scratch, written by the schedule pass)
  int32_t* hist;              // [kNumXcd * kSchedBuckets] bucket sizes (device scratch, zero
                              // between decodes)
  // list units (decode)
  const int32_t* lu_head;     // [U]
  const int32_t* lu_m0;       // [U]
  const int32_t* lu_nb;       // [U]
  const int32_t* lu_off;      // [U + 1]
  const int32_t* lu_work0;    // [U]
  const int32_t* lu_nwork;    // [U]
  const int32_t* lu_len;      // [U] piece length (a bound of the list when not split)
  const UnitRec* urec;        // [U] the list units in decode write order
  int2* steps;                // [lu_off[U]] (device scratch)
  int4* kvb;                  // [lu_off[U]] per step, T < 64 only: word q = the first K/V row
                              // of the step's key sub-tile q minus q T (the step's 64 keys
                              // are G tiles, not always adjacent ones; words past the
                              // step's tiles repeat a valid one) (device scratch)
  const int4* splits;         // [NS] {record of the first piece, first slot, slots, 0}
  void* part_o;               // [slots][kUnitRows][head_dim], output type (device scratch)
  void* part_lo;              // bf16 output: the same shape, part_o's bf16 rounding error
  float2* part_ml;            // [slots][kUnitRows] {reference max, row sum}
  int32_t* seg_base;          // [Hq * S] decode: each (head, segment)'s rows' list total,
                              // then their first list entry (device scratch)
  int32_t* decode_done;       // decode: finished count blocks (device scratch, zero between
                              // decodes)
  int32_t* head_tot;          // [Hq] decode: each query head's list entries (device scratch)
  uint8_t* ca_mark;           // [Hq * M] decode: per (head, tile) 1 when a document tile's
                              // page is CA-marked, else 0; written by the per-(head, segment)
                              // count, whose write pass walks every page (device scratch)
  int32_t* seg_cross;         // [Hq * S] decode: CA-marked pages of the earlier documents
                              // of each segment's prompt (device scratch)
  int32_t* cross_col;         // [Hq * M] decode: per head, each prompt's CA-marked tiles in
                              // tile order from its first tile's index on; nullptr when the
                              // count pass does not build them (device scratch)
  int2* cross_rows;           // [Hq * M] the same tiles' {first K/V row, length}
  int32_t* sched_done;        // [kNumXcd] schedule: finished blocks per chunk (device
                              // scratch, zero between decodes)
  int32_t* redo;              // [3] bf16 attention: {flag: do every unit again exactly,
                              // finished workgroups of that pass (both zero between
                              // launches), launches whose exact pass ran (a count kept
                              // for the plan's life)} (device scratch)
  int32_t num_units;          // U
  int32_t num_urec;           // records of the decode write pass (units and parts)
  int32_t num_work;           // W
  int32_t num_splits;         // NS
  int32_t chunk_size;         // work units per XCD chunk
  int32_t sched_blocks;       // schedule blocks per chunk
  int32_t grid;               // kNumXcd * chunk_size
};

// Step counts of a list unit's work units w0 .. w0 + nw - 1 (pieces of len
// steps), from the length of its list, counted in their schedule buckets.
// Thread `part` of `parts` takes pieces part, part + parts, ...
__device__ __forceinline__ void write_work_counts(const WorkTables& wt, int32_t w0, int32_t nw,
                                                  int32_t len, int32_t cnt, int part, int parts) {
  for (int32_t k = part; k < nw; k += parts) {
    const int32_t rest = cnt - k * len;
    const int32_t c = rest < 0 ? 0 : (rest > len ? len : rest);
    wt.rec[w0 + k].step_cnt = c;
    const int32_t x = (w0 + k) / wt.chunk_size;
    wt.rec[w0 + k].rank = atomicAdd(&wt.hist[x * kSchedBuckets + sched_bucket(c)], 1);
  }
}

constexpr int kStepLenMask = 0xff;
constexpr int kStepListedShift = 8;
constexpr int kStepDiagShift = 12;

// The steps (64-key blocks of the bf16 kernel) of key tile n for the list
// unit of M-blocks m0 .. m0 + nb - 1, which list it as `listed` says (bit k:
// M-block m0 + k).  Bit b of a step's listed / diagonal fields refers to the
// unit's 64-row kernel block b.  T <= 64: one step, kernel blocks are the
// M-blocks.  T = 128 (halves == 2, nb == 1): the M-block is two kernel
// blocks and the tile up to two steps of 64 keys; on the diagonal tile the
// first key half is the first row half's diagonal and precedes the second
// row half entirely, the second key half is the second row half's diagonal.
struct TileSteps {
  int cnt;
  int2 s[2];
};

__device__ __forceinline__ TileSteps tile_steps_at(const PlanTables& pt, int32_t n, unsigned listed,
                                                   int32_t m0, int32_t nb, int32_t row0,
                                                   int32_t len, unsigned rows) {
  TileSteps t;
  t.cnt = 0;
  if (listed == 0u) return t;
  if (pt.halves == 1) {
    const unsigned diag = (n >= m0 && n < m0 + nb) ? 1u << (n - m0) : 0u;
    t.cnt = 1;
    t.s[0] = make_int2(row0, len | static_cast<int>(listed << kStepListedShift) |
                                 static_cast<int>(diag << kStepDiagShift));
    return t;
  }
  const unsigned d0 = n == m0 ? 1u : 0u;
  t.cnt = len > 64 ? 2 : 1;
  t.s[0] = make_int2(row0, min(len, 64) | static_cast<int>(rows << kStepListedShift) |
                               static_cast<int>(d0 << kStepDiagShift));
  if (len > 64) {
    const unsigned r1 = n == m0 ? 2u : rows;
    t.s[1] = make_int2(row0 + 64, (len - 64) | static_cast<int>(r1 << kStepListedShift) |
                                      static_cast<int>((d0 << 1) << kStepDiagShift));
  }
  return t;
}

__device__ __forceinline__ TileSteps tile_steps(const PlanTables& pt, const KvPages& pg, int32_t n,
                                                unsigned listed, int32_t m0, int32_t nb) {
  if (listed == 0u) return TileSteps{0, {}};
  const unsigned rows = pt.tile_len[m0] > 64 ? 3u : 1u;  // kernel blocks of the M-block
  return tile_steps_at(pt, n, listed, m0, nb, kv_row0(pt, pg, n), pt.tile_len[n], rows);
}

// Decode (Section 5.1): count, write, schedule.  The count pass gives each
// row its offset inside its head and each head its total (or, for layouts of
// more than 1024 segments, offsets inside and totals of each (head,
// segment)), and the heads' cross lists; the write pass runs per unit,
// writes its rows' row_ptr, its M-blocks' lists and the unit's merged step
// list; the schedule pass orders the work units for the attention launch.
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

// Offline extraction (extract.hip).  One record per document; the bit-vector
// offsets are those of the online path's buffers (document-major, query heads
// inside), the flag and count offsets index the extraction workspace.
struct ExtractDoc {
  int32_t tok0;      // first token on the packed axis
  int32_t len;       // tokens
  int32_t P;         // pages, ceil(len / T)
  int32_t pad;
  int64_t la_off;    // byte offset of head 0's LA vector
  int64_t ca_off;    // byte offset of head 0's CA vector
  int64_t flag_off;  // first tile flag (bytes, Hq * P(P+1)/2 per document)
  int64_t cnt_off;   // first page count (int32, Hq * P per document)
};

struct ExtractArgs {
  const ExtractDoc* docs;
  const int2* blocks;       // {document, 128-row query block}, longest first
  const __bf16* q;          // [tokens][hq][D]
  const __bf16* k;          // [tokens][hkv][D]
  uint8_t* flags;
  int32_t* counts;
  int32_t hq, hkv;
  float c;                  // softmax scale * log2(e)
  float log2_alpha, log2_beta;
  double gamma;
};

// Zeroes zero_words_n words at zero_base (the flags and counts), runs the
// extraction over num_blocks query blocks x hq heads, then packs the bits.
hipError_t launch_extract(const ExtractArgs& a, int32_t num_docs, int32_t num_blocks,
                          int32_t head_dim, int32_t tile, uint32_t* zero_base, int64_t zero_words_n,
                          uint8_t* la, uint8_t* ca, hipStream_t stream);

// Rotary position embedding of q [tokens][hq][D] and k [tokens][hkv][D]
// (bf16, in place), angle = positions[t] * inv_freq[i] (rope.hip).
hipError_t launch_rope(void* q, int64_t tokens, int hq, void* k, int hkv, int head_dim,
                       const int32_t* positions, const float* inv_freq, hipStream_t stream);

}  // namespace sift
