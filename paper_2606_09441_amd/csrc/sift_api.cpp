// Host side of libsift: argument checks, the plan (tables derived from the
// prompt layout, Sections 4.3 and 5.1), the attention schedule, and the
// C ABI declared in include/sift.h.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <mutex>
#include <new>
#include <numeric>
#include <vector>

#include "sift.h"
#include "sift_internal.h"

namespace {


int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t la_nbytes(int64_t P) { return ceil_div(P * (P + 1), 16); }  // Section 4.3
int64_t ca_nbytes(int64_t P) { return ceil_div(P, 8); }             // Section 4.3

}  // namespace

struct sift_plan {
  int device = 0;
  sift_plan_info info{};
  // one device allocation holds every table, then the decode scratch
  void* dev = nullptr;
  size_t dev_bytes = 0;
  bool owns_dev = true;  // false: the caller's workspace (sift_sparse_prefill_ex)
  sift::PlanTables pt{};
  sift::WorkTables wt{};
  int32_t* counts = nullptr;   // [num_rows]
  int32_t* row_ptr = nullptr;  // [num_rows + 1]
  int32_t* col_idx = nullptr;  // [list_capacity]
  bool steps_paged = false;    // the last decode wrote page-pool rows into the steps
  hipStream_t last_stream = nullptr;  // the stream of the plan's last enqueued work
};

namespace {
// Everything an attention launch needs from the plan.
sift::WorkTables work(const sift_plan* p) { return p->wt; }
}  // namespace

namespace {

sift_status check_tensor(const sift_tensor* t, int32_t tokens, int32_t heads, int32_t dim) {
  if (t == nullptr) return SIFT_E_NULL;
  if (t->data == nullptr && static_cast<int64_t>(t->tokens) * t->heads * t->head_dim > 0)
    return SIFT_E_NULL;
  if (t->dtype != SIFT_F32 && t->dtype != SIFT_BF16) return SIFT_E_UNSUPPORTED;
  if (t->tokens != tokens || t->heads != heads || t->head_dim != dim) return SIFT_E_SHAPE;
  return SIFT_OK;
}

sift_status check_device(const sift_plan* plan) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SIFT_E_HIP;
  return dev == plan->device ? SIFT_OK : SIFT_E_PLAN;
}

// Shapes and dtypes of one call against the plan's sizes.
sift_status check_io(const sift_tensor* q, const sift_tensor* k, const sift_tensor* v,
                     const sift_tensor* out, int32_t tokens, int32_t hq, int32_t hkv, int32_t dim,
                     int32_t tile) {
  sift_status st;
  if ((st = check_tensor(q, tokens, hq, dim)) != SIFT_OK) return st;
  if ((st = check_tensor(k, tokens, hkv, dim)) != SIFT_OK) return st;
  if ((st = check_tensor(v, tokens, hkv, dim)) != SIFT_OK) return st;
  if ((st = check_tensor(out, tokens, hq, dim)) != SIFT_OK) return st;
  if (q->dtype != k->dtype || q->dtype != v->dtype) return SIFT_E_UNSUPPORTED;
  if (q->dtype == SIFT_BF16 && dim != 128) return SIFT_E_UNSUPPORTED;
  if (q->dtype == SIFT_F32 && (out->dtype != SIFT_F32 || tile > 64)) return SIFT_E_UNSUPPORTED;
  return SIFT_OK;
}

// Host tables of a validated layout.
struct HostPlan {
  std::vector<int32_t> seg_tile0, seg_pages, seg_kind, seg_first, seg_la_off, seg_ca_off;
  std::vector<int32_t> tile_seg, tile_tok0, tile_len, tile_lo;
  std::vector<int32_t> tile_info;  // int4 per tile (see PlanTables::tile_info)
  std::vector<int32_t> unit_head, unit_m0, unit_nb, step_off;  // list units
  std::vector<int32_t> lu_work0, lu_nwork, lu_len;
  std::vector<sift::UnitRec> urec;  // list units by descending cost (the decode write order)
  std::vector<int32_t> wk_head, wk_m0, wk_nb, wk_off, wk_slot;        // work units
  std::vector<int32_t> splits;  // int4 records (see WorkTables)
  std::vector<sift::WorkRec> rec;     // work units in locality order
  std::vector<sift::WorkRec> launch;  // launch slots, initially empty
  int64_t chunk_size = 0;
  int64_t part_slots = 0;
  int64_t dense_tiles = 0;  // causal tiles of all prompts, one head
  int64_t la_bytes = 0, ca_bytes = 0;
  int32_t num_tokens = 0, num_segments = 0, num_tiles = 0;
};

sift_status build_host_plan(const sift_layout* lay, int32_t hq, int32_t hkv, int32_t tile,
                            HostPlan& hp) {
  if (lay->num_prompts < 1) return SIFT_E_LAYOUT;
  if (lay->prompt_seg_ptr == nullptr || lay->seg_offsets == nullptr) return SIFT_E_NULL;
  const int32_t B = lay->num_prompts;
  const int32_t* psp = lay->prompt_seg_ptr;
  const int32_t* so = lay->seg_offsets;
  if (psp[0] != 0) return SIFT_E_LAYOUT;
  for (int32_t b = 0; b < B; ++b)
    if (psp[b + 1] <= psp[b]) return SIFT_E_LAYOUT;  // every prompt has its query segment
  const int32_t S = psp[B];
  if (so[0] != 0) return SIFT_E_LAYOUT;
  for (int32_t s = 0; s < S; ++s)
    if (so[s + 1] < so[s]) return SIFT_E_LAYOUT;
  hp.num_segments = S;
  hp.num_tokens = so[S];
  hp.seg_tile0.resize(S);
  hp.seg_pages.resize(S);
  hp.seg_kind.resize(S);
  hp.seg_first.resize(S);
  hp.seg_la_off.resize(S);
  hp.seg_ca_off.resize(S);
  int64_t tiles = 0, la_off = 0, ca_off = 0, dense = 0;
  const int64_t i32max = std::numeric_limits<int32_t>::max();
  for (int32_t b = 0; b < B; ++b) {
    const int64_t lo = tiles;
    for (int32_t s = psp[b]; s < psp[b + 1]; ++s) {
      const bool is_query = s == psp[b + 1] - 1;
      const int64_t len = static_cast<int64_t>(so[s + 1]) - so[s];
      if (!is_query && len < 1) return SIFT_E_LAYOUT;  // documents are not empty
      const int64_t P = ceil_div(len, tile);
      hp.seg_tile0[s] = static_cast<int32_t>(tiles);
      hp.seg_pages[s] = static_cast<int32_t>(P);
      hp.seg_kind[s] = is_query ? sift::kQuery : sift::kDocument;
      hp.seg_first[s] = psp[b];
      hp.seg_la_off[s] = static_cast<int32_t>(la_off);
      hp.seg_ca_off[s] = static_cast<int32_t>(ca_off);
      if (!is_query) {
        la_off += hq * la_nbytes(P);
        ca_off += hq * ca_nbytes(P);
        if (la_off > i32max || ca_off > i32max) return SIFT_E_CAPACITY;
      }
      // causal tiles of rows i = 0..P-1 of this segment: (tiles - lo) + i + 1
      dense += P * (tiles - lo) + P * (P + 1) / 2;
      tiles += P;
      if (tiles > i32max) return SIFT_E_CAPACITY;
    }
  }
  hp.num_tiles = static_cast<int32_t>(tiles);
  hp.la_bytes = la_off;
  hp.ca_bytes = ca_off;
  hp.dense_tiles = dense;
  if (dense * hq >= i32max) return SIFT_E_CAPACITY;  // int32 list offsets
  if (static_cast<int64_t>(tiles) * hq >= i32max) return SIFT_E_CAPACITY;

  hp.tile_seg.resize(tiles);
  hp.tile_tok0.resize(tiles);
  hp.tile_len.resize(tiles);
  hp.tile_lo.resize(tiles);
  hp.tile_info.resize(4 * tiles);
  for (int32_t b = 0; b < B; ++b) {
    const int32_t lo = hp.seg_tile0[psp[b]];
    for (int32_t s = psp[b]; s < psp[b + 1]; ++s) {
      const bool doc = hp.seg_kind[s] == sift::kDocument;
      const int32_t P = hp.seg_pages[s];
      for (int32_t i = 0; i < P; ++i) {
        const int32_t m = hp.seg_tile0[s] + i;
        hp.tile_seg[m] = s;
        hp.tile_tok0[m] = so[s] + i * tile;
        hp.tile_len[m] = std::min<int32_t>(tile, so[s + 1] - (so[s] + i * tile));
        hp.tile_lo[m] = lo;
        int32_t* ti = &hp.tile_info[4 * static_cast<int64_t>(m)];
        ti[0] = hp.tile_tok0[m];
        ti[1] = hp.tile_len[m];
        ti[2] = doc ? hp.seg_ca_off[s] + (i >> 3) : -1;
        ti[3] = doc ? static_cast<int32_t>(ca_nbytes(P) << 3) | (i & 7) : 0;
      }
    }
  }

  // Attention work units: (query head, M-blocks ub*p .. of a segment).  The
  // M-blocks of one document share the cross-attention part of their lists
  // (it depends on the key document only), so a unit stages each of those
  // key tiles once for all of its query rows.  The bf16 kernel works on
  // units of two 64-row blocks: 128 / T M-blocks of T <= 64 per unit (G =
  // 64 / T of them per kernel block), or one M-block of T = 128 (two halves,
  // each tile up to two steps).
  const int32_t halves = tile == 128 ? 2 : 1;
  const int32_t ub = tile == 128 ? 1 : sift::kUnitRows / tile;
  const int32_t G = tile < 64 ? 64 / tile : 1;
  struct Group {
    int32_t m0, nb;
    int64_t cost;  // causal tiles of the group's last M-block: the union's length bound
  };
  std::vector<Group> groups;
  for (int32_t s = 0; s < S; ++s) {
    const int32_t lo = hp.seg_tile0[hp.seg_first[s]];  // first tile of the prompt
    for (int32_t p = 0; p < hp.seg_pages[s]; p += ub) {
      const int32_t m0 = hp.seg_tile0[s] + p;
      const int32_t nb = std::min<int32_t>(ub, hp.seg_pages[s] - p);
      groups.push_back({m0, nb, (m0 + nb - 1 - lo + 1) * halves});
    }
  }
  // Units in locality order: kv head, then longest group first, then the
  // query heads of the kv group side by side (they read the same key tiles).
  const int32_t g = hq / hkv;
  std::vector<int32_t> gord(groups.size());
  std::iota(gord.begin(), gord.end(), 0);
  std::stable_sort(gord.begin(), gord.end(),
                   [&](int32_t x, int32_t y) { return groups[x].cost > groups[y].cost; });
  const int64_t U = static_cast<int64_t>(groups.size()) * hq;
  if (U > i32max / 2) return SIFT_E_CAPACITY;
  std::vector<int32_t> order;  // unit ids
  order.reserve(U);
  hp.unit_head.resize(U);
  hp.unit_m0.resize(U);
  hp.unit_nb.resize(U);
  std::vector<int64_t> unit_cost(U);
  int32_t u = 0;
  for (int32_t kv = 0; kv < hkv; ++kv)
    for (int32_t gi : gord)
      for (int32_t j = 0; j < g; ++j) {
        hp.unit_head[u] = kv * g + j;
        hp.unit_m0[u] = groups[gi].m0;
        hp.unit_nb[u] = groups[gi].nb;
        unit_cost[u] = groups[gi].cost;
        order.push_back(u);
        ++u;
      }
  // A unit's merged list is a subset of the tiles from the prompt's first
  // to its last M-block.
  hp.step_off.assign(U + 1, 0);
  for (int64_t k = 0; k < U; ++k) {
    if (hp.step_off[k] + unit_cost[k] > i32max) return SIFT_E_CAPACITY;
    hp.step_off[k + 1] = hp.step_off[k] + static_cast<int32_t>(unit_cost[k]);
  }
  // Work units.  A query unit lists every tile of its prompt up to its last
  // M-block, so its list length is its cost.  The launch runs the longest
  // work units first (see WorkRec), so a unit only delays the end when it is
  // longer than the work per workgroup slot; a query unit is cut into pieces
  // of at most `piece` steps, piece = that work's lower bound (the query
  // units' steps plus one diagonal step per document M-block, over
  // kSlots resident workgroups), at least kMinPiece.  The piece length
  // doubles until at most kMaxSlots partial slots are needed.
  constexpr int64_t kMaxSlots = 4096;
  constexpr int64_t kMinPiece = 32;
  constexpr int64_t kSlots = 512;  // 256 CUs x 2 resident attention workgroups
  auto is_query = [&](int64_t k) { return hp.seg_kind[hp.tile_seg[hp.unit_m0[k]]] == sift::kQuery; };
  int64_t lower = 0;
  for (int64_t k = 0; k < U; ++k) lower += is_query(k) ? unit_cost[k] : hp.unit_nb[k];
  int64_t piece = std::max<int64_t>(kMinPiece, (lower + kSlots - 1) / kSlots);
  auto slots_for = [&](int64_t pc) {
    int64_t n = 0;
    for (int64_t k = 0; k < U; ++k)
      if (is_query(k) && unit_cost[k] > pc) n += (unit_cost[k] + pc - 1) / pc;
    return n;
  };
  while (slots_for(piece) > kMaxSlots) piece *= 2;
  hp.lu_work0.assign(U, 0);
  hp.lu_nwork.assign(U, 1);
  hp.lu_len.assign(U, 0);
  int64_t W = 0;
  for (int32_t uu : order) {
    const int64_t cost = unit_cost[uu];
    const int64_t parts = is_query(uu) && cost > piece ? (cost + piece - 1) / piece : 1;
    const int64_t len = (cost + parts - 1) / parts;
    hp.lu_work0[uu] = static_cast<int32_t>(hp.wk_head.size());
    hp.lu_nwork[uu] = static_cast<int32_t>(parts);
    hp.lu_len[uu] = static_cast<int32_t>(len);
    if (parts > 1)
      hp.splits.insert(hp.splits.end(), {static_cast<int32_t>(hp.wk_head.size()),
                                         static_cast<int32_t>(hp.part_slots),
                                         static_cast<int32_t>(parts), 0});
    for (int64_t i = 0; i < parts; ++i) {
      ++W;
      hp.wk_head.push_back(hp.unit_head[uu]);
      hp.wk_m0.push_back(hp.unit_m0[uu]);
      hp.wk_nb.push_back(hp.unit_nb[uu]);
      hp.wk_off.push_back(static_cast<int32_t>(hp.step_off[uu] + i * len));
      hp.wk_slot.push_back(parts > 1 ? static_cast<int32_t>(hp.part_slots + i) : -1);
    }
    if (parts > 1) hp.part_slots += parts;
  }
  if (W > i32max / 2) return SIFT_E_CAPACITY;
  // Records of the decode write pass: one per unit, except that at T < 64 a
  // query unit's walk (segment by segment over its prompt, in steps of G
  // adjacent tiles) is cut into parts of whole segments of about kPartTiles
  // tiles, one wavefront each.  They run longest walk first over all heads,
  // so that no long walk starts late.
  constexpr int64_t kPartTiles = 256;
  std::vector<int64_t> rcost;
  for (int64_t uu = 0; uu < U; ++uu) {
    const int32_t m0 = hp.unit_m0[uu], sg = hp.tile_seg[m0];
    const bool query = hp.seg_kind[sg] == sift::kQuery;
    sift::UnitRec r{};
    r.head = hp.unit_head[uu];
    r.m0 = m0;
    r.nb = hp.unit_nb[uu];
    r.seg = sg;
    r.lo = hp.tile_lo[m0];
    r.sd0 = hp.seg_tile0[sg];
    r.pages = hp.seg_pages[sg];
    r.la_off = hp.seg_la_off[sg];
    r.step_off = hp.step_off[uu];
    r.work0 = hp.lu_work0[uu];
    r.nwork = hp.lu_nwork[uu];
    r.plen = hp.lu_len[uu];
    r.flags = (query ? sift::kUnitQuery : 0) | ((hp.tile_len[m0] > 64 ? 3 : 1) << 1);
    r.part_d0 = hp.seg_first[sg];
    r.part_d1 = sg + 1;
    r.part_skip = 0;
    if (!(query && G > 1)) {
      r.flags |= sift::kUnitFirstPart | sift::kUnitLastPart;
      hp.urec.push_back(r);
      rcost.push_back(unit_cost[uu]);
      continue;
    }
    // segment d's tiles walked by the unit, and its steps (groups of G)
    const int32_t mlast = m0 + r.nb - 1;
    auto tiles = [&](int32_t d) { return d < sg ? hp.seg_pages[d] : mlast - hp.seg_tile0[sg] + 1; };
    int32_t skip = 0;
    for (int32_t d0 = r.part_d0; d0 <= sg;) {
      int32_t d1 = d0;
      int64_t t = 0, g = 0;
      while (d1 <= sg && (d1 == d0 || t + tiles(d1) <= kPartTiles)) {
        t += tiles(d1);
        g += (tiles(d1) + G - 1) / G;
        ++d1;
      }
      sift::UnitRec p = r;
      p.part_d0 = d0;
      p.part_d1 = d1;
      p.part_skip = skip;
      if (d0 == r.part_d0) p.flags |= sift::kUnitFirstPart;
      if (d1 == sg + 1) p.flags |= sift::kUnitLastPart;
      hp.urec.push_back(p);
      rcost.push_back(t);
      skip += static_cast<int32_t>(g);
      d0 = d1;
    }
  }
  {
    std::vector<int32_t> ro(hp.urec.size());
    std::iota(ro.begin(), ro.end(), 0);
    std::stable_sort(ro.begin(), ro.end(), [&](int32_t x, int32_t y) { return rcost[x] > rcost[y]; });
    std::vector<sift::UnitRec> sorted(hp.urec.size());
    for (size_t q = 0; q < ro.size(); ++q) sorted[q] = hp.urec[ro[q]];
    hp.urec.swap(sorted);
  }
  if (hp.urec.size() > static_cast<size_t>(i32max / 2)) return SIFT_E_CAPACITY;
  // Work-unit records in locality order (work unit w is record w); the
  // launch order is made on the device after each decode, from the step
  // counts.
  hp.rec.assign(W, sift::WorkRec{});
  for (int64_t w = 0; w < W; ++w) {
    sift::WorkRec& r = hp.rec[w];
    r.head = hp.wk_head[w];
    r.kv_head = hp.wk_head[w] / (hq / hkv);
    r.slot = hp.wk_slot[w];
    if (halves == 1) {
      // kernel block b: M-blocks m0 + G b .. m0 + G b + G - 1 of the unit
      const int32_t m0 = hp.wk_m0[w], nb = hp.wk_nb[w];
      const int32_t blocks = (nb + G - 1) / G;
      for (int b = 0; b < blocks; ++b) {
        r.tok0[b] = hp.tile_tok0[m0 + G * b];
        r.len[b] = 0;
        for (int32_t m = m0 + G * b; m < std::min(m0 + nb, m0 + G * b + G); ++m)
          r.len[b] += hp.tile_len[m];
      }
    } else {  // one M-block of T = 128: two kernel blocks of 64 rows
      const int32_t m = hp.wk_m0[w], len = hp.tile_len[m];
      r.tok0[0] = hp.tile_tok0[m];
      r.len[0] = std::min<int32_t>(len, 64);
      r.tok0[1] = len > 64 ? hp.tile_tok0[m] + 64 : 0;
      r.len[1] = len > 64 ? len - 64 : 0;
    }
    r.step_off = hp.wk_off[w];
  }
  // launch slots start empty (one M-block of no rows, no steps); the
  // schedule pass fills those of the work units
  hp.chunk_size = (W + sift::kNumXcd - 1) / sift::kNumXcd;
  sift::WorkRec empty{};
  empty.slot = -1;
  hp.launch.assign(hp.chunk_size * sift::kNumXcd, empty);
  return SIFT_OK;
}

template <class T>
size_t put(std::vector<uint8_t>& blob, const std::vector<T>& v) {
  const size_t off = (blob.size() + 255) & ~size_t(255);
  blob.resize(off + v.size() * sizeof(T));
  if (!v.empty()) std::memcpy(blob.data() + off, v.data(), v.size() * sizeof(T));
  return off;
}

}  // namespace

extern "C" {

const char* sift_status_string(int32_t status) {
  switch (status) {
    case SIFT_OK: return "ok";
    case SIFT_E_NULL: return "a required pointer is NULL";
    case SIFT_E_SHAPE: return "tensor shapes do not match each other or the layout";
    case SIFT_E_LAYOUT: return "malformed prompt layout";
    case SIFT_E_UNSUPPORTED: return "tile size, head size or dtype not supported";
    case SIFT_E_CAPACITY: return "a buffer or index range is too small";
    case SIFT_E_HIP: return "a HIP runtime call failed";
    case SIFT_E_PLAN: return "the plan does not match the arguments or the device";
    default: return "unknown status";
  }
}

}  // extern "C"

namespace {

// Pinned host staging for stream-ordered uploads of plan tables.  A buffer
// is handed out to one call at a time; after the call has enqueued its copy
// it records an event, and the buffer is reused once that event has
// completed (the copy has read it).  Buffers live until the process ends.
struct StagingBuf {
  int device;
  void* host;
  size_t cap;
  hipEvent_t done;
  bool taken;
};
std::mutex g_staging_mu;
std::vector<StagingBuf> g_staging;

// Index of a free pinned buffer of at least n bytes on the current device.
sift_status staging_acquire(size_t n, size_t* idx) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SIFT_E_HIP;
  std::lock_guard<std::mutex> lock(g_staging_mu);
  for (size_t i = 0; i < g_staging.size(); ++i) {
    StagingBuf& b = g_staging[i];
    if (b.taken || b.device != dev || b.cap < n) continue;
    const hipError_t q = hipEventQuery(b.done);
    if (q == hipErrorNotReady) continue;
    if (q != hipSuccess) return SIFT_E_HIP;
    b.taken = true;
    *idx = i;
    return SIFT_OK;
  }
  size_t cap = 1 << 16;
  while (cap < n) cap <<= 1;
  StagingBuf b{dev, nullptr, cap, nullptr, true};
  if (hipHostMalloc(&b.host, cap, hipHostMallocDefault) != hipSuccess) return SIFT_E_HIP;
  if (hipEventCreateWithFlags(&b.done, hipEventDisableTiming) != hipSuccess) {
    (void)hipHostFree(b.host);
    return SIFT_E_HIP;
  }
  g_staging.push_back(b);
  *idx = g_staging.size() - 1;
  return SIFT_OK;
}

// Hand a buffer back; with a stream, once the copies enqueued on it so far
// are done.
sift_status staging_release(size_t idx, hipStream_t stream, bool record) {
  std::lock_guard<std::mutex> lock(g_staging_mu);
  StagingBuf& b = g_staging[idx];
  b.taken = false;
  if (record && hipEventRecord(b.done, stream) != hipSuccess) return SIFT_E_HIP;
  return SIFT_OK;
}

// How the plan's tables reach the device.
enum class Upload {
  kBlocking,   // hipMemcpy into the plan's own hipMalloc (sift_plan_create)
  kStaged,     // hipMemcpyAsync on `stream` from pinned staging: no host wait
  kPageable,   // hipMemcpyAsync on `stream` from host memory, then a wait for
               // `stream` (no allocation at all)
};

// The plan's device memory: with ws == nullptr a hipMalloc of its own, else
// ws (ws_bytes, 256-byte aligned): the caller's workspace, stream-ordered
// scratch or static scratch, written on `stream` as `up` says.  With
// bytes_only != nullptr only the size is computed.
//
// Layout: the tables, then the schedule's bucket sizes and the attention's
// redo flag (zero: uploaded with the tables, and left so by every pass that
// uses them), then the decode and merge scratch.
sift_status create_plan(const sift_layout* layout, int32_t num_q_heads, int32_t num_kv_heads,
                        int32_t head_dim, int32_t tile, void* ws, size_t ws_bytes,
                        hipStream_t stream, Upload up, size_t* bytes_only,
                        sift_plan** plan_out) {
  if (layout == nullptr || (plan_out == nullptr && bytes_only == nullptr)) return SIFT_E_NULL;
  if (plan_out != nullptr) *plan_out = nullptr;
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads != 0) return SIFT_E_SHAPE;
  if (head_dim != 64 && head_dim != 128) return SIFT_E_UNSUPPORTED;
  if (tile != 16 && tile != 32 && tile != 64 && tile != 128) return SIFT_E_UNSUPPORTED;
  HostPlan hp;
  sift_status st = build_host_plan(layout, num_q_heads, num_kv_heads, tile, hp);
  if (st != SIFT_OK) return st;

  std::vector<uint8_t> blob;
  const size_t o_seg_tile0 = put(blob, hp.seg_tile0);
  const size_t o_seg_pages = put(blob, hp.seg_pages);
  const size_t o_seg_kind = put(blob, hp.seg_kind);
  const size_t o_seg_first = put(blob, hp.seg_first);
  const size_t o_seg_la = put(blob, hp.seg_la_off);
  const size_t o_seg_ca = put(blob, hp.seg_ca_off);
  const size_t o_tile_seg = put(blob, hp.tile_seg);
  const size_t o_tile_tok0 = put(blob, hp.tile_tok0);
  const size_t o_tile_len = put(blob, hp.tile_len);
  const size_t o_tile_lo = put(blob, hp.tile_lo);
  const size_t o_tile_info = put(blob, hp.tile_info);
  const size_t o_uh = put(blob, hp.unit_head);
  const size_t o_um0 = put(blob, hp.unit_m0);
  const size_t o_unb = put(blob, hp.unit_nb);
  const size_t o_soff = put(blob, hp.step_off);
  const size_t o_lw0 = put(blob, hp.lu_work0);
  const size_t o_lnw = put(blob, hp.lu_nwork);
  const size_t o_llen = put(blob, hp.lu_len);
  const size_t o_urec = put(blob, hp.urec);
  const size_t o_rec = put(blob, hp.rec);  // step counts and first steps: written by decode
  const size_t o_launch = put(blob, hp.launch);  // written by the schedule pass
  const size_t o_splits = put(blob, hp.splits);
  // the schedule's bucket sizes, the bf16 attention's redo flag and
  // counters, the decode's finished-block count: zeros, uploaded with the
  // tables
  constexpr size_t kHistWords = sift::kNumXcd * sift::kSchedBuckets + 4 + sift::kNumXcd;
  const size_t o_hist = put(blob, std::vector<int32_t>(kHistWords, 0));
  const int64_t rows = static_cast<int64_t>(hp.num_tiles) * num_q_heads;
  const int64_t cap = hp.dense_tiles * num_q_heads;
  const int64_t U = static_cast<int64_t>(hp.unit_head.size());
  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t o_counts = align(blob.size());
  const size_t o_segbase = align(o_counts + rows * 4);
  const size_t o_headtot = align(o_segbase + static_cast<int64_t>(hp.num_segments) * num_q_heads * 4);
  const size_t o_camark = align(o_headtot + static_cast<int64_t>(num_q_heads) * 4);
  const size_t o_segcross = align(o_camark + rows);
  const size_t o_crosscol =
      align(o_segcross + static_cast<int64_t>(hp.num_segments) * num_q_heads * 4);
  const size_t o_crossrows = align(o_crosscol + rows * 4);
  const size_t o_rowptr = align(o_crossrows + rows * 8);
  const size_t o_col = align(o_rowptr + (rows + 1) * 4);
  const int64_t W = static_cast<int64_t>(hp.wk_head.size());
  const size_t o_steps = align(o_col + std::max<int64_t>(cap, 1) * 4);
  // steps: the units' lists, plus a few entries read (never used) past the end
  // (the lists' total length bound: one step per listed tile at T <= 64, up
  // to two at T = 128)
  const int64_t step_cap = hp.step_off.empty() ? 0 : hp.step_off.back();
  // per-step K/V row bases, T < 64 only
  const size_t o_kvb = align(o_steps + (std::max<int64_t>(step_cap, 1) + 8) * 8);
  const size_t o_part_o =
      align(o_kvb + (tile < 64 ? (std::max<int64_t>(step_cap, 1) + 8) * 16 : 0));
  const int64_t slot_rows = hp.part_slots * sift::kUnitRows;
  // the pieces' outputs: fp32, or bf16 plus the bf16 of its rounding error
  const size_t o_part_lo = align(o_part_o + slot_rows * head_dim * 4);
  const size_t o_part_ml = align(o_part_lo + slot_rows * head_dim * 2);
  const size_t total = o_part_ml + std::max<int64_t>(slot_rows, 1) * 8;

  if (bytes_only != nullptr) {
    *bytes_only = total;
    return SIFT_OK;
  }
  if (ws != nullptr) {
    if (ws_bytes < total) return SIFT_E_CAPACITY;
    if (reinterpret_cast<uintptr_t>(ws) % 256 != 0) return SIFT_E_UNSUPPORTED;
  }
  sift_plan* plan = new (std::nothrow) sift_plan();
  if (plan == nullptr) return SIFT_E_HIP;
  if (hipGetDevice(&plan->device) != hipSuccess) {
    delete plan;
    return SIFT_E_HIP;
  }
  auto fail = [plan]() {
    if (plan->owns_dev && plan->dev != nullptr) (void)hipFree(plan->dev);
    delete plan;
    return SIFT_E_HIP;
  };
  plan->dev_bytes = total;
  if (ws == nullptr) {
    if (hipMalloc(&plan->dev, total) != hipSuccess) return fail();
    if (hipMemcpy(plan->dev, blob.data(), blob.size(), hipMemcpyHostToDevice) != hipSuccess)
      return fail();
  } else {
    plan->dev = ws;
    plan->owns_dev = false;
    plan->last_stream = stream;
    if (up == Upload::kStaged) {
      // copy from pinned staging: the call returns without waiting, and the
      // staging buffer is reused only after the copy has read it
      size_t idx = 0;
      if (staging_acquire(blob.size(), &idx) != SIFT_OK) return fail();
      std::memcpy(g_staging[idx].host, blob.data(), blob.size());
      const bool ok = hipMemcpyAsync(plan->dev, g_staging[idx].host, blob.size(),
                                     hipMemcpyHostToDevice, stream) == hipSuccess;
      if (staging_release(idx, stream, ok) != SIFT_OK || !ok) return fail();
    } else {
      // host memory: the blob must outlive the copy, so wait for the stream
      if (hipMemcpyAsync(plan->dev, blob.data(), blob.size(), hipMemcpyHostToDevice,
                         stream) != hipSuccess)
        return fail();
      if (hipStreamSynchronize(stream) != hipSuccess) return fail();
    }
  }
  auto P = [plan](size_t off) {
    return reinterpret_cast<int32_t*>(static_cast<uint8_t*>(plan->dev) + off);
  };
  plan->pt.seg_tile0 = P(o_seg_tile0);
  plan->pt.seg_pages = P(o_seg_pages);
  plan->pt.seg_kind = P(o_seg_kind);
  plan->pt.seg_first = P(o_seg_first);
  plan->pt.seg_la_off = P(o_seg_la);
  plan->pt.seg_ca_off = P(o_seg_ca);
  plan->pt.tile_seg = P(o_tile_seg);
  plan->pt.tile_tok0 = P(o_tile_tok0);
  plan->pt.tile_len = P(o_tile_len);
  plan->pt.tile_lo = P(o_tile_lo);
  plan->pt.tile_info = reinterpret_cast<const int4*>(P(o_tile_info));
  plan->pt.tile = tile;
  plan->pt.halves = tile == 128 ? 2 : 1;
  plan->pt.group = tile < 64 ? 64 / tile : 1;
  plan->pt.num_tiles = hp.num_tiles;
  plan->pt.num_segments = hp.num_segments;
  plan->pt.num_q_heads = num_q_heads;
  plan->wt.rec = reinterpret_cast<sift::WorkRec*>(P(o_rec));
  plan->wt.launch = reinterpret_cast<sift::WorkRec*>(P(o_launch));
  plan->wt.hist = P(o_hist);
  plan->wt.lu_head = P(o_uh);
  plan->wt.lu_m0 = P(o_um0);
  plan->wt.lu_nb = P(o_unb);
  plan->wt.lu_off = P(o_soff);
  plan->wt.lu_work0 = P(o_lw0);
  plan->wt.lu_nwork = P(o_lnw);
  plan->wt.lu_len = P(o_llen);
  plan->wt.urec = reinterpret_cast<const sift::UnitRec*>(P(o_urec));
  plan->wt.steps = reinterpret_cast<int2*>(P(o_steps));
  plan->wt.kvb = tile < 64 ? reinterpret_cast<int4*>(P(o_kvb)) : nullptr;
  plan->wt.splits = reinterpret_cast<const int4*>(P(o_splits));
  plan->wt.part_o = static_cast<void*>(P(o_part_o));
  plan->wt.part_lo = static_cast<void*>(P(o_part_lo));
  plan->wt.part_ml = reinterpret_cast<float2*>(P(o_part_ml));
  plan->wt.redo = P(o_hist) + sift::kNumXcd * sift::kSchedBuckets;
  plan->wt.decode_done = plan->wt.redo + 3;
  plan->wt.sched_done = plan->wt.redo + 4;
  plan->wt.seg_base = P(o_segbase);
  plan->wt.head_tot = P(o_headtot);
  plan->wt.ca_mark = reinterpret_cast<uint8_t*>(P(o_camark));
  plan->wt.seg_cross = P(o_segcross);
  plan->wt.cross_col = P(o_crosscol);
  plan->wt.cross_rows = reinterpret_cast<int2*>(P(o_crossrows));
  plan->wt.num_units = static_cast<int32_t>(U);
  plan->wt.num_urec = static_cast<int32_t>(hp.urec.size());
  plan->wt.num_work = static_cast<int32_t>(W);
  plan->wt.num_splits = static_cast<int32_t>(hp.splits.size() / 4);
  plan->wt.chunk_size = static_cast<int32_t>(hp.chunk_size);
  plan->wt.sched_blocks = static_cast<int32_t>(
      std::min<int64_t>(8, std::max<int64_t>(1, ceil_div(hp.chunk_size, sift::kSchedPerBlock))));
  plan->wt.grid = static_cast<int32_t>(hp.launch.size());
  plan->counts = P(o_counts);
  plan->row_ptr = P(o_rowptr);
  plan->col_idx = P(o_col);

  sift_plan_info& in = plan->info;
  in.num_tokens = hp.num_tokens;
  in.num_segments = hp.num_segments;
  in.num_tiles = hp.num_tiles;
  in.num_q_heads = num_q_heads;
  in.num_kv_heads = num_kv_heads;
  in.head_dim = head_dim;
  in.tile = tile;
  in.num_work_units = static_cast<int32_t>(W);
  in.num_rows = rows;
  in.list_capacity = cap;
  in.la_bytes = hp.la_bytes;
  in.ca_bytes = hp.ca_bytes;
  in.scratch_bytes = static_cast<int64_t>(total);
  *plan_out = plan;
  return SIFT_OK;
}

// Arguments of the one-shot forms, checked on the host before anything is
// enqueued; *need receives the scratch bytes of their plan.
sift_status check_prefill(const sift_tensor* q, const sift_tensor* k, const sift_tensor* v,
                          const sift_layout* layout, const uint8_t* la, const uint8_t* ca,
                          int32_t tile, const sift_tensor* out, size_t* need) {
  if (q == nullptr || k == nullptr || v == nullptr || out == nullptr || layout == nullptr)
    return SIFT_E_NULL;
  if (q->heads < 1 || k->heads < 1 || q->heads % k->heads != 0) return SIFT_E_SHAPE;
  if (q->head_dim != 64 && q->head_dim != 128) return SIFT_E_UNSUPPORTED;
  if (tile != 16 && tile != 32 && tile != 64 && tile != 128) return SIFT_E_UNSUPPORTED;
  HostPlan hp;
  sift_status st = build_host_plan(layout, q->heads, k->heads, tile, hp);
  if (st != SIFT_OK) return st;
  st = check_io(q, k, v, out, hp.num_tokens, q->heads, k->heads, q->head_dim, tile);
  if (st != SIFT_OK) return st;
  if (hp.la_bytes > 0 && la == nullptr) return SIFT_E_NULL;
  if (hp.ca_bytes > 0 && ca == nullptr) return SIFT_E_NULL;
  return create_plan(layout, q->heads, k->heads, q->head_dim, tile, nullptr, 0, nullptr,
                     Upload::kBlocking, need, nullptr);
}

// Scratch for sift_sparse_prefill_static: one array per GPU, held from the
// library's load on that GPU until the process ends.  Host code never uses
// the array's name as an address: each device's address is taken once with
// hipGetSymbolAddress, with that device current, and kept here.
constexpr size_t kStaticScratchBytes = size_t(256) << 20;
__device__ __align__(256) uint8_t scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices] = {};
hipError_t g_scratch_err[kMaxDevices] = {};

// The current device's address of the scratch array.
sift_status static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SIFT_E_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SIFT_E_UNSUPPORTED;
  std::call_once(g_scratch_once[dev], [dev]() {
    g_scratch_err[dev] = hipGetSymbolAddress(&g_scratch_ptr[dev], HIP_SYMBOL(scratch));
  });
  if (g_scratch_err[dev] != hipSuccess || g_scratch_ptr[dev] == nullptr) return SIFT_E_HIP;
  *out = g_scratch_ptr[dev];
  return SIFT_OK;
}

// Plans made only to decode lists: the lists do not depend on the kv heads
// or the head size, so the smallest attention scratch is taken.
constexpr int32_t kDecodeKvHeads = 1;
constexpr int32_t kDecodeHeadDim = 64;

}  // namespace

extern "C" {

sift_status sift_plan_create(const sift_layout* layout, int32_t num_q_heads,
                             int32_t num_kv_heads, int32_t head_dim, int32_t tile,
                             sift_plan** plan_out) {
  if (plan_out == nullptr) return SIFT_E_NULL;
  return create_plan(layout, num_q_heads, num_kv_heads, head_dim, tile, nullptr, 0, nullptr,
                     Upload::kBlocking, nullptr, plan_out);
}

sift_status sift_workspace_bytes(const sift_layout* layout, int32_t num_q_heads,
                                 int32_t num_kv_heads, int32_t head_dim, int32_t tile,
                                 size_t* bytes) {
  if (bytes == nullptr) return SIFT_E_NULL;
  return create_plan(layout, num_q_heads, num_kv_heads, head_dim, tile, nullptr, 0, nullptr,
                     Upload::kBlocking, bytes, nullptr);
}

sift_status sift_plan_destroy(sift_plan* plan) {
  if (plan == nullptr) return SIFT_OK;
  sift_status st = SIFT_OK;
  if (plan->dev != nullptr && plan->owns_dev) {
    // the plan's last work may still read its memory
    if (hipStreamSynchronize(plan->last_stream) != hipSuccess) st = SIFT_E_HIP;
    if (hipFree(plan->dev) != hipSuccess) st = SIFT_E_HIP;
  }
  delete plan;
  return st;
}

sift_status sift_plan_exact_passes(const sift_plan* plan, int64_t* count) {
  if (plan == nullptr || count == nullptr) return SIFT_E_NULL;
  if (check_device(plan) != SIFT_OK) return SIFT_E_PLAN;
  int32_t n = 0;
  if (hipMemcpyAsync(&n, plan->wt.redo + 2, sizeof(n), hipMemcpyDeviceToHost,
                     plan->last_stream) != hipSuccess ||
      hipStreamSynchronize(plan->last_stream) != hipSuccess)
    return SIFT_E_HIP;
  *count = n;
  return SIFT_OK;
}

sift_status sift_plan_get_info(const sift_plan* plan, sift_plan_info* info) {
  if (plan == nullptr || info == nullptr) return SIFT_E_NULL;
  *info = plan->info;
  return SIFT_OK;
}

sift_status sift_plan_decode_tiles(sift_plan* plan, const uint8_t* local_bitmap,
                                   const uint8_t* cross_bitmap, int32_t* row_ptr,
                                   int32_t* col_idx, int64_t col_capacity, void* stream) {
  if (plan == nullptr || row_ptr == nullptr) return SIFT_E_NULL;
  if (plan->info.la_bytes > 0 && local_bitmap == nullptr) return SIFT_E_NULL;
  if (plan->info.ca_bytes > 0 && cross_bitmap == nullptr) return SIFT_E_NULL;
  if (plan->info.list_capacity > 0 && col_idx == nullptr) return SIFT_E_NULL;
  if (col_capacity < plan->info.list_capacity) return SIFT_E_CAPACITY;
  sift_status st = check_device(plan);
  if (st != SIFT_OK) return st;
  const hipError_t e = sift::launch_decode(plan->pt, work(plan), local_bitmap, cross_bitmap,
                                           plan->counts, row_ptr, col_idx,
                                           sift::KvPages{nullptr, 0},
                                           static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return SIFT_E_HIP;
  plan->steps_paged = false;
  plan->last_stream = static_cast<hipStream_t>(stream);
  return SIFT_OK;
}

sift_status sift_plan_decode(sift_plan* plan, const uint8_t* local_bitmap,
                             const uint8_t* cross_bitmap, void* stream) {
  if (plan == nullptr) return SIFT_E_NULL;
  return sift_plan_decode_tiles(plan, local_bitmap, cross_bitmap, plan->row_ptr, plan->col_idx,
                                plan->info.list_capacity, stream);
}

sift_status sift_sparse_attention(sift_plan* plan, const sift_tensor* q, const sift_tensor* k,
                                  const sift_tensor* v, const int32_t* row_ptr,
                                  const int32_t* col_idx, int64_t col_capacity,
                                  float softmax_scale, sift_tensor* out, void* stream) {
  if (plan == nullptr || row_ptr == nullptr) return SIFT_E_NULL;
  const sift_plan_info& in = plan->info;
  sift_status st = check_io(q, k, v, out, in.num_tokens, in.num_q_heads, in.num_kv_heads,
                            in.head_dim, in.tile);
  if (st != SIFT_OK) return st;
  if (col_capacity < 0) return SIFT_E_CAPACITY;
  if (col_capacity > 0 && col_idx == nullptr) return SIFT_E_NULL;
  const bool bf16 = q->dtype == SIFT_BF16;
  if (!(softmax_scale > 0.f) || !std::isfinite(softmax_scale))
    softmax_scale = 1.0f / std::sqrt(static_cast<float>(in.head_dim));
  if ((st = check_device(plan)) != SIFT_OK) return st;
  sift::AttnArgs a{};
  a.q = q->data;
  a.k = k->data;
  a.v = v->data;
  a.out = out->data;
  a.row_ptr = row_ptr;
  a.col_idx = col_idx;
  a.col_capacity = col_capacity;
  a.hq = in.num_q_heads;
  a.hkv = in.num_kv_heads;
  a.head_dim = in.head_dim;
  a.tile = in.tile;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  a.out_f32 = out->dtype == SIFT_F32 ? 1 : 0;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (bf16) {
    // the bf16 kernel walks merged per-unit step lists: build them from the lists
    e = sift::launch_merge_steps(plan->pt, work(plan), row_ptr, col_idx, col_capacity, s);
    if (e == hipSuccess) plan->steps_paged = false;
    if (e == hipSuccess) e = sift::launch_attn_bf16(plan->pt, work(plan), a, s);
  } else {
    e = sift::launch_attn_f32(plan->pt, a, s);
  }
  plan->last_stream = s;
  return e == hipSuccess ? SIFT_OK : SIFT_E_HIP;
}

sift_status sift_plan_attention(sift_plan* plan, const sift_tensor* q, const sift_tensor* k,
                                const sift_tensor* v, float softmax_scale, sift_tensor* out,
                                void* stream) {
  if (plan == nullptr) return SIFT_E_NULL;
  const sift_plan_info& in = plan->info;
  sift_status st = check_io(q, k, v, out, in.num_tokens, in.num_q_heads, in.num_kv_heads,
                            in.head_dim, in.tile);
  if (st != SIFT_OK) return st;
  if (plan->steps_paged && q->dtype == SIFT_BF16) return SIFT_E_PLAN;  // steps index a page pool
  if ((st = check_device(plan)) != SIFT_OK) return st;
  if (!(softmax_scale > 0.f) || !std::isfinite(softmax_scale))
    softmax_scale = 1.0f / std::sqrt(static_cast<float>(in.head_dim));
  sift::AttnArgs a{};
  a.q = q->data;
  a.k = k->data;
  a.v = v->data;
  a.out = out->data;
  a.row_ptr = plan->row_ptr;
  a.col_idx = plan->col_idx;
  a.col_capacity = in.list_capacity;
  a.hq = in.num_q_heads;
  a.hkv = in.num_kv_heads;
  a.head_dim = in.head_dim;
  a.tile = in.tile;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  a.out_f32 = out->dtype == SIFT_F32 ? 1 : 0;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t e = q->dtype == SIFT_BF16 ? sift::launch_attn_bf16(plan->pt, work(plan), a, s)
                                             : sift::launch_attn_f32(plan->pt, a, s);
  plan->last_stream = s;
  return e == hipSuccess ? SIFT_OK : SIFT_E_HIP;
}

sift_status sift_plan_run(sift_plan* plan, const sift_tensor* q, const sift_tensor* k,
                          const sift_tensor* v, const uint8_t* local_bitmap,
                          const uint8_t* cross_bitmap, float softmax_scale, sift_tensor* out,
                          void* stream) {
  if (plan == nullptr) return SIFT_E_NULL;
  const sift_plan_info& in = plan->info;
  // check everything before enqueuing the decode
  sift_status st = check_io(q, k, v, out, in.num_tokens, in.num_q_heads, in.num_kv_heads,
                            in.head_dim, in.tile);
  if (st != SIFT_OK) return st;
  if (in.la_bytes > 0 && local_bitmap == nullptr) return SIFT_E_NULL;
  if (in.ca_bytes > 0 && cross_bitmap == nullptr) return SIFT_E_NULL;
  st = sift_plan_decode(plan, local_bitmap, cross_bitmap, stream);
  if (st != SIFT_OK) return st;
  return sift_plan_attention(plan, q, k, v, softmax_scale, out, stream);
}


sift_status sift_plan_run_paged(sift_plan* plan, const sift_tensor* q, const sift_tensor* k_pages,
                                const sift_tensor* v_pages, const int32_t* page_table,
                                const uint8_t* local_bitmap, const uint8_t* cross_bitmap,
                                float softmax_scale, sift_tensor* out, void* stream) {
  if (plan == nullptr || k_pages == nullptr || v_pages == nullptr) return SIFT_E_NULL;
  const sift_plan_info& in = plan->info;
  sift_status st;
  if ((st = check_tensor(q, in.num_tokens, in.num_q_heads, in.head_dim)) != SIFT_OK) return st;
  if ((st = check_tensor(out, in.num_tokens, in.num_q_heads, in.head_dim)) != SIFT_OK) return st;
  // the pools: whole pages of T rows, at least one when there are tiles
  const int32_t rows = k_pages->tokens;
  if (rows < 0 || rows % in.tile != 0) return SIFT_E_SHAPE;
  const int32_t num_pages = rows / in.tile;
  if ((st = check_tensor(k_pages, rows, in.num_kv_heads, in.head_dim)) != SIFT_OK) return st;
  if ((st = check_tensor(v_pages, rows, in.num_kv_heads, in.head_dim)) != SIFT_OK) return st;
  if (in.num_tiles > 0 && num_pages < 1) return SIFT_E_SHAPE;
  if (in.num_tiles > 0 && page_table == nullptr) return SIFT_E_NULL;
  if (q->dtype != k_pages->dtype || q->dtype != v_pages->dtype) return SIFT_E_UNSUPPORTED;
  // bf16 at T < 64: a 64-key step's tiles each come from their own page
  if (q->dtype == SIFT_BF16 && in.head_dim != 128) return SIFT_E_UNSUPPORTED;
  if (q->dtype == SIFT_F32 && (out->dtype != SIFT_F32 || in.tile > 64)) return SIFT_E_UNSUPPORTED;
  if (in.la_bytes > 0 && local_bitmap == nullptr) return SIFT_E_NULL;
  if (in.ca_bytes > 0 && cross_bitmap == nullptr) return SIFT_E_NULL;
  if ((st = check_device(plan)) != SIFT_OK) return st;
  if (!(softmax_scale > 0.f) || !std::isfinite(softmax_scale))
    softmax_scale = 1.0f / std::sqrt(static_cast<float>(in.head_dim));
  const sift::KvPages pages{page_table, num_pages};
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = sift::launch_decode(plan->pt, work(plan), local_bitmap, cross_bitmap,
                                     plan->counts, plan->row_ptr, plan->col_idx, pages, s);
  plan->last_stream = s;
  if (e != hipSuccess) return SIFT_E_HIP;
  plan->steps_paged = true;
  sift::AttnArgs a{};
  a.q = q->data;
  a.k = k_pages->data;
  a.v = v_pages->data;
  a.out = out->data;
  a.row_ptr = plan->row_ptr;
  a.col_idx = plan->col_idx;
  a.col_capacity = in.list_capacity;
  a.hq = in.num_q_heads;
  a.hkv = in.num_kv_heads;
  a.head_dim = in.head_dim;
  a.tile = in.tile;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  a.out_f32 = out->dtype == SIFT_F32 ? 1 : 0;
  a.pages = pages;
  e = q->dtype == SIFT_BF16 ? sift::launch_attn_bf16(plan->pt, work(plan), a, s)
                            : sift::launch_attn_f32(plan->pt, a, s);
  plan->last_stream = s;
  return e == hipSuccess ? SIFT_OK : SIFT_E_HIP;
}

sift_status sift_sparse_prefill(const sift_tensor* q, const sift_tensor* k, const sift_tensor* v,
                                const sift_layout* doc_offsets, const uint8_t* local_bitmap,
                                const uint8_t* cross_bitmap, int32_t tile, sift_tensor* out,
                                void* stream) {
  size_t need = 0;
  sift_status st = check_prefill(q, k, v, doc_offsets, local_bitmap, cross_bitmap, tile, out,
                                 &need);
  if (st != SIFT_OK) return st;
  // stream-ordered scratch: allocated, used and freed in the order of `stream`
  const hipStream_t s = static_cast<hipStream_t>(stream);
  void* ws = nullptr;
  if (hipMallocAsync(&ws, need, s) != hipSuccess) return SIFT_E_HIP;
  sift_plan* plan = nullptr;
  st = create_plan(doc_offsets, q->heads, k->heads, q->head_dim, tile, ws, need, s,
                   Upload::kStaged, nullptr, &plan);
  if (st == SIFT_OK)
    st = sift_plan_run(plan, q, k, v, local_bitmap, cross_bitmap, 0.f, out, stream);
  const sift_status st2 = sift_plan_destroy(plan);  // host state only: ws is freed below
  if (hipFreeAsync(ws, s) != hipSuccess && st == SIFT_OK) return SIFT_E_HIP;
  return st != SIFT_OK ? st : st2;
}

sift_status sift_sparse_prefill_ex(const sift_tensor* q, const sift_tensor* k,
                                   const sift_tensor* v, const sift_layout* doc_offsets,
                                   const uint8_t* local_bitmap, const uint8_t* cross_bitmap,
                                   int32_t tile, float softmax_scale, void* workspace,
                                   size_t workspace_bytes, sift_tensor* out, void* stream) {
  size_t need = 0;
  sift_status st = check_prefill(q, k, v, doc_offsets, local_bitmap, cross_bitmap, tile, out,
                                 &need);
  if (st != SIFT_OK) return st;
  if (workspace == nullptr) return SIFT_E_NULL;
  if (workspace_bytes < need) return SIFT_E_CAPACITY;
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return SIFT_E_UNSUPPORTED;
  sift_plan* plan = nullptr;
  st = create_plan(doc_offsets, q->heads, k->heads, q->head_dim, tile, workspace,
                   workspace_bytes, static_cast<hipStream_t>(stream), Upload::kStaged, nullptr,
                   &plan);
  if (st != SIFT_OK) return st;
  st = sift_plan_run(plan, q, k, v, local_bitmap, cross_bitmap, softmax_scale, out, stream);
  const sift_status st2 = sift_plan_destroy(plan);  // host state only: the workspace is the caller's
  return st != SIFT_OK ? st : st2;
}

sift_status sift_decode_workspace_bytes(const sift_layout* layout, int32_t num_q_heads,
                                        int32_t tile, size_t* bytes) {
  if (bytes == nullptr) return SIFT_E_NULL;
  return create_plan(layout, num_q_heads, kDecodeKvHeads, kDecodeHeadDim, tile, nullptr, 0,
                     nullptr, Upload::kBlocking, bytes, nullptr);
}

sift_status sift_decode_tiles(const sift_layout* layout, const uint8_t* local_bitmap,
                              const uint8_t* cross_bitmap, int32_t tile, int32_t num_q_heads,
                              int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                              void* workspace, size_t workspace_bytes, void* stream) {
  if (layout == nullptr || row_ptr == nullptr || workspace == nullptr) return SIFT_E_NULL;
  if (num_q_heads < 1) return SIFT_E_SHAPE;
  if (tile != 16 && tile != 32 && tile != 64 && tile != 128) return SIFT_E_UNSUPPORTED;
  HostPlan hp;
  sift_status st = build_host_plan(layout, num_q_heads, kDecodeKvHeads, tile, hp);
  if (st != SIFT_OK) return st;
  if (hp.la_bytes > 0 && local_bitmap == nullptr) return SIFT_E_NULL;
  if (hp.ca_bytes > 0 && cross_bitmap == nullptr) return SIFT_E_NULL;
  const int64_t cap = hp.dense_tiles * num_q_heads;
  if (cap > 0 && col_idx == nullptr) return SIFT_E_NULL;
  if (col_capacity < cap) return SIFT_E_CAPACITY;
  size_t need = 0;
  if ((st = sift_decode_workspace_bytes(layout, num_q_heads, tile, &need)) != SIFT_OK) return st;
  if (workspace_bytes < need) return SIFT_E_CAPACITY;
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return SIFT_E_UNSUPPORTED;
  sift_plan* plan = nullptr;
  st = create_plan(layout, num_q_heads, kDecodeKvHeads, kDecodeHeadDim, tile, workspace,
                   workspace_bytes, static_cast<hipStream_t>(stream), Upload::kStaged, nullptr,
                   &plan);
  if (st != SIFT_OK) return st;
  st = sift_plan_decode_tiles(plan, local_bitmap, cross_bitmap, row_ptr, col_idx, col_capacity,
                              stream);
  const sift_status st2 = sift_plan_destroy(plan);  // host state only
  return st != SIFT_OK ? st : st2;
}

sift_status sift_sparse_prefill_static(const sift_tensor* q, const sift_tensor* k,
                                       const sift_tensor* v, const sift_layout* doc_offsets,
                                       const uint8_t* local_bitmap, const uint8_t* cross_bitmap,
                                       int32_t tile, float softmax_scale, sift_tensor* out,
                                       void* stream) {
  size_t need = 0;
  sift_status st = check_prefill(q, k, v, doc_offsets, local_bitmap, cross_bitmap, tile, out,
                                 &need);
  if (st != SIFT_OK) return st;
  if (need > kStaticScratchBytes) return SIFT_E_CAPACITY;
  void* ws = nullptr;
  if ((st = static_scratch(&ws)) != SIFT_OK) return st;
  // tables from host memory: the call waits for the copy, so nothing is
  // allocated to hold them
  sift_plan* plan = nullptr;
  st = create_plan(doc_offsets, q->heads, k->heads, q->head_dim, tile, ws, kStaticScratchBytes,
                   static_cast<hipStream_t>(stream), Upload::kPageable, nullptr, &plan);
  if (st != SIFT_OK) return st;
  st = sift_plan_run(plan, q, k, v, local_bitmap, cross_bitmap, softmax_scale, out, stream);
  const sift_status st2 = sift_plan_destroy(plan);  // host state only
  return st != SIFT_OK ? st : st2;
}

size_t sift_static_scratch_bytes(void) { return kStaticScratchBytes; }

}  // extern "C"
