// C ABI of the offline metadata extraction (Sections 4.1, 4.2, 4.4): host
// validation, the per-document tables and the workspace layout.  The kernels
// are in extract.hip.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "sift.h"
#include "sift_internal.h"

namespace {

constexpr int kQueryBlock = 128;  // query rows per extraction workgroup

struct ExtractPlan {
  std::vector<sift::ExtractDoc> docs;
  std::vector<int32_t> blocks;  // int2 {document, query block}, longest first
  size_t la_bytes = 0, ca_bytes = 0;
  size_t o_docs = 0, o_blocks = 0, o_flags = 0, o_counts = 0, end = 0;
  int64_t flag_bytes = 0, count_words = 0;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

sift_status build_extract_plan(int32_t num_docs, const int32_t* offs, int32_t hq, int32_t tile,
                               ExtractPlan& ep) {
  if (offs == nullptr) return SIFT_E_NULL;
  if (num_docs < 0 || hq < 1) return SIFT_E_LAYOUT;
  if (tile != 16 && tile != 32 && tile != 64 && tile != 128) return SIFT_E_UNSUPPORTED;
  if (offs[0] != 0) return SIFT_E_LAYOUT;
  ep.docs.resize(num_docs);
  int64_t la = 0, ca = 0, fl = 0, cn = 0;
  std::vector<std::pair<int32_t, int32_t>> blk;
  for (int32_t d = 0; d < num_docs; ++d) {
    const int64_t len = static_cast<int64_t>(offs[d + 1]) - offs[d];
    if (len < 1) return SIFT_E_LAYOUT;
    const int64_t P = (len + tile - 1) / tile;
    sift::ExtractDoc& e = ep.docs[d];
    e.tok0 = offs[d];
    e.len = static_cast<int32_t>(len);
    e.P = static_cast<int32_t>(P);
    e.pad = 0;
    e.la_off = la;
    e.ca_off = ca;
    e.flag_off = fl;
    e.cnt_off = cn;
    la += hq * ((P * (P + 1) / 2 + 7) / 8);
    ca += hq * ((P + 7) / 8);
    fl += hq * (P * (P + 1) / 2);
    cn += hq * P;
    for (int32_t b = 0; b * kQueryBlock < len; ++b) blk.push_back({d, b});
  }
  // the causal work of a block grows with its index: longest first
  std::stable_sort(blk.begin(), blk.end(),
                   [](const auto& x, const auto& y) { return x.second > y.second; });
  if (blk.size() > static_cast<size_t>(INT32_MAX)) return SIFT_E_CAPACITY;
  ep.blocks.resize(2 * blk.size());
  for (size_t i = 0; i < blk.size(); ++i) {
    ep.blocks[2 * i] = blk[i].first;
    ep.blocks[2 * i + 1] = blk[i].second;
  }
  ep.la_bytes = static_cast<size_t>(la);
  ep.ca_bytes = static_cast<size_t>(ca);
  ep.flag_bytes = fl;
  ep.count_words = cn;
  ep.o_docs = 0;
  ep.o_blocks = align256(ep.o_docs + ep.docs.size() * sizeof(sift::ExtractDoc));
  ep.o_flags = align256(ep.o_blocks + ep.blocks.size() * sizeof(int32_t));
  ep.o_counts = align256(ep.o_flags + static_cast<size_t>(fl));
  ep.end = align256(ep.o_counts + static_cast<size_t>(cn) * 4);
  return SIFT_OK;
}

}  // namespace

extern "C" {

sift_status sift_extract_sizes(int32_t num_docs, const int32_t* doc_offsets, int32_t num_q_heads,
                               int32_t tile, size_t* la_bytes, size_t* ca_bytes,
                               size_t* workspace_bytes) {
  ExtractPlan ep;
  const sift_status st = build_extract_plan(num_docs, doc_offsets, num_q_heads, tile, ep);
  if (st != SIFT_OK) return st;
  if (la_bytes != nullptr) *la_bytes = ep.la_bytes;
  if (ca_bytes != nullptr) *ca_bytes = ep.ca_bytes;
  if (workspace_bytes != nullptr) *workspace_bytes = ep.end;
  return SIFT_OK;
}

sift_status sift_extract_bits(const sift_tensor* q, const sift_tensor* k, int32_t num_docs,
                              const int32_t* doc_offsets, int32_t tile, double alpha, double beta,
                              double gamma, float softmax_scale, uint8_t* la_out, uint8_t* ca_out,
                              void* workspace, size_t workspace_bytes, void* stream) {
  if (q == nullptr || k == nullptr || doc_offsets == nullptr) return SIFT_E_NULL;
  if (q->data == nullptr || k->data == nullptr) return SIFT_E_NULL;
  ExtractPlan ep;
  sift_status st = build_extract_plan(num_docs, doc_offsets, q->heads, tile, ep);
  if (st != SIFT_OK) return st;
  const int32_t tokens = doc_offsets[num_docs];
  if (q->tokens != tokens || k->tokens != tokens) return SIFT_E_SHAPE;
  if (k->heads < 1 || q->heads % k->heads != 0) return SIFT_E_SHAPE;
  if (q->head_dim != k->head_dim) return SIFT_E_SHAPE;
  if (q->dtype != SIFT_BF16 || k->dtype != SIFT_BF16) return SIFT_E_UNSUPPORTED;
  if (q->head_dim != 64 && q->head_dim != 128) return SIFT_E_UNSUPPORTED;
  if (!(alpha >= 0.0) || !(beta >= 0.0) || !(gamma >= 0.0 && gamma <= 1.0) || !std::isfinite(alpha) ||
      !std::isfinite(beta))
    return SIFT_E_UNSUPPORTED;
  if (ep.la_bytes > 0 && la_out == nullptr) return SIFT_E_NULL;
  if (ep.ca_bytes > 0 && ca_out == nullptr) return SIFT_E_NULL;
  if (workspace == nullptr && ep.end > 0) return SIFT_E_NULL;
  if (workspace_bytes < ep.end) return SIFT_E_CAPACITY;
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return SIFT_E_UNSUPPORTED;
  if (num_docs == 0) return SIFT_OK;

  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  // the workspace may still be read by earlier work on the stream
  if (hipStreamSynchronize(s) != hipSuccess) return SIFT_E_HIP;
  if (hipMemcpy(ws + ep.o_docs, ep.docs.data(), ep.docs.size() * sizeof(sift::ExtractDoc),
                hipMemcpyHostToDevice) != hipSuccess)
    return SIFT_E_HIP;
  if (hipMemcpy(ws + ep.o_blocks, ep.blocks.data(), ep.blocks.size() * sizeof(int32_t),
                hipMemcpyHostToDevice) != hipSuccess)
    return SIFT_E_HIP;

  sift::ExtractArgs a;
  a.docs = reinterpret_cast<const sift::ExtractDoc*>(ws + ep.o_docs);
  a.blocks = reinterpret_cast<const int2*>(ws + ep.o_blocks);
  a.q = static_cast<const __bf16*>(q->data);
  a.k = static_cast<const __bf16*>(k->data);
  a.flags = ws + ep.o_flags;
  a.counts = reinterpret_cast<int32_t*>(ws + ep.o_counts);
  a.hq = q->heads;
  a.hkv = k->heads;
  const float scale = softmax_scale > 0.f ? softmax_scale
                                          : 1.0f / std::sqrt(static_cast<float>(q->head_dim));
  a.c = scale * 1.4426950408889634f;
  a.log2_alpha = static_cast<float>(std::log2(alpha));
  a.log2_beta = static_cast<float>(std::log2(beta));
  a.gamma = gamma;
  const int64_t zero_words = static_cast<int64_t>((ep.end - ep.o_flags) / 4);
  const hipError_t e = sift::launch_extract(
      a, num_docs, static_cast<int32_t>(ep.blocks.size() / 2), q->head_dim, tile,
      reinterpret_cast<uint32_t*>(ws + ep.o_flags), zero_words, la_out, ca_out, s);
  return e == hipSuccess ? SIFT_OK : SIFT_E_HIP;
}

}  // extern "C"
