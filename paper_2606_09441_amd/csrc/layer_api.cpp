// C ABI of the pieces the decoder-layer prefill slice adds around the sparse
// attention: the rotary position embedding (rope.hip).  The projections are
// library GEMMs called by the caller.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "sift.h"
#include "sift_internal.h"

extern "C" {

sift_status sift_rope(const sift_tensor* q, const sift_tensor* k, const int32_t* positions,
                      const float* inv_freq, void* stream) {
  if (q == nullptr || k == nullptr) return SIFT_E_NULL;
  if (q->tokens > 0 && (q->data == nullptr || k->data == nullptr || positions == nullptr ||
                        inv_freq == nullptr))
    return SIFT_E_NULL;
  if (q->tokens != k->tokens || q->tokens < 0) return SIFT_E_SHAPE;
  if (q->head_dim != k->head_dim || q->heads < 1 || k->heads < 1) return SIFT_E_SHAPE;
  if (q->dtype != SIFT_BF16 || k->dtype != SIFT_BF16) return SIFT_E_UNSUPPORTED;
  if (q->head_dim < 2 || q->head_dim % 2 != 0) return SIFT_E_UNSUPPORTED;
  if (q->tokens == 0) return SIFT_OK;
  const hipError_t e = sift::launch_rope(q->data, q->tokens, q->heads, k->data, k->heads,
                                         q->head_dim, positions, inv_freq,
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SIFT_OK : SIFT_E_HIP;
}

}  // extern "C"
