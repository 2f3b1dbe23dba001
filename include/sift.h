/*
 * sift.h - C ABI of libsift: bitmap-driven sparse prefill attention for
 * AMD Instinct MI355X (gfx950), after SIFT (arXiv 2606.09441).
 *
 * One call computes, for one layer, causal GQA attention of a packed batch
 * of RAG prompts, evaluating only the tiles that two bit vectors per
 * (document, query head) mark (Sections 4.1-4.2), with the user-query rows
 * dense (Section 3.1).  It runs as two device steps (Section 5):
 *   1. decode: the bit vectors become, for every (query head, M-block), a
 *      packed ascending int32 list of the key tiles (N-blocks) to compute
 *      (Section 5.1, "sparse_n_indices"): a count pass, a prefix sum, a
 *      write pass;
 *   2. attention: a flash-style kernel walks only the listed tiles with an
 *      online softmax (Section 5.2).
 *
 * Conventions used by every entry point
 * -------------------------------------
 * Tensors: q, out are [tokens][Hq][D], k, v are [tokens][Hkv][D], dense,
 *   row-major, in device memory.  Query head h reads kv head h / (Hq/Hkv).
 * Layout (host memory): prompt b owns segments prompt_seg_ptr[b] ..
 *   prompt_seg_ptr[b+1]-1 of the packed token axis; the last one is its user
 *   query, the ones before it its documents in prompt order.  Segment s
 *   covers tokens seg_offsets[s] .. seg_offsets[s+1]-1.  Documents hold at
 *   least one token; a query may be empty.  Prompts never attend to each
 *   other.
 * Tiles: tile size T.  Tiles are segment-local: tile i of segment s covers
 *   tokens seg_offsets[s] + i*T .. + T-1, clipped to the segment, so the last
 *   tile of a segment may be partial.  P_s = ceil(len_s / T) (Section 4.3).
 *   The global number of tile i of segment s is i plus the tile count of all
 *   earlier segments (of all prompts); M is the total.  Every tile is both
 *   an M-block (query rows) and an N-block (keys).
 * Bit vectors (device memory, Sections 4.1-4.3): local_bitmap holds, for
 *   every document of every prompt in layout order and, inside it, for query
 *   heads h = 0..Hq-1, ceil(P(P+1)/16) bytes: one bit per tile (i, j), j <= i,
 *   of the document's lower triangle, enumerated (0,0),(1,0),(1,1),(2,0),...,
 *   most significant bit first.  cross_bitmap holds, in the same order,
 *   ceil(P/8) bytes per vector: bit p (MSB first) says whether key page p of
 *   the document is computed for the rows of later documents of the prompt.
 *   Stored diagonal bits and padding bits are ignored: diagonal tiles are
 *   always computed.
 * Lists: row h*M + m of row_ptr/col_idx holds query head h, M-block m.
 *   Document M-block i of document d lists, in ascending order, the marked
 *   pages of every earlier document of its prompt, the marked tiles j < i of
 *   d, then i itself.  A query M-block lists every tile of its prompt up to
 *   and including itself.
 * Streams: `stream` is a hipStream_t (NULL = the null stream).  All device
 *   work is enqueued on it; entry points return once it is enqueued.
 * Errors: arguments are checked on the host before anything is enqueued; on
 *   any error nothing is written and nothing is enqueued.  SIFT_E_HIP
 *   reports a failed HIP call; faults of enqueued kernels surface at the
 *   caller's next synchronisation.
 * Threads: plans are not shared between concurrent calls: calls that use
 *   the same plan must be ordered (same stream, or synchronised), since they
 *   share the plan's device scratch.
 */
#ifndef SIFT_H_
#define SIFT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sift_status {
  SIFT_OK = 0,
  SIFT_E_NULL = 1,        /* a required pointer is NULL                       */
  SIFT_E_SHAPE = 2,       /* tensor shapes disagree (with each other/layout)  */
  SIFT_E_LAYOUT = 3,      /* malformed layout                                 */
  SIFT_E_UNSUPPORTED = 4, /* valid, but not implemented (tile, D, dtype)      */
  SIFT_E_CAPACITY = 5,    /* a caller buffer is too small                     */
  SIFT_E_HIP = 6,         /* a HIP runtime call failed                        */
  SIFT_E_PLAN = 7         /* the plan does not match the arguments            */
} sift_status;

typedef enum sift_dtype { SIFT_F32 = 0, SIFT_BF16 = 1 } sift_dtype;

/* A dense device tensor [tokens][heads][head_dim]. */
typedef struct sift_tensor {
  void* data;
  int32_t dtype; /* sift_dtype */
  int32_t tokens;
  int32_t heads;
  int32_t head_dim;
} sift_tensor;

/* The prompt layout, in host memory; see "Layout" above. */
typedef struct sift_layout {
  int32_t num_prompts;            /* B >= 1                                  */
  const int32_t* prompt_seg_ptr;  /* [B + 1], prompt_seg_ptr[0] == 0         */
  const int32_t* seg_offsets;     /* [prompt_seg_ptr[B] + 1], [0] == 0       */
} sift_layout;

/* Opaque: a validated layout, its device tables and scratch. */
typedef struct sift_plan sift_plan;

typedef struct sift_plan_info {
  int32_t num_tokens;
  int32_t num_segments;
  int32_t num_tiles;        /* M                                            */
  int32_t num_q_heads;      /* Hq                                           */
  int32_t num_kv_heads;     /* Hkv                                          */
  int32_t head_dim;         /* D                                            */
  int32_t tile;             /* T                                            */
  int32_t num_work_units;   /* attention workgroups' units (pieces counted) */
  int64_t num_rows;         /* Hq * M; row_ptr holds num_rows + 1 entries   */
  int64_t list_capacity;    /* Hq * (dense causal tile count): >= any nnz   */
  int64_t la_bytes;         /* size local_bitmap must have                  */
  int64_t ca_bytes;         /* size cross_bitmap must have                  */
  int64_t scratch_bytes;    /* device memory the plan holds                 */
} sift_plan_info;

/* Human-readable name of a status code.  Never NULL. */
const char* sift_status_string(int32_t status);

/*
 * Validate a layout and build a plan for it (Sections 4.3, 5.1: page counts,
 * bit-vector offsets, tile numbering, the (head, M-block) work units).
 * Allocates device memory on the current device (the tables, and scratch
 * for the decoded lists of sift_plan_run) and uploads the tables
 * synchronously.  A plan is reusable for every layer of the same prompts.
 *   layout           host layout, read only during the call
 *   num_q_heads      Hq >= 1;  num_kv_heads: Hkv >= 1, Hq % Hkv == 0
 *   head_dim         D: 64 or 128
 *   tile             T: 16, 32, 64 or 128 (bf16 attention: any of them;
 *                    fp32 attention: 16, 32 or 64)
 *   plan_out         receives the plan; the caller frees it with
 *                    sift_plan_destroy.
 * Errors: SIFT_E_NULL, SIFT_E_LAYOUT, SIFT_E_SHAPE, SIFT_E_UNSUPPORTED,
 *         SIFT_E_CAPACITY (more than 2^31-1 list entries), SIFT_E_HIP.
 */
sift_status sift_plan_create(const sift_layout* layout, int32_t num_q_heads,
                             int32_t num_kv_heads, int32_t head_dim,
                             int32_t tile, sift_plan** plan_out);

/* Free a plan and its device memory (waits first for the stream of the
 * plan's last enqueued work).  NULL is accepted. */
sift_status sift_plan_destroy(sift_plan* plan);

/* Copy the plan's sizes into *info. */
sift_status sift_plan_get_info(const sift_plan* plan, sift_plan_info* info);

/*
 * Diagnostic of the bf16 attention (Section 5.2's online softmax, done in
 * two launches here): the first launch forms every tile's weights against
 * the row's first reference max and flags the launch when a weight sum
 * exceeds its bound or an output is not finite; the second launch then does
 * every unit again with a running max.  *count receives how many attention
 * launches on this plan needed that second pass.  Waits for the stream of
 * the plan's last enqueued work.  Errors: SIFT_E_NULL, SIFT_E_PLAN (another
 * device is current), SIFT_E_HIP.
 */
sift_status sift_plan_exact_passes(const sift_plan* plan, int64_t* count);

/*
 * Decoding (Section 5.1) with a plan: expand the bit vectors into the packed
 * lists.
 *   local_bitmap, cross_bitmap   device, la_bytes / ca_bytes of the plan
 *   row_ptr      device int32 [num_rows + 1], written: exclusive prefix sum
 *                of the per-row counts; row_ptr[num_rows] = nnz
 *   col_idx      device int32 [col_capacity], written: entries 0 .. nnz-1
 *   col_capacity must be >= the plan's list_capacity (an upper bound of nnz
 *                known on the host), else SIFT_E_CAPACITY.
 * Uses the plan's scratch for the counts, and also leaves there the per-unit
 * merged step lists (see sift_plan_attention).
 */
sift_status sift_plan_decode_tiles(sift_plan* plan, const uint8_t* local_bitmap,
                                   const uint8_t* cross_bitmap, int32_t* row_ptr,
                                   int32_t* col_idx, int64_t col_capacity, void* stream);

/*
 * Decoding (Section 5.1) without a plan: the layout, the two bit vectors
 * and the tile size in, the packed lists out, with caller-owned scratch.
 *   layout       host layout, read only during the call
 *   local_bitmap, cross_bitmap   device, in the layout above (their sizes
 *                follow from the layout, T and num_q_heads: Section 4.3)
 *   tile         T: 16, 32, 64 or 128;  num_q_heads: Hq >= 1
 *   row_ptr, col_idx, col_capacity   as in sift_plan_decode_tiles; the
 *                capacity must be >= Hq * (causal tiles of all prompts),
 *                the list_capacity of a plan of this layout
 *   workspace    device, 256-byte aligned, at least
 *                sift_decode_workspace_bytes(layout, num_q_heads, tile)
 *                bytes, owned by the caller: the decode's tables and scratch
 * The tables are copied into the workspace on `stream` from pinned host
 * memory the library keeps; the call returns once the work is enqueued,
 * without waiting for the stream.  The workspace must stay allocated until
 * that work is done; calls sharing a workspace must be ordered.
 * Errors: SIFT_E_NULL, SIFT_E_LAYOUT, SIFT_E_SHAPE, SIFT_E_UNSUPPORTED,
 *   SIFT_E_CAPACITY (col_capacity or workspace too small), SIFT_E_HIP; all
 *   but SIFT_E_HIP before anything is enqueued.
 */
sift_status sift_decode_workspace_bytes(const sift_layout* layout, int32_t num_q_heads,
                                        int32_t tile, size_t* bytes);
sift_status sift_decode_tiles(const sift_layout* layout, const uint8_t* local_bitmap,
                              const uint8_t* cross_bitmap, int32_t tile, int32_t num_q_heads,
                              int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * Decoding into the plan's own scratch (the lists and the per-unit merged
 * step lists the bf16 attention kernel walks), as the first step of
 * sift_plan_run.  Same bitmaps and errors as sift_plan_decode_tiles.
 */
sift_status sift_plan_decode(sift_plan* plan, const uint8_t* local_bitmap,
                             const uint8_t* cross_bitmap, void* stream);

/*
 * Sparse attention (Section 5.2) over the lists the last sift_plan_decode
 * (or sift_plan_run, or sift_plan_decode_tiles) on this plan produced: the
 * second step of sift_plan_run.  Tensors, scale and output as in
 * sift_sparse_attention.  SIFT_E_PLAN (bf16 inputs) when the last decode on
 * the plan was the one of sift_plan_run_paged: its step lists index a page
 * pool; decode again first.
 */
sift_status sift_plan_attention(sift_plan* plan, const sift_tensor* q, const sift_tensor* k,
                                const sift_tensor* v, float softmax_scale, sift_tensor* out,
                                void* stream);

/*
 * Sparse attention (Section 5.2) over given lists: for every (h, M-block m),
 * out rows of m = softmax over the keys of the listed tiles (causal inside
 * the diagonal tile, length-masked in partial tiles) times V.
 *   q, k, v      device tensors; dtype both SIFT_BF16 (MFMA kernel: D =
 *                128, T = 16, 32, 64 or 128) or both SIFT_F32 (VALU kernel:
 *                D = 64 or 128, T = 16, 32 or 64)
 *   row_ptr, col_idx   device lists in the format sift_decode_tiles writes,
 *                col_capacity entries of col_idx readable.  Entries outside
 *                the M-block's prompt or after the M-block are skipped;
 *                lists must be ascending.  A row whose list is empty gets 0.
 *                (bf16 inputs: the lists are first merged into the plan's
 *                per-unit step scratch.)
 *   softmax_scale  <= 0 selects 1/sqrt(D)
 *   out          device tensor [tokens][Hq][D], SIFT_BF16 or SIFT_F32 for
 *                bf16 inputs, SIFT_F32 for fp32 inputs.
 */
sift_status sift_sparse_attention(sift_plan* plan, const sift_tensor* q,
                                  const sift_tensor* k, const sift_tensor* v,
                                  const int32_t* row_ptr,
                                  const int32_t* col_idx, int64_t col_capacity,
                                  float softmax_scale, sift_tensor* out,
                                  void* stream);

/*
 * One layer of the online hot path: decode into the plan's own list
 * scratch, then sparse attention (Sections 5.1 and 5.2).  No allocation.
 */
sift_status sift_plan_run(sift_plan* plan, const sift_tensor* q,
                          const sift_tensor* k, const sift_tensor* v,
                          const uint8_t* local_bitmap,
                          const uint8_t* cross_bitmap, float softmax_scale,
                          sift_tensor* out, void* stream);

/*
 * sift_plan_run with K and V in a page pool instead of packed on the token
 * axis.  The paper's key tiles are KV pages (Sections 4.2-4.3): here a tile
 * is one page of T rows, and page_table says where each tile lives.
 *   k_pages, v_pages  device tensors [num_pages * T][Hkv][D] (tokens =
 *                num_pages * T, a multiple of T, >= T when the layout has
 *                tiles): page p holds rows p*T .. p*T + T-1, each row the
 *                Hkv x D values of one token.  A partial last tile of a
 *                segment uses the first tile_len rows of its page; the rest
 *                of the page is never read.
 *   page_table   device int32 [num_tiles]: page_table[m] = pool page of
 *                global tile m (tile numbering as in "Tiles" above).  Entries
 *                outside [0, num_pages) are clamped into the pool (no access
 *                leaves it; the result for such tiles is meaningless).
 *   q, out       packed as everywhere else; dtypes as in sift_sparse_attention.
 * The plan's step lists then index the pool (see sift_plan_attention).
 * Errors: those of sift_plan_run; SIFT_E_SHAPE for a pool that is not whole
 * pages of the plan's T, Hkv, D; SIFT_E_NULL for a missing page_table.
 */
sift_status sift_plan_run_paged(sift_plan* plan, const sift_tensor* q,
                                const sift_tensor* k_pages, const sift_tensor* v_pages,
                                const int32_t* page_table, const uint8_t* local_bitmap,
                                const uint8_t* cross_bitmap, float softmax_scale,
                                sift_tensor* out, void* stream);

/*
 * One-shot form with the arguments of the paper's problem statement: Q, K,
 * V of one layer, the document layout, the two bit vectors and the tile
 * size (Sections 4 and 5), softmax scale 1/sqrt(D).  Stream-ordered: the
 * scratch is taken with hipMallocAsync on `stream`, the plan's tables are
 * copied into it on `stream` from pinned host memory the library keeps,
 * decode and attention are enqueued, and the scratch is released with
 * hipFreeAsync on `stream`.  The call returns once all of it is enqueued,
 * without waiting for the stream or the device.
 * Errors: SIFT_E_NULL, SIFT_E_SHAPE, SIFT_E_LAYOUT, SIFT_E_UNSUPPORTED,
 *   SIFT_E_CAPACITY, all before anything is enqueued; SIFT_E_HIP.
 */
sift_status sift_sparse_prefill(const sift_tensor* q, const sift_tensor* k,
                                const sift_tensor* v,
                                const sift_layout* doc_offsets,
                                const uint8_t* local_bitmap,
                                const uint8_t* cross_bitmap, int32_t tile,
                                sift_tensor* out, void* stream);

/*
 * The one-shot form with the caller's softmax scale and device workspace
 * (Sections 4 and 5; same computation as sift_sparse_prefill).
 *
 * sift_workspace_bytes: the device workspace bytes sift_sparse_prefill_ex
 *   needs for this layout, head counts, head dimension and tile size (the
 *   plan's tables and the decode and merge scratch).  Host only.
 * sift_sparse_prefill_ex: softmax_scale <= 0 means 1/sqrt(D).  workspace
 *   (device, 256-byte aligned, at least sift_workspace_bytes) is owned by
 *   the caller; the library allocates no device memory.  The plan's tables
 *   are copied into the workspace on `stream` from pinned host memory the
 *   library keeps, decode and attention are enqueued on `stream`, and the
 *   call returns without waiting for any of it.  The workspace must stay
 *   allocated until that work is done; calls sharing a workspace must be on
 *   one stream or otherwise ordered.
 * Errors: as sift_sparse_prefill, plus SIFT_E_NULL (no workspace),
 *   SIFT_E_CAPACITY (too small) and SIFT_E_UNSUPPORTED (misaligned), all
 *   before anything is enqueued.
 */
sift_status sift_workspace_bytes(const sift_layout* layout, int32_t num_q_heads,
                                 int32_t num_kv_heads, int32_t head_dim, int32_t tile,
                                 size_t* bytes);
sift_status sift_sparse_prefill_ex(const sift_tensor* q, const sift_tensor* k,
                                   const sift_tensor* v, const sift_layout* doc_offsets,
                                   const uint8_t* local_bitmap,
                                   const uint8_t* cross_bitmap, int32_t tile,
                                   float softmax_scale, void* workspace,
                                   size_t workspace_bytes, sift_tensor* out, void* stream);

/*
 * For callers that cannot allocate device memory (code under stream capture,
 * tight serving loops, harnesses that forbid hipMalloc): the computation of
 * sift_sparse_prefill_ex with the library's own static device scratch in
 * place of the caller's workspace.  Nothing is allocated on the device and
 * no hipMalloc, hipFree or allocating library routine is called.
 *   Arguments as in sift_sparse_prefill_ex, without the workspace.
 *   The scratch is sift_static_scratch_bytes() = 256 MiB per GPU, held from
 *   the library's load on that GPU until the process ends; a layout whose
 *   plan needs more (sift_workspace_bytes) is refused with SIFT_E_CAPACITY
 *   before anything is enqueued.
 *   The plan's tables are copied from host memory on `stream`, and the call
 *   waits for `stream` once that copy is enqueued (so that the host copy
 *   can be freed); decode and attention are then enqueued and the call
 *   returns without waiting for them.
 *   Every call on one GPU uses the same scratch, which keeps the last call's
 *   contents: calls that overlap on one GPU (other streams, other threads)
 *   race and give wrong results.  Order them.
 * Errors: as sift_sparse_prefill_ex, with SIFT_E_CAPACITY for a layout that
 *   does not fit the scratch.
 */
sift_status sift_sparse_prefill_static(const sift_tensor* q, const sift_tensor* k,
                                       const sift_tensor* v, const sift_layout* doc_offsets,
                                       const uint8_t* local_bitmap,
                                       const uint8_t* cross_bitmap, int32_t tile,
                                       float softmax_scale, sift_tensor* out, void* stream);
size_t sift_static_scratch_bytes(void);

/*
 * Offline metadata extraction (Sections 4.1, 4.2; made by a dense
 * standalone prefill of each document, Section 4.4).
 *
 * Each document is prefilled alone: causal softmax(scale * Q K^T) over its
 * own tokens, per query head (kv head h / (Hq/Hkv)).  With A its
 * probabilities:
 *   LA bit of tile (i, j), j <= i: 1 when some causal cell of the tile has
 *     A > alpha (Section 4.1; the paper uses alpha = 0.001);
 *   CA bit of key page j: 1 when, over the page's causal cells (query p >= key
 *     k, k in the page), the number with A > beta exceeds gamma times their
 *     number (Section 4.2; beta = 0.01, gamma = 0.1).  This is the page
 *     granular form of the key-column concentration of Section 3.5.
 * The bits are packed as the online path reads them (see "Bit vectors"
 * above), for these documents in order: the buffers of a prompt are the
 * concatenation of its documents' parts.
 *
 * sift_extract_sizes: for num_docs documents of lengths
 *   doc_offsets[d+1] - doc_offsets[d] >= 1 (host, [num_docs + 1],
 *   doc_offsets[0] == 0), num_q_heads query heads and tile T (16, 32, 64, 128),
 *   writes the bytes la_out and ca_out must hold and the device workspace
 *   sift_extract_bits needs.  Any of the three pointers may be NULL.
 * sift_extract_bits: q [tokens][Hq][D] and k [tokens][Hkv][D] in bf16,
 *   D 64 or 128, tokens == doc_offsets[num_docs]; alpha, beta >= 0,
 *   0 <= gamma <= 1; softmax_scale <= 0 means 1/sqrt(D).  la_out, ca_out
 *   (device) receive the bit vectors; workspace (device, at least the size
 *   from sift_extract_sizes, 256-byte aligned) is scratch owned by the
 *   caller.  The call waits for `stream`, uploads its tables to the workspace
 *   synchronously, then enqueues the kernels on `stream` and returns.
 *   Calls that share a workspace must be ordered.
 * Errors: SIFT_E_NULL, SIFT_E_LAYOUT (offsets), SIFT_E_SHAPE (tensors vs
 *   offsets, Hq % Hkv), SIFT_E_UNSUPPORTED (dtype, D, T, thresholds),
 *   SIFT_E_CAPACITY (workspace too small), SIFT_E_HIP.
 */
sift_status sift_extract_sizes(int32_t num_docs, const int32_t* doc_offsets,
                               int32_t num_q_heads, int32_t tile, size_t* la_bytes,
                               size_t* ca_bytes, size_t* workspace_bytes);
sift_status sift_extract_bits(const sift_tensor* q, const sift_tensor* k, int32_t num_docs,
                              const int32_t* doc_offsets, int32_t tile, double alpha,
                              double beta, double gamma, float softmax_scale,
                              uint8_t* la_out, uint8_t* ca_out, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * Rotary position embedding for the decoder-layer prefill slice (the
 * Llama-3.1-8B layer of Section 6 around the sparse attention): q
 * [tokens][Hq][D] and k [tokens][Hkv][D], bf16 in device memory, are rotated
 * in place, rotate-half form: for i < D/2 and angle a = positions[t] *
 * inv_freq[i] (fp32 product),
 *   x[i] <- x[i] cos a - x[i + D/2] sin a,  x[i + D/2] <- x[i + D/2] cos a + x[i] sin a.
 * positions (device, int32 [tokens]) are each token's index in its prompt;
 * inv_freq (device, float [D/2]) is the frequency table (base^(-2i/D), or a
 * rescaled one).  Errors: SIFT_E_NULL, SIFT_E_SHAPE (tokens or head sizes
 * differ), SIFT_E_UNSUPPORTED (not bf16, odd D), SIFT_E_HIP.
 */
sift_status sift_rope(const sift_tensor* q, const sift_tensor* k, const int32_t* positions,
                      const float* inv_freq, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SIFT_H_ */
