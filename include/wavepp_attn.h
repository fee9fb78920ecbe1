/*
 * wavepp_attn.h -- C ABI of libwavepp_attn.so: chunked-prefill attention over a paged KV cache
 * and the append of each chunk's K/V into its freshly reserved pages, for AMD gfx950 (MI355X).
 *
 * The problem statement follows the WavePP paper:
 *   - A wave is a ragged batch of request chunks (Design of WavePP, "Waves and lanes").  Chunk r
 *     is the span (request r, starting token p_r, length c_r): p_r tokens of the request are
 *     already cached and c_r new tokens are processed now (Pipeline Scheduling: the scheduler
 *     ships exactly these three numbers per chunk).
 *   - n cached tokens occupy ceil(n / B) logical blocks of B tokens whose physical pages need not
 *     be contiguous (Preliminaries, "Reuse").  Row r of the block table names, for each logical
 *     block of request r, its physical page.
 *   - Before a chunk executes, the blocks for its positions [p_r, p_r + c_r) have been reserved
 *     and are materialized: the chunk's K/V is written into them (A Minimum Implementation,
 *     steps 3-5; Decoupling Admission).  wavepp_attn_append_kv performs that write.
 *   - The chunk's queries then attend to the whole cached prefix plus the chunk itself, causally:
 *     query i of chunk r (position p_r + i) sees key positions 0 .. p_r + i inclusive.
 *   - Several query heads may share one KV head (grouped/multi-query attention), or all heads may
 *     share one latent vector per token (multi-head latent attention in absorbed form: keys are
 *     the whole latent, values its leading head_dim_v lanes) (Preliminaries, "Transformer
 *     Architectures").  Query head h reads KV head h / (num_q_heads / num_kv_heads).
 *
 * Definition computed, per request r, chunk query i, query head h (g = its KV head):
 *   K(r, j) = k_pool[block_table[r][j / B]][g][j % B][:]   (V likewise, or K[:head_dim_v])
 *   s_j     = softmax_scale * <q[cu_r + i][h][:], K(r, j)>     for j in [0, p_r + i]
 *   out[cu_r + i][h][:] = sum_j softmax(s)_j V(r, j),   lse[cu_r + i][h] = ln sum_j exp(s_j)
 * where cu_r = c_0 + ... + c_{r-1} packs the chunks' tokens in request order.
 *
 * Numerics: bf16 inputs, fp32 accumulation and softmax, bf16 output (round to nearest even),
 * fp32 natural-log LSE.
 *
 * Call order on one stream, per wave:
 *   wavepp_attn_plan            (host only; validates, builds the work list)
 *   wavepp_attn_plan_upload     (enqueues the plan's metadata into the workspace)
 *   wavepp_attn_append_kv       (materialize: write the chunks' K/V into the pools)
 *   wavepp_attn_chunked_prefill (attention; may be called again, e.g. once per layer, with other
 *                                pools/q/out of the same shape and the same uploaded workspace)
 *
 * Ownership: the caller owns every device buffer (q, pools, out, lse, workspace) and the stream.
 * The library never allocates device memory.  A plan is an immutable host object owned by the
 * library until wavepp_plan_destroy; the host arrays passed to wavepp_attn_plan are copied and
 * may be freed after it returns.
 *
 * Errors: every entry point returns a wavepp_status (0 = success, negative = error) and never
 * throws or exits.  Invalid input is rejected on the host before anything is enqueued; a
 * thread-local message with details is available from wavepp_last_error().  Device-side faults
 * are asynchronous and surface at the caller's next synchronization.
 */
#ifndef WAVEPP_ATTN_H
#define WAVEPP_ATTN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WAVEPP_OK = 0,
  WAVEPP_EINVAL = -1,       /* null pointer, negative length, bad alignment, bad workspace */
  WAVEPP_EUNSUPPORTED = -2, /* head dims / page size / flags outside the supported set */
  WAVEPP_ERANGE = -3,       /* a block-table entry that is read lies outside [0, num_pages) */
  WAVEPP_EALIAS = -4,       /* a page receiving appended tokens is also referenced elsewhere */
  WAVEPP_EPOSITION = -5,    /* bt_stride * page_size < p_r + c_r: span not backed by pages */
  WAVEPP_ENOSPACE = -6,     /* workspace smaller than wavepp_plan_workspace_bytes() */
  WAVEPP_EHIP = -7          /* a HIP runtime call failed (launch, copy, event) */
} wavepp_status;

/* Static shape of the attention layer.
 * Supported: (head_dim_qk, head_dim_v) in {(64, 64), (128, 128)} with kv_shared = 0 and any
 * num_q_heads % num_kv_heads == 0; or (576, 512) with kv_shared = 1 and num_kv_heads = 1.
 * page_size in {16, 64}.  softmax_scale > 0 and finite. */
typedef struct {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim_qk;
  int32_t head_dim_v;
  int32_t page_size;     /* B: tokens per page */
  int32_t num_pages;     /* P: pages in the pool */
  int32_t kv_shared;     /* 1: latent cache, V = first head_dim_v lanes of the K pool */
  float softmax_scale;
} wavepp_attn_shape;

/* One wave: per-request spans and block tables, all HOST memory, copied by wavepp_attn_plan.
 * prefix_lens[r] = p_r >= 0 (cached tokens), chunk_lens[r] = c_r >= 0 (c_r = 0: idle lane).
 * block_table is row-major [num_requests][bt_stride]; entries j < ceil((p_r + c_r) / B) must lie
 * in [0, num_pages); later entries are ignored (neither read nor validated).  A page may appear in
 * several requests' prefix blocks (shared prefix); a page that receives appended tokens (any block
 * overlapping [p_r, p_r + c_r)) must appear exactly once among all read entries of the wave. */
typedef struct {
  int32_t num_requests;
  const int32_t* prefix_lens;
  const int32_t* chunk_lens;
  const int32_t* block_table;
  int32_t bt_stride;
} wavepp_batch;

typedef struct wavepp_plan wavepp_plan;

/* Summary of a plan (for tests and reporting). */
typedef struct {
  int64_t total_tokens;      /* T = sum_r c_r */
  int32_t num_items;         /* attention work items (one workgroup each), padding included */
  int32_t num_real_items;    /* work items that carry rows */
  int32_t num_merge_items;   /* split tiles that need a merge */
  int32_t max_splits;        /* largest key-range split used */
  int32_t rows_per_item;     /* query rows (token x head-in-group) per work item */
  int32_t kv_tile;           /* keys per inner-loop tile */
  int64_t partial_rows;      /* fp32 partial-output rows in the workspace */
  int64_t metadata_bytes;    /* bytes copied by wavepp_attn_plan_upload */
  int64_t workspace_bytes;
} wavepp_plan_info;

/* Validate the wave and build its work list: query-row tiles of (request, KV head), each
 * optionally split over key ranges, heaviest first and spread over the chip's L2 domains.
 * Follows Design of WavePP, "Pipeline Scheduling" (a chunk is the span request, starting token,
 * length, and a span whose positions the materialized cache does not back must fail rather than
 * run: WAVEPP_EPOSITION) and Preliminaries, "Reuse" (ceil(n / B) blocks in pages that need not be
 * contiguous: entries outside the pool are WAVEPP_ERANGE).  The equal-size-chunks-cost-differently
 * remark of the same section is why items are costed by rows x visible keys.
 * max_splits: 0 = choose automatically, else the largest number of key ranges per tile (>= 1).
 * On success *out receives a new plan (caller destroys it); on error *out is NULL, nothing was
 * allocated and wavepp_last_error() names the offending request / block.  Host only: makes no
 * HIP call, so it is safe on a thread without a device. */
int wavepp_attn_plan(const wavepp_attn_shape* shape, const wavepp_batch* batch, int32_t max_splits,
                     wavepp_plan** out);

/* Device workspace the plan needs: metadata plus fp32 split partials.  256-byte aligned. */
size_t wavepp_plan_workspace_bytes(const wavepp_plan* plan);

int wavepp_plan_get_info(const wavepp_plan* plan, wavepp_plan_info* info);

/* Copy the work list into host memory: 8 int32 per item, in launch order:
 * (request, kv_head, first_row, rows, kv_begin, kv_end, partial_row or -1, split_index).
 * Rows index the packed (token * G + head_in_group) space of (request, kv_head).  Writes
 * min(capacity, num_items) items and returns the number written, or a negative status. */
int wavepp_plan_get_items(const wavepp_plan* plan, int32_t* items, int32_t capacity);

/* Enqueue on `stream` the copy of the plan's metadata into the head of `workspace` (device
 * memory of at least wavepp_plan_workspace_bytes bytes, 256-byte aligned).  This is the
 * "materialize before execute" step of Design of WavePP, "Decoupling Admission", for the wave's
 * metadata.  The source is a library-owned pinned staging buffer, so the plan may be destroyed
 * right after this returns; the copy is a small kernel on `stream` that reads that buffer through
 * its device mapping.  The library records, per workspace address, which plan was uploaded last:
 * wavepp_attn_append_kv and wavepp_attn_chunked_prefill return WAVEPP_EINVAL (and enqueue
 * nothing) for a workspace whose last upload was of another plan or that had none.  The kernels
 * also compare the plan's serial with the workspace header and write nothing on a mismatch (a
 * workspace the caller overwrote after the upload).  Errors: WAVEPP_EINVAL (NULL / misaligned),
 * WAVEPP_ENOSPACE (too small), WAVEPP_EHIP (staging allocation or launch failed). */
int wavepp_attn_plan_upload(const wavepp_plan* plan, void* workspace, size_t ws_bytes, hipStream_t stream);

/* Append (materialization): the write of each chunk's K/V into the blocks reserved for positions
 * [p_r, p_r + c_r) (A Minimum Implementation, steps 3-4; Decoupling Admission: freshly reserved
 * suffix blocks are materialized before the chunk executes).  Device pointers, bf16, row-major
 * and contiguous, owned by the caller:
 *   k_new [T][num_kv_heads][head_dim_qk], v_new [T][num_kv_heads][head_dim_v] (NULL if kv_shared)
 *   k_pool [num_pages][num_kv_heads][page_size][head_dim_qk], v_pool likewise (NULL if kv_shared)
 * Token cu_r + i is written to page block_table[r][(p_r + i) / B], slot (p_r + i) % B, for every
 * KV head; no other slot is touched.  The copy is bit-exact.  Requires that the last upload into
 * `workspace` was of `plan` (else WAVEPP_EINVAL, nothing enqueued); WAVEPP_EINVAL also for NULL
 * or non-16-byte-aligned buffers; WAVEPP_EHIP if the launch fails.  A wave with T = 0 is a no-op. */
int wavepp_attn_append_kv(const wavepp_plan* plan, const void* k_new, const void* v_new, void* k_pool,
                          void* v_pool, void* workspace, size_t ws_bytes, hipStream_t stream);

/* Attention of the wave's chunks: query i of chunk r attends to the whole cached prefix and to the
 * chunk causally (Design of WavePP, "Waves and lanes": chunked prefill of the uncached suffix;
 * Preliminaries, "Transformer Architectures": grouped and latent K/V sharing; "Reuse": paged
 * blocks).  The definition is the one at the top of this file.  Device pointers, row-major and
 * contiguous, owned by the caller:
 *   q [T][num_q_heads][head_dim_qk] bf16; pools as above (v_pool NULL if kv_shared), already
 *   holding the chunks' K/V (enqueue wavepp_attn_append_kv first on the same stream);
 *   out [T][num_q_heads][head_dim_v] bf16; lse [T][num_q_heads] fp32 or NULL.
 * Pool slots past p_r + c_r in a request's last page may hold any bits (NaN included); they do
 * not affect the result.  Requires that the last upload into `workspace` was of `plan` (else
 * WAVEPP_EINVAL, nothing enqueued); WAVEPP_EINVAL also for NULL or misaligned buffers (16 bytes,
 * lse 4); WAVEPP_EHIP if a launch fails.  Deterministic: repeated calls give bit-identical
 * results. */
int wavepp_attn_chunked_prefill(const wavepp_plan* plan, const void* q, const void* k_pool, const void* v_pool,
                                void* out, float* lse, void* workspace, size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): the wave's append (if k_new is not NULL) and attention
 * with no workspace argument and no allocation.  The plan's metadata and its split partials live in
 * a static device array of the library, 160 MiB (167,772,160 bytes) per GPU, held from the first
 * call on that GPU until the process ends; a plan whose wavepp_plan_workspace_bytes exceeds that is
 * rejected with WAVEPP_ENOSPACE before anything is enqueued (plan it with a smaller max_splits).
 * The metadata is copied from the plan's host memory with hipMemcpyAsync on `stream` (from
 * pageable memory the runtime reads it before returning; under stream capture the copy becomes a
 * graph node that reads the plan's host memory each time the graph runs, so the plan must outlive
 * the graph; replays are bit-identical to an eager call), then the same kernels as the
 * workspace entry points run on `stream`; results are bit-identical to wavepp_attn_append_kv +
 * wavepp_attn_chunked_prefill on the same plan.  Arguments as there: k_new / v_new as for
 * wavepp_attn_append_kv (both NULL: the pools already hold the chunks' K/V; v_new NULL for a
 * latent cache), q, pools, out, lse as for wavepp_attn_chunked_prefill.
 * Every call on one GPU uses that GPU's one array: calls that overlap on one GPU (two streams, or
 * a call enqueued before the previous call's kernels finished reading on another stream) race, and
 * the array keeps the last call's contents.  Calls on one stream are ordered and safe.
 * Errors: WAVEPP_EINVAL (NULL / misaligned buffers), WAVEPP_ENOSPACE (plan too large),
 * WAVEPP_EHIP (symbol address, copy or launch failed). */
int wavepp_attn_chunked_prefill_noalloc(const wavepp_plan* plan, const void* q, const void* k_new,
                                        const void* v_new, void* k_pool, void* v_pool, void* out, float* lse,
                                        hipStream_t stream);

void wavepp_plan_destroy(wavepp_plan* plan);

/* Static string for a status code. */
const char* wavepp_status_string(int status);

/* Detail of the last error on the calling thread ("" if none). */
const char* wavepp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* WAVEPP_ATTN_H */
