/*
 * wavepp_kda.h -- C ABI of the KDA part of libwavepp_attn.so: chunked prefill of a Kimi Delta
 * Attention (gated delta-rule) layer that resumes from a recurrent-state snapshot and writes the
 * snapshot at the chunk boundary, for AMD gfx950 (MI355X).
 *
 * The operation (Preliminaries, "Transformer Architectures", Eq. 1-3): a linear-attention layer
 * keeps, per head, a d_k x d_v state S that summarizes the prefix.  For each token t, with a
 * per-channel decay alpha_t (d_k entries), a scalar write strength beta_t, key k_t, value v_t and
 * query q_t,
 *     S_t = (I - beta_t k_t k_t^T) Diag(alpha_t) S_{t-1} + beta_t k_t v_t^T,     o_t = S_t^T q_t.
 * Resume semantics (Preliminaries, "Reuse", on linear attention): a request with r cached tokens
 * can resume only from S_r itself.  Chunk r of a wave therefore starts from the snapshot in slot
 * state_in[r] (or from the zero state), runs its c_r tokens, and leaves S_{r + c_r} in slot
 * state_out[r]; the next chunk of that request resumes from there.  One snapshot of one layer
 * holds num_heads * d_k * d_v fp32 values (Eq. 4 with b = 4 bytes).
 *
 * Layouts (row-major, contiguous; tokens packed by request in order, cu_r = c_0 + ... + c_{r-1}):
 *   q, k      [T][num_heads][head_dim_k]   bf16
 *   v         [T][num_heads][head_dim_v]   bf16
 *   alpha     [T][num_heads][head_dim_k]   fp32, each in [0, 1]
 *   beta      [T][num_heads]               fp32, each in [0, 1]
 *   state_pool[num_state_slots][num_heads][head_dim_k][head_dim_v]   fp32
 *   out       [T][num_heads][head_dim_v]   bf16
 *
 * Numerics: chunkwise form in 64-token blocks with bf16 MFMA operands and fp32 accumulation; the
 * state is carried in fp32 and written to the snapshot in fp32; outputs are rounded to bf16
 * (nearest even).
 *
 * Call order on one stream, per wave: wavepp_kda_plan (host only) -> wavepp_kda_upload (enqueues
 * the plan's metadata into the workspace) -> wavepp_kda_chunked_prefill (once per KDA layer, each
 * layer with its own tensors and state pool).
 *
 * Ownership: the caller owns every device buffer and the stream; the library never allocates
 * device memory.  A plan is an immutable host object owned by the library until
 * wavepp_kda_destroy; the host arrays passed to wavepp_kda_plan are copied.
 *
 * Errors: the wavepp_status codes of wavepp_attn.h.  Invalid input is rejected on the host before
 * anything is enqueued, with details in wavepp_last_error().  Device-side faults are asynchronous
 * and surface at the caller's next synchronization.
 */
#ifndef WAVEPP_KDA_H
#define WAVEPP_KDA_H

#include "wavepp_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Static shape of one KDA layer.  Supported: head_dim_k = head_dim_v = 128, num_heads >= 1. */
typedef struct {
  int32_t num_heads;
  int32_t head_dim_k;
  int32_t head_dim_v;
  int32_t num_state_slots;   /* slots in the snapshot pool */
} wavepp_kda_shape;

/* One wave, HOST memory, copied by wavepp_kda_plan.
 *   chunk_lens[r] = c_r >= 0; c_r = 0 is an idle lane that reads and writes nothing.
 *   state_in[r]   = slot to resume from, in [0, num_state_slots), or -1 for the zero state.
 *   state_out[r]  = slot that receives the final state, in [0, num_state_slots).
 * Among requests with c_r > 0, the state_out slots must be distinct, and no state_out slot may be
 * another request's state_in slot (state_in[r] == state_out[r], resuming in place, is allowed);
 * otherwise WAVEPP_EALIAS. */
typedef struct {
  int32_t num_requests;
  const int32_t* chunk_lens;
  const int32_t* state_in;
  const int32_t* state_out;
} wavepp_kda_batch;

typedef struct wavepp_kda_plan_s wavepp_kda_plan_t;

typedef struct {
  int64_t total_tokens;      /* T */
  int32_t num_items;         /* requests with c_r > 0; the kernel runs one workgroup per (item, head) */
  int32_t block_tokens;      /* tokens per block of the chunkwise form (64) */
  int64_t metadata_bytes;
  int64_t workspace_bytes;
} wavepp_kda_info;

/* Validate the wave and build the work list (longest chunks first).  Host only. */
int wavepp_kda_plan(const wavepp_kda_shape* shape, const wavepp_kda_batch* batch, wavepp_kda_plan_t** out);

/* Device workspace the plan needs (metadata only), 256-byte aligned. */
size_t wavepp_kda_workspace_bytes(const wavepp_kda_plan_t* plan);

int wavepp_kda_get_info(const wavepp_kda_plan_t* plan, wavepp_kda_info* info);

/* Enqueue on `stream` the copy of the plan's metadata into `workspace` (device memory of at least
 * wavepp_kda_workspace_bytes, 256-byte aligned) from a library-owned pinned buffer, by a small copy
 * kernel on `stream`.  The library records which plan each workspace address was given last (see
 * wavepp_kda_chunked_prefill).  Errors: WAVEPP_EINVAL, WAVEPP_ENOSPACE, WAVEPP_EHIP. */
int wavepp_kda_upload(const wavepp_kda_plan_t* plan, void* workspace, size_t ws_bytes, hipStream_t stream);

/* Chunked prefill of one KDA layer.  Device pointers with the layouts above; q, k, v, alpha, beta,
 * state_pool and out 16-byte aligned.  Reads the snapshots named by state_in and writes out and
 * the snapshots named by state_out; every other slot and every other byte is left untouched.  A
 * snapshot slot that a request resumes from but does not write keeps its contents (Preliminaries,
 * "Reuse": a chunk resumes only from the exact snapshot of its prefix).  Requires that the last
 * upload into `workspace` was of `plan`: otherwise WAVEPP_EINVAL and nothing is enqueued (the
 * kernel also checks the plan's serial against the workspace header and writes nothing on a
 * mismatch).  Deterministic: repeated calls give bit-identical results. */
int wavepp_kda_chunked_prefill(const wavepp_kda_plan_t* plan, const void* q, const void* k, const void* v,
                               const float* alpha, const float* beta, float* state_pool, void* out,
                               void* workspace, size_t ws_bytes, hipStream_t stream);

void wavepp_kda_destroy(wavepp_kda_plan_t* plan);

#ifdef __cplusplus
}
#endif

#endif /* WAVEPP_KDA_H */
