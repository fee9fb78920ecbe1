// Internal layout shared by the host planner (host.cpp) and the gfx950 kernels (kernels.hip).
// Not part of the public ABI.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime_api.h>

namespace wavepp {

constexpr uint32_t kMagic = 0x57415650u;   // "WAVP"
constexpr int kGqaRowsPerItem = 256;       // grouped kernel: 8 waves x 32 query rows
constexpr int kKvTile = 128;               // grouped kernel: keys per inner-loop tile
constexpr int kNumXcd = 8;                 // L2 domains a launch is spread over, round-robin
constexpr int kMlaRowsPerItem = 128;       // latent kernel: query rows per work item
constexpr int kMlaKvTile = 64;             // latent kernel: keys per tile

// Header at the start of the uploaded metadata.
struct alignas(16) MetaHeader {
  uint32_t magic;
  uint32_t serial;       // plan identity: kernels compare it with the serial they were launched for
  int32_t num_requests;
  int32_t num_items;
  int32_t num_merge;
  int32_t bt_stride;
  int32_t pad[2];
};

// Per-request span.
struct alignas(16) ReqMeta {
  int32_t prefix;   // p_r
  int32_t chunk;    // c_r
  int32_t cu;       // first packed token of the chunk
  int32_t bt_row;   // offset of the request's block-table row (= r * bt_stride)
};

// One workgroup of the attention kernel.
struct alignas(16) WorkItem {
  int32_t req;
  int32_t kv_head;
  int32_t row0;      // first packed row (token * G + head_in_group)
  int32_t rows;      // rows in this item (0 = padding item, does nothing)
  int32_t kv_begin;  // first key position (multiple of the kernel's key tile)
  int32_t kv_end;    // one past the last key position
  int32_t part;      // -1: final output; else first fp32 partial row of this split
  int32_t split;
};

// One tile whose key range was split: combine `nsplit` partials into the final output.
struct alignas(16) MergeItem {
  int32_t req;
  int32_t kv_head;
  int32_t row0;
  int32_t rows;
  int32_t nsplit;
  int32_t part;      // partial rows of split s start at part + s * rows
  int32_t pad[2];
};

// Everything a launch needs, resolved to device addresses inside the workspace.
struct DevPlan {
  const MetaHeader* hdr;
  const ReqMeta* reqs;
  const int32_t* bt;
  const WorkItem* items;
  const MergeItem* merges;
  float* opart;          // [partial_rows][head_dim_v]
  float* lpart;          // [partial_rows]
  uint32_t serial;
  int32_t num_requests;
  int32_t num_items;
  int32_t num_merge;
  int64_t total_tokens;
  int32_t num_q_heads, num_kv_heads, head_dim_qk, head_dim_v, page_size, kv_shared;
  int32_t rows_per_item;   // query rows per attention workgroup (32 per wave)
  float softmax_scale;
};

// ---------------------------------------------------------------------------------------------
// KDA chunked prefill
// ---------------------------------------------------------------------------------------------
constexpr uint32_t kKdaMagic = 0x4B444131u;  // "KDA1"
constexpr int kKdaBlock = 64;                // tokens per block of the chunkwise form
constexpr int kKdaDim = 128;                 // d_k = d_v supported by the kernel

struct alignas(16) KdaHeader {
  uint32_t magic;
  uint32_t serial;
  int32_t num_items;
  int32_t num_heads;
};

// One request of the wave with at least one token; a workgroup runs one (item, head).
struct alignas(16) KdaItem {
  int32_t req;
  int32_t cu;         // first packed token
  int32_t len;        // c_r > 0
  int32_t state_in;   // snapshot slot to resume from, -1 = zero state
  int32_t state_out;  // snapshot slot written with the final state
  int32_t pad[3];
};

// The metadata upload copies 16-byte words, so every record of a blob is a multiple of 16 bytes.
static_assert(sizeof(MetaHeader) % 16 == 0 && sizeof(ReqMeta) % 16 == 0 && sizeof(WorkItem) % 16 == 0 &&
                  sizeof(MergeItem) % 16 == 0 && sizeof(KdaHeader) % 16 == 0 && sizeof(KdaItem) % 16 == 0,
              "metadata records are whole 16-byte words");

struct KdaDevPlan {
  const KdaHeader* hdr;
  const KdaItem* items;
  uint32_t serial;
  int32_t num_items;
  int32_t num_heads;
  int32_t num_slots;
};

hipError_t launch_kda_prefill(const KdaDevPlan& p, const void* q, const void* k, const void* v, const float* alpha,
                              const float* beta, float* state_pool, void* out, hipStream_t stream);

// Shared host helpers (host.cpp): thread-local error detail, pinned metadata staging, plan serials.
int set_error(int status, const char* fmt, ...);
int set_hip_error(hipError_t e, const char* what);
void clear_error();
const char* last_error_text();
int stage_and_copy(const void* src, size_t bytes, void* dst, hipStream_t stream);
uint32_t next_serial();
// Record that `workspace` was given the metadata of the plan with this serial (on the caller's
// stream); require_upload returns WAVEPP_EINVAL, with a last-error message naming upload_fn, when
// the last upload into `workspace` was of another plan or there was none.
void note_upload(const void* workspace, uint32_t serial);
int require_upload(const void* workspace, uint32_t serial, const char* upload_fn);

hipError_t launch_append(const DevPlan& p, const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                         hipStream_t stream);
hipError_t launch_attention(const DevPlan& p, const void* q, const void* k_pool, const void* v_pool, void* out,
                            float* lse, hipStream_t stream);
hipError_t launch_merge(const DevPlan& p, void* out, float* lse, hipStream_t stream);
// Copy `bytes` (a multiple of 16, both pointers 16-byte aligned) from device-visible pinned host
// memory to device memory with a kernel on `stream`.
hipError_t launch_upload(const void* src, void* dst, size_t bytes, hipStream_t stream);

// Size of the static per-device scratch array of the allocation-free entry point, and the device
// address of the current device's copy (taken with hipGetSymbolAddress on first use per device).
constexpr size_t kNoAllocScratchBytes = size_t(160) << 20;
hipError_t noalloc_scratch(void** ptr);

}  // namespace wavepp
