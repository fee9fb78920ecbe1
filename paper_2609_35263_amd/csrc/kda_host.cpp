// Host side of the KDA chunked prefill: validation of the wave, the work list and the launch.
//
// Resume semantics follow the paper's statement that a recurrent layer resumes only from the exact
// state at its prefix boundary (Preliminaries, "Reuse"): each request names the snapshot slot it
// resumes from and the slot that receives its state at the chunk boundary.  Because a wave's
// workgroups run concurrently, a slot written by one request may not be read or written by another.
#include "wavepp_kda.h"
#include "internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <numeric>
#include <vector>

using namespace wavepp;

struct wavepp_kda_plan_s {
  wavepp_kda_shape shape;
  int64_t total_tokens = 0;
  uint32_t serial = 0;
  std::vector<KdaItem> items;
  std::vector<unsigned char> blob;
  size_t off_items = 0;
  size_t workspace_bytes = 0;
};

namespace {

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int check_ws(const wavepp_kda_plan_t* plan, void* ws, size_t ws_bytes) {
  if (!ws) return set_error(WAVEPP_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return set_error(WAVEPP_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < plan->workspace_bytes)
    return set_error(WAVEPP_ENOSPACE, "workspace has %zu bytes, plan needs %zu", ws_bytes, plan->workspace_bytes);
  return WAVEPP_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

extern "C" {

int wavepp_kda_plan(const wavepp_kda_shape* shape, const wavepp_kda_batch* batch, wavepp_kda_plan_t** out) {
  clear_error();
  if (!shape || !batch || !out) return set_error(WAVEPP_EINVAL, "null argument");
  *out = nullptr;
  const wavepp_kda_shape s = *shape;
  if (s.num_heads <= 0 || s.head_dim_k <= 0 || s.head_dim_v <= 0 || s.num_state_slots < 0)
    return set_error(WAVEPP_EINVAL, "non-positive shape field");
  if (s.head_dim_k != kKdaDim || s.head_dim_v != kKdaDim)
    return set_error(WAVEPP_EUNSUPPORTED, "unsupported head dims (d_k=%d, d_v=%d): only %d x %d", s.head_dim_k,
                     s.head_dim_v, kKdaDim, kKdaDim);
  if (int64_t(s.num_heads) * kKdaDim > INT32_MAX / 4) return set_error(WAVEPP_EINVAL, "too many heads");
  const int32_t R = batch->num_requests;
  if (R < 0) return set_error(WAVEPP_EINVAL, "num_requests < 0");
  if (R > 0 && (!batch->chunk_lens || !batch->state_in || !batch->state_out))
    return set_error(WAVEPP_EINVAL, "null chunk_lens / state_in / state_out");

  int64_t total = 0;
  std::vector<int32_t> writer(size_t(s.num_state_slots), -1);
  for (int32_t r = 0; r < R; ++r) {
    const int32_t c = batch->chunk_lens[r];
    if (c < 0) return set_error(WAVEPP_EINVAL, "request %d: negative chunk length %d", r, c);
    total += c;
    if (total > INT32_MAX / 2) return set_error(WAVEPP_EINVAL, "too many tokens in the wave");
    if (c == 0) continue;
    const int32_t si = batch->state_in[r], so = batch->state_out[r];
    if (si < -1 || si >= s.num_state_slots)
      return set_error(WAVEPP_ERANGE, "request %d: state_in %d outside [-1, %d)", r, si, s.num_state_slots);
    if (so < 0 || so >= s.num_state_slots)
      return set_error(WAVEPP_ERANGE, "request %d: state_out %d outside [0, %d)", r, so, s.num_state_slots);
    if (writer[so] >= 0)
      return set_error(WAVEPP_EALIAS, "requests %d and %d both write snapshot slot %d", writer[so], r, so);
    writer[so] = r;
  }
  if (int64_t(total) * s.num_heads > int64_t(INT32_MAX) * 4)
    return set_error(WAVEPP_EINVAL, "wave too large");
  for (int32_t r = 0; r < R; ++r) {
    if (batch->chunk_lens[r] == 0) continue;
    const int32_t si = batch->state_in[r];
    if (si >= 0 && writer[si] >= 0 && writer[si] != r)
      return set_error(WAVEPP_EALIAS, "request %d resumes from slot %d, which request %d writes", r, si, writer[si]);
  }

  auto plan = new (std::nothrow) wavepp_kda_plan_t();
  if (!plan) return set_error(WAVEPP_EINVAL, "out of host memory");
  plan->shape = s;
  plan->total_tokens = total;
  plan->serial = next_serial();
  int64_t cu = 0;
  for (int32_t r = 0; r < R; ++r) {
    const int32_t c = batch->chunk_lens[r];
    if (c > 0) {
      KdaItem it{};
      it.req = r;
      it.cu = int32_t(cu);
      it.len = c;
      it.state_in = batch->state_in[r];
      it.state_out = batch->state_out[r];
      plan->items.push_back(it);
    }
    cu += c;
  }
  // longest chunks first: workgroups are dispatched in index order
  std::stable_sort(plan->items.begin(), plan->items.end(),
                   [](const KdaItem& a, const KdaItem& b) { return a.len > b.len; });
  if (int64_t(plan->items.size()) * s.num_heads > INT32_MAX / 2) {
    delete plan;
    return set_error(WAVEPP_EINVAL, "too many workgroups");
  }
  plan->off_items = align_up(sizeof(KdaHeader), 16);
  plan->blob.assign(plan->off_items + sizeof(KdaItem) * plan->items.size(), 0);
  KdaHeader h{};
  h.magic = kKdaMagic;
  h.serial = plan->serial;
  h.num_items = int32_t(plan->items.size());
  h.num_heads = s.num_heads;
  memcpy(plan->blob.data(), &h, sizeof(h));
  if (!plan->items.empty())
    memcpy(plan->blob.data() + plan->off_items, plan->items.data(), sizeof(KdaItem) * plan->items.size());
  plan->workspace_bytes = align_up(plan->blob.size(), 256);
  *out = plan;
  return WAVEPP_OK;
}

size_t wavepp_kda_workspace_bytes(const wavepp_kda_plan_t* plan) { return plan ? plan->workspace_bytes : 0; }

int wavepp_kda_get_info(const wavepp_kda_plan_t* plan, wavepp_kda_info* info) {
  if (!plan || !info) return set_error(WAVEPP_EINVAL, "null argument");
  info->total_tokens = plan->total_tokens;
  info->num_items = int32_t(plan->items.size());
  info->block_tokens = kKdaBlock;
  info->metadata_bytes = int64_t(plan->blob.size());
  info->workspace_bytes = int64_t(plan->workspace_bytes);
  return WAVEPP_OK;
}

int wavepp_kda_upload(const wavepp_kda_plan_t* plan, void* workspace, size_t ws_bytes, hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(WAVEPP_EINVAL, "plan is NULL");
  int st = check_ws(plan, workspace, ws_bytes);
  if (st) return st;
  st = stage_and_copy(plan->blob.data(), plan->blob.size(), workspace, stream);
  if (st) return st;
  note_upload(workspace, plan->serial);
  return WAVEPP_OK;
}

int wavepp_kda_chunked_prefill(const wavepp_kda_plan_t* plan, const void* q, const void* k, const void* v,
                               const float* alpha, const float* beta, float* state_pool, void* out,
                               void* workspace, size_t ws_bytes, hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(WAVEPP_EINVAL, "plan is NULL");
  int st = check_ws(plan, workspace, ws_bytes);
  if (st) return st;
  if (plan->items.empty()) return WAVEPP_OK;
  st = require_upload(workspace, plan->serial, "wavepp_kda_upload");
  if (st) return st;
  if (!q || !k || !v || !alpha || !beta || !state_pool || !out)
    return set_error(WAVEPP_EINVAL, "q / k / v / alpha / beta / state_pool / out is NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(alpha) || !aligned16(beta) ||
      !aligned16(state_pool) || !aligned16(out))
    return set_error(WAVEPP_EINVAL, "device buffers must be 16-byte aligned");
  KdaDevPlan d{};
  auto* base = static_cast<unsigned char*>(workspace);
  d.hdr = reinterpret_cast<const KdaHeader*>(base);
  d.items = reinterpret_cast<const KdaItem*>(base + plan->off_items);
  d.serial = plan->serial;
  d.num_items = int32_t(plan->items.size());
  d.num_heads = plan->shape.num_heads;
  d.num_slots = plan->shape.num_state_slots;
  hipError_t e = launch_kda_prefill(d, q, k, v, alpha, beta, state_pool, out, stream);
  if (e != hipSuccess) return set_hip_error(e, "kda launch");
  return WAVEPP_OK;
}

void wavepp_kda_destroy(wavepp_kda_plan_t* plan) { delete plan; }

}  // extern "C"
