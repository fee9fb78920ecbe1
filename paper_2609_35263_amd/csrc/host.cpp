// Host side of libwavepp_attn: validation, work-list planning, metadata staging and launches.
//
// The plan turns a wave -- per-request spans (request, cached length p_r, chunk length c_r) and
// block tables over a page pool -- into a list of attention work items.  Spans and paging follow
// the paper's problem statement (Preliminaries, "Reuse": ceil(n / B) blocks in non-contiguous
// pages; Pipeline Scheduling: spans of request id, starting token and length, where a position
// that does not match the materialized cache must fail rather than run).
#include "wavepp_attn.h"
#include "internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <numeric>
#include <string>
#include <unordered_map>
#include <vector>

using namespace wavepp;

struct wavepp_plan {
  wavepp_attn_shape shape;
  int32_t num_requests = 0;
  int32_t bt_stride = 0;
  int64_t total_tokens = 0;
  uint32_t serial = 0;
  int32_t rows_per_item = 0;
  int32_t kv_tile = 0;
  int32_t max_splits_used = 1;
  int32_t num_real_items = 0;
  std::vector<WorkItem> items;
  std::vector<MergeItem> merges;
  int64_t partial_rows = 0;
  // metadata blob (uploaded as is) and its sub-array offsets
  std::vector<unsigned char> blob;
  size_t off_reqs = 0, off_bt = 0, off_items = 0, off_merges = 0;
  size_t meta_bytes = 0;       // blob size rounded up to 256
  size_t off_opart = 0, off_lpart = 0;
  size_t workspace_bytes = 0;
};

namespace wavepp {
namespace {
thread_local std::string g_last_error;
std::atomic<uint32_t> g_serial{1};
}  // namespace

int set_error(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int set_hip_error(hipError_t e, const char* what) {
  return set_error(WAVEPP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

void clear_error() { g_last_error.clear(); }

const char* last_error_text() { return g_last_error.c_str(); }

uint32_t next_serial() { return g_serial.fetch_add(1); }

// Which plan's metadata each workspace was last given, by the serial of the plan whose upload this
// library enqueued into it.  The entry points that launch kernels consult it before enqueuing
// anything, so a missing or stale upload is an error on the host; the kernels' own serial check
// stays as a second guard (e.g. for a workspace the caller overwrote in between).
namespace {
std::mutex g_ws_mu;
std::unordered_map<uintptr_t, uint32_t> g_ws_serial;
}  // namespace

void note_upload(const void* workspace, uint32_t serial) {
  std::lock_guard<std::mutex> lock(g_ws_mu);
  g_ws_serial[reinterpret_cast<uintptr_t>(workspace)] = serial;
}

int require_upload(const void* workspace, uint32_t serial, const char* upload_fn) {
  uint32_t have = 0;
  bool found = false;
  {
    std::lock_guard<std::mutex> lock(g_ws_mu);
    auto it = g_ws_serial.find(reinterpret_cast<uintptr_t>(workspace));
    if (it != g_ws_serial.end()) {
      found = true;
      have = it->second;
    }
  }
  if (!found)
    return set_error(WAVEPP_EINVAL, "workspace %p holds no uploaded plan: call %s(plan, workspace) first", workspace,
                     upload_fn);
  if (have != serial)
    return set_error(WAVEPP_EINVAL, "workspace %p holds the metadata of another plan (serial %u, this plan %u): call "
                     "%s(plan, workspace) first", workspace, have, serial, upload_fn);
  return WAVEPP_OK;
}

}  // namespace wavepp

namespace {

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool supported_shape(const wavepp_attn_shape& s) {
  if (s.page_size != 16 && s.page_size != 64) return false;
  if (s.kv_shared) return s.head_dim_qk == 576 && s.head_dim_v == 512 && s.num_kv_heads == 1;
  return (s.head_dim_qk == 64 && s.head_dim_v == 64) || (s.head_dim_qk == 128 && s.head_dim_v == 128);
}

bool env_flag(const char* name, bool dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  return !(v[0] == '0' || v[0] == 'n' || v[0] == 'N' || v[0] == 'f' || v[0] == 'F');
}

// Estimated cost of an item: rows times the keys they see on average.
double item_cost(const WorkItem& it, int G) {
  double keys = double(it.kv_end - it.kv_begin) - 0.5 * double(it.rows) / double(G);
  return double(it.rows) * std::max(keys, 1.0);
}

// Order items heaviest first and spread them over the L2 domains: consecutive workgroup ids go
// round-robin to the kNumXcd domains, so item index k*kNumXcd + x runs on domain x.  Items of one
// (request, KV head) read the same K/V pages; keeping them on one domain lets its L2 serve the
// re-reads.  With few such streams, balance wins and items are placed individually.
// WAVEPP_STREAM_MAJOR=0 keeps each domain's items in plain heaviest-first order.
std::vector<WorkItem> order_items(std::vector<WorkItem> items, int G, bool xcd_aware, bool stream_major) {
  std::vector<double> cost(items.size());
  for (size_t i = 0; i < items.size(); ++i) cost[i] = item_cost(items[i], G);
  std::vector<size_t> idx(items.size());
  std::iota(idx.begin(), idx.end(), 0);
  std::stable_sort(idx.begin(), idx.end(), [&](size_t a, size_t b) { return cost[a] > cost[b]; });
  if (!xcd_aware || items.size() <= 1) {
    std::vector<WorkItem> out;
    out.reserve(items.size());
    for (size_t i : idx) out.push_back(items[i]);
    return out;
  }
  // streams = (req, kv_head)
  std::vector<std::pair<int64_t, double>> stream_cost;  // key -> total
  auto key_of = [](const WorkItem& w) { return (int64_t(w.req) << 32) | uint32_t(w.kv_head); };
  std::vector<int64_t> keys;
  for (auto& w : items) keys.push_back(key_of(w));
  std::vector<int64_t> uniq = keys;
  std::sort(uniq.begin(), uniq.end());
  uniq.erase(std::unique(uniq.begin(), uniq.end()), uniq.end());
  std::vector<double> scost(uniq.size(), 0.0);
  for (size_t i = 0; i < items.size(); ++i)
    scost[std::lower_bound(uniq.begin(), uniq.end(), keys[i]) - uniq.begin()] += cost[i];
  double total = std::accumulate(scost.begin(), scost.end(), 0.0);
  double biggest = uniq.empty() ? 0.0 : *std::max_element(scost.begin(), scost.end());
  std::vector<std::vector<size_t>> lists(kNumXcd);
  std::vector<double> load(kNumXcd, 0.0);
  bool by_stream = uniq.size() >= size_t(2 * kNumXcd) && biggest <= 0.5 * total / kNumXcd;
  if (by_stream) {
    std::vector<size_t> sidx(uniq.size());
    std::iota(sidx.begin(), sidx.end(), 0);
    std::stable_sort(sidx.begin(), sidx.end(), [&](size_t a, size_t b) { return scost[a] > scost[b]; });
    std::vector<int> where(uniq.size(), 0);
    for (size_t s : sidx) {
      int x = int(std::min_element(load.begin(), load.end()) - load.begin());
      where[s] = x;
      load[x] += scost[s];
    }
    if (stream_major) {
      // inside a domain, stream by stream (heaviest stream first), each stream's items heaviest
      // first: the items running together on the domain's CUs then mostly belong to one stream and
      // read its tiles at about the same time, so the domain's L2 serves the re-reads
      std::vector<std::vector<size_t>> by(uniq.size());
      for (size_t i : idx) by[std::lower_bound(uniq.begin(), uniq.end(), keys[i]) - uniq.begin()].push_back(i);
      for (size_t s : sidx) lists[where[s]].insert(lists[where[s]].end(), by[s].begin(), by[s].end());
    } else {
      for (size_t i : idx) lists[where[std::lower_bound(uniq.begin(), uniq.end(), keys[i]) - uniq.begin()]].push_back(i);
    }
  } else {
    for (size_t i : idx) {
      int x = int(std::min_element(load.begin(), load.end()) - load.begin());
      lists[x].push_back(i);
      load[x] += cost[i];
    }
  }
  size_t longest = 0;
  for (auto& l : lists) longest = std::max(longest, l.size());
  std::vector<WorkItem> out;
  out.reserve(longest * kNumXcd);
  WorkItem pad{};
  pad.part = -1;
  for (size_t k = 0; k < longest; ++k)
    for (int x = 0; x < kNumXcd; ++x) out.push_back(k < lists[x].size() ? items[lists[x][k]] : pad);
  // trim trailing padding
  while (!out.empty() && out.back().rows == 0) out.pop_back();
  return out;
}

}  // namespace

namespace wavepp {

// ---------------------------------------------------------------------------------------------
// Pinned staging for metadata uploads: a small ring of page-locked buffers per device, each
// guarded by an event so a buffer is refilled only after its previous copy has completed.  The
// buffers are coherent and mapped into the device's address space; a copy kernel on the caller's
// stream moves them into the workspace (see launch_upload).
// ---------------------------------------------------------------------------------------------
struct StagingSlot {
  void* host = nullptr;
  void* dev = nullptr;     // the same buffer's device address
  size_t cap = 0;
  hipEvent_t done = nullptr;
  bool pending = false;
};
struct DeviceStaging {
  std::vector<StagingSlot> slots;
  size_t next = 0;
};
std::mutex g_stage_mu;
std::vector<DeviceStaging> g_stage;   // indexed by device id
constexpr int kStageSlots = 8;

int stage_and_copy(const void* src, size_t bytes, void* dst, hipStream_t stream) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_hip_error(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_stage_mu);
  if (g_stage.size() <= size_t(dev)) g_stage.resize(dev + 1);
  DeviceStaging& ds = g_stage[dev];
  if (ds.slots.empty()) ds.slots.resize(kStageSlots);
  StagingSlot& s = ds.slots[ds.next];
  ds.next = (ds.next + 1) % ds.slots.size();
  if (!s.done) {
    e = hipEventCreateWithFlags(&s.done, hipEventDisableTiming);
    if (e != hipSuccess) return set_hip_error(e, "hipEventCreateWithFlags");
  }
  if (s.pending) {
    e = hipEventSynchronize(s.done);
    if (e != hipSuccess) return set_hip_error(e, "hipEventSynchronize");
    s.pending = false;
  }
  if (s.cap < bytes) {
    if (s.host) {
      e = hipHostFree(s.host);
      s.host = nullptr;
      s.dev = nullptr;
      s.cap = 0;
      if (e != hipSuccess) return set_hip_error(e, "hipHostFree");
    }
    size_t cap = align_up(std::max<size_t>(bytes, 64 << 10), 4096);
    void* host = nullptr;
    void* mapped = nullptr;
    e = hipHostMalloc(&host, cap, hipHostMallocCoherent | hipHostMallocMapped);
    if (e != hipSuccess) return set_hip_error(e, "hipHostMalloc");
    e = hipHostGetDevicePointer(&mapped, host, 0);
    if (e != hipSuccess) {
      (void)hipHostFree(host);
      return set_hip_error(e, "hipHostGetDevicePointer");
    }
    s.host = host;
    s.dev = mapped;
    s.cap = cap;
  }
  memcpy(s.host, src, bytes);
  e = launch_upload(s.dev, dst, bytes, stream);
  if (e != hipSuccess) return set_hip_error(e, "metadata upload launch");
  e = hipEventRecord(s.done, stream);
  if (e != hipSuccess) return set_hip_error(e, "hipEventRecord");
  s.pending = true;
  return WAVEPP_OK;
}

}  // namespace wavepp

namespace {

int check_workspace(const wavepp_plan* plan, void* ws, size_t ws_bytes) {
  if (!ws) return set_error(WAVEPP_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return set_error(WAVEPP_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < plan->workspace_bytes)
    return set_error(WAVEPP_ENOSPACE, "workspace has %zu bytes, plan needs %zu", ws_bytes, plan->workspace_bytes);
  return WAVEPP_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

DevPlan make_dev(const wavepp_plan* plan, void* ws) {
  auto* base = static_cast<unsigned char*>(ws);
  DevPlan d{};
  d.hdr = reinterpret_cast<const MetaHeader*>(base);
  d.reqs = reinterpret_cast<const ReqMeta*>(base + plan->off_reqs);
  d.bt = reinterpret_cast<const int32_t*>(base + plan->off_bt);
  d.items = reinterpret_cast<const WorkItem*>(base + plan->off_items);
  d.merges = reinterpret_cast<const MergeItem*>(base + plan->off_merges);
  d.opart = reinterpret_cast<float*>(base + plan->off_opart);
  d.lpart = reinterpret_cast<float*>(base + plan->off_lpart);
  d.serial = plan->serial;
  d.num_requests = plan->num_requests;
  d.num_items = int32_t(plan->items.size());
  d.num_merge = int32_t(plan->merges.size());
  d.total_tokens = plan->total_tokens;
  d.num_q_heads = plan->shape.num_q_heads;
  d.num_kv_heads = plan->shape.num_kv_heads;
  d.head_dim_qk = plan->shape.head_dim_qk;
  d.head_dim_v = plan->shape.head_dim_v;
  d.page_size = plan->shape.page_size;
  d.kv_shared = plan->shape.kv_shared;
  d.softmax_scale = plan->shape.softmax_scale;
  d.rows_per_item = plan->rows_per_item;
  return d;
}

}  // namespace

extern "C" {

const char* wavepp_status_string(int status) {
  switch (status) {
    case WAVEPP_OK: return "WAVEPP_OK";
    case WAVEPP_EINVAL: return "WAVEPP_EINVAL: invalid argument";
    case WAVEPP_EUNSUPPORTED: return "WAVEPP_EUNSUPPORTED: unsupported shape";
    case WAVEPP_ERANGE: return "WAVEPP_ERANGE: block-table entry outside the page pool";
    case WAVEPP_EALIAS: return "WAVEPP_EALIAS: appended page also referenced elsewhere";
    case WAVEPP_EPOSITION: return "WAVEPP_EPOSITION: span not backed by the block table";
    case WAVEPP_ENOSPACE: return "WAVEPP_ENOSPACE: workspace too small";
    case WAVEPP_EHIP: return "WAVEPP_EHIP: HIP runtime error";
    default: return "unknown wavepp status";
  }
}

const char* wavepp_last_error(void) { return last_error_text(); }

int wavepp_attn_plan(const wavepp_attn_shape* shape, const wavepp_batch* batch, int32_t max_splits,
                     wavepp_plan** out) {
  clear_error();
  if (!shape || !batch || !out) return set_error(WAVEPP_EINVAL, "null argument");
  *out = nullptr;
  const wavepp_attn_shape s = *shape;
  if (s.num_q_heads <= 0 || s.num_kv_heads <= 0 || s.num_pages <= 0 || s.page_size <= 0 ||
      s.head_dim_qk <= 0 || s.head_dim_v <= 0)
    return set_error(WAVEPP_EINVAL, "non-positive shape field");
  if (!(s.softmax_scale > 0.0f) || !std::isfinite(s.softmax_scale))
    return set_error(WAVEPP_EINVAL, "softmax_scale must be positive and finite");
  if (s.num_q_heads % s.num_kv_heads)
    return set_error(WAVEPP_EINVAL, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)", s.num_q_heads,
                s.num_kv_heads);
  if (s.kv_shared != 0 && s.kv_shared != 1) return set_error(WAVEPP_EINVAL, "kv_shared must be 0 or 1");
  if (!supported_shape(s))
    return set_error(WAVEPP_EUNSUPPORTED, "unsupported (head_dim_qk=%d, head_dim_v=%d, page_size=%d, kv_shared=%d, "
                "num_kv_heads=%d)", s.head_dim_qk, s.head_dim_v, s.page_size, s.kv_shared, s.num_kv_heads);
  if (max_splits < 0) return set_error(WAVEPP_EINVAL, "max_splits must be >= 0");
  const int32_t R = batch->num_requests;
  if (R < 0) return set_error(WAVEPP_EINVAL, "num_requests < 0");
  if (R > 0 && (!batch->prefix_lens || !batch->chunk_lens || !batch->block_table))
    return set_error(WAVEPP_EINVAL, "null span or block-table array");
  if (R > 0 && batch->bt_stride <= 0) return set_error(WAVEPP_EINVAL, "bt_stride must be positive");
  const int32_t B = s.page_size, P = s.num_pages, stride = R > 0 ? batch->bt_stride : 0;
  const int G = s.num_q_heads / s.num_kv_heads;

  // --- spans and block tables ------------------------------------------------------------------
  int64_t total = 0;
  std::vector<int32_t> refcount(P, 0);
  for (int32_t r = 0; r < R; ++r) {
    const int64_t p = batch->prefix_lens[r], c = batch->chunk_lens[r];
    if (p < 0 || c < 0) return set_error(WAVEPP_EINVAL, "request %d: negative length (p=%lld, c=%lld)", r, (long long)p,
                                    (long long)c);
    const int64_t n = p + c;
    if (n > INT32_MAX / 2) return set_error(WAVEPP_EINVAL, "request %d: length %lld too large", r, (long long)n);
    if (n > int64_t(stride) * B)
      return set_error(WAVEPP_EPOSITION, "request %d: positions up to %lld but the block table covers %lld", r,
                  (long long)n, (long long)stride * B);
    const int64_t nb = ceil_div(n, B);
    const int32_t* row = batch->block_table + int64_t(r) * stride;
    for (int64_t b = 0; b < nb; ++b) {
      if (row[b] < 0 || row[b] >= P)
        return set_error(WAVEPP_ERANGE, "request %d block %lld: page %d outside [0, %d)", r, (long long)b, row[b], P);
      refcount[row[b]]++;
    }
    total += c;
    if (total > INT32_MAX / 2) return set_error(WAVEPP_EINVAL, "too many tokens in the wave");
  }
  for (int32_t r = 0; r < R; ++r) {
    const int64_t p = batch->prefix_lens[r], c = batch->chunk_lens[r];
    if (c == 0) continue;
    const int32_t* row = batch->block_table + int64_t(r) * stride;
    for (int64_t b = p / B; b < ceil_div(p + c, B); ++b)
      if (refcount[row[b]] != 1)
        return set_error(WAVEPP_EALIAS, "request %d block %lld: page %d receives appended tokens but is referenced %d "
                    "times in the wave", r, (long long)b, row[b], refcount[row[b]]);
  }

  auto plan = new (std::nothrow) wavepp_plan();
  if (!plan) return set_error(WAVEPP_EINVAL, "out of host memory");
  plan->shape = s;
  plan->num_requests = R;
  plan->bt_stride = stride;
  plan->total_tokens = total;
  plan->serial = next_serial();
  const bool mla = s.kv_shared != 0;
  // grouped kernel: 8 waves (256 rows) per workgroup and one workgroup per CU, so that each K/V tile
  // staged in LDS serves 256 rows.  When no (request, KV head) has more than 128 rows (short
  // chunks: the wave is bound by streaming the prefix K/V), half of those waves would idle: the
  // plan then uses 128-row items, run by the 4-wave form of the kernel, two workgroups per CU.
  // WAVEPP_GQA_WAVES=4 or 8 forces one form.
  int64_t max_rows = 0;
  for (int32_t r = 0; r < R; ++r) max_rows = std::max<int64_t>(max_rows, int64_t(batch->chunk_lens[r]) * (s.num_q_heads / s.num_kv_heads));
  const char* gw = getenv("WAVEPP_GQA_WAVES");
  const int gw_n = gw ? atoi(gw) : 0;
  const bool small_rows = gw_n == 4 || (gw_n != 8 && max_rows <= kGqaRowsPerItem / 2);
  const int gqa_rows = small_rows ? kGqaRowsPerItem / 2 : kGqaRowsPerItem;
  const int M = mla ? kMlaRowsPerItem : gqa_rows;
  // keys per tile of the kernel that will run the plan (the 4-wave grouped form uses half tiles);
  // split boundaries fall on whole tiles of it
  const int KT = mla ? kMlaKvTile : (small_rows ? kKvTile / 2 : kKvTile);
  plan->rows_per_item = M;
  plan->kv_tile = KT;

  // --- work items --------------------------------------------------------------------------------
  std::vector<WorkItem> base;
  std::vector<ReqMeta> reqs(R);
  int64_t cu = 0;
  for (int32_t r = 0; r < R; ++r) {
    const int32_t p = batch->prefix_lens[r], c = batch->chunk_lens[r];
    reqs[r] = ReqMeta{p, c, int32_t(cu), int32_t(int64_t(r) * stride)};
    cu += c;
    const int64_t rows_total = int64_t(c) * G;
    for (int32_t g = 0; g < s.num_kv_heads; ++g)
      for (int64_t r0 = 0; r0 < rows_total; r0 += M) {
        WorkItem w{};
        w.req = r;
        w.kv_head = g;
        w.row0 = int32_t(r0);
        w.rows = int32_t(std::min<int64_t>(M, rows_total - r0));
        const int64_t last_tok = (r0 + w.rows - 1) / G;
        w.kv_begin = 0;
        w.kv_end = int32_t(p + last_tok + 1);
        w.part = -1;
        w.split = 0;
        base.push_back(w);
      }
  }
  // key-range splits: forced by max_splits, or chosen so that a small wave still fills the chip,
  // each automatic split keeping at least 1,024 keys (grouped kernel) or 512 (latent kernel).
  // Split a wave with fewer base items than this until it has about that many.  512 items are two
  // workgroups per CU of the 4-wave form, or two rounds of the one-per-CU forms; on the short-chunk
  // waves (c = 16 .. 128) it gave the fastest or within 0.5 % of the fastest split count, against
  // 1,024 items, which cost 2-11 % in the extra partials and merge work.
  // Automatic splits share the wave's tiles out evenly rather than giving every (request, KV head,
  // row tile) the same number of splits: such a wave runs as one round of workgroups and lasts as
  // long as its longest item, so requests with longer prefixes take more splits.  T is the smallest
  // tile count per split for which the wave stays within the target; an item of n tiles then takes
  // ceil(n / T) splits (at most n / min_split_tiles).
  const int64_t fill_target = 512;
  const int64_t min_split_tiles = (mla ? 512 : 1024) / KT;
  std::vector<int64_t> nsplit(base.size(), 1);
  if (max_splits >= 1) {
    for (size_t i = 0; i < base.size(); ++i)
      nsplit[i] = std::min<int64_t>(max_splits, ceil_div(base[i].kv_end, KT));
  } else if (int64_t(base.size()) < fill_target) {
    auto auto_splits = [&](int64_t ntiles, int64_t T) {
      return std::max<int64_t>(1, std::min<int64_t>(ceil_div(ntiles, T), ntiles / min_split_tiles));
    };
    auto total = [&](int64_t T) {
      int64_t n = 0;
      for (const WorkItem& w : base) n += auto_splits(ceil_div(w.kv_end, KT), T);
      return n;
    };
    int64_t lo = std::max<int64_t>(1, min_split_tiles), hi = lo;
    for (const WorkItem& w : base) hi = std::max<int64_t>(hi, ceil_div(w.kv_end, KT));
    // total(T) does not grow with T, and total(hi) = base.size() < fill_target
    if (total(lo) > fill_target) {
      while (hi - lo > 1) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (total(mid) <= fill_target) hi = mid; else lo = mid;
      }
      lo = hi;
    }
    for (size_t i = 0; i < base.size(); ++i) nsplit[i] = auto_splits(ceil_div(base[i].kv_end, KT), lo);
  }
  std::vector<WorkItem> items;
  int64_t part_rows = 0;
  int max_used = 1;
  for (size_t bi = 0; bi < base.size(); ++bi) {
    const WorkItem& w = base[bi];
    const int64_t ntiles = ceil_div(w.kv_end, KT);
    int64_t S = nsplit[bi];
    const int64_t tps = ceil_div(ntiles, S);
    S = ceil_div(ntiles, tps);
    if (S == 1) {
      items.push_back(w);
      continue;
    }
    max_used = std::max<int>(max_used, int(S));
    MergeItem m{};
    m.req = w.req;
    m.kv_head = w.kv_head;
    m.row0 = w.row0;
    m.rows = w.rows;
    m.nsplit = int32_t(S);
    m.part = int32_t(part_rows);
    plan->merges.push_back(m);
    for (int64_t si = 0; si < S; ++si) {
      WorkItem x = w;
      x.kv_begin = int32_t(si * tps * KT);
      x.kv_end = int32_t(std::min<int64_t>(w.kv_end, (si + 1) * tps * KT));
      x.part = int32_t(part_rows + si * w.rows);
      x.split = int32_t(si);
      items.push_back(x);
    }
    part_rows += S * w.rows;
    if (part_rows > INT32_MAX / 2) {
      delete plan;
      return set_error(WAVEPP_EINVAL, "split partials too large");
    }
  }
  plan->num_real_items = int32_t(items.size());
  plan->max_splits_used = max_used;
  plan->partial_rows = part_rows;
  plan->items = order_items(std::move(items), G, env_flag("WAVEPP_XCD_ORDER", true),
                            env_flag("WAVEPP_STREAM_MAJOR", true));
  if (plan->items.size() > size_t(INT32_MAX / 2)) {
    delete plan;
    return set_error(WAVEPP_EINVAL, "too many work items");
  }

  // --- metadata blob -------------------------------------------------------------------------------
  size_t off = align_up(sizeof(MetaHeader), 16);
  plan->off_reqs = off;
  off = align_up(off + sizeof(ReqMeta) * R, 16);
  plan->off_bt = off;
  off = align_up(off + sizeof(int32_t) * size_t(R) * size_t(stride), 16);
  plan->off_items = off;
  off = align_up(off + sizeof(WorkItem) * plan->items.size(), 16);
  plan->off_merges = off;
  off = align_up(off + sizeof(MergeItem) * plan->merges.size(), 16);
  plan->blob.assign(off, 0);
  MetaHeader h{};
  h.magic = kMagic;
  h.serial = plan->serial;
  h.num_requests = R;
  h.num_items = int32_t(plan->items.size());
  h.num_merge = int32_t(plan->merges.size());
  h.bt_stride = stride;
  memcpy(plan->blob.data(), &h, sizeof(h));
  if (R) {
    memcpy(plan->blob.data() + plan->off_reqs, reqs.data(), sizeof(ReqMeta) * R);
    memcpy(plan->blob.data() + plan->off_bt, batch->block_table, sizeof(int32_t) * size_t(R) * size_t(stride));
  }
  if (!plan->items.empty())
    memcpy(plan->blob.data() + plan->off_items, plan->items.data(), sizeof(WorkItem) * plan->items.size());
  if (!plan->merges.empty())
    memcpy(plan->blob.data() + plan->off_merges, plan->merges.data(), sizeof(MergeItem) * plan->merges.size());
  plan->meta_bytes = align_up(off, 256);
  plan->off_opart = plan->meta_bytes;
  plan->off_lpart = align_up(plan->off_opart + sizeof(float) * size_t(part_rows) * size_t(s.head_dim_v), 256);
  plan->workspace_bytes = align_up(plan->off_lpart + sizeof(float) * size_t(part_rows), 256);
  *out = plan;
  return WAVEPP_OK;
}

size_t wavepp_plan_workspace_bytes(const wavepp_plan* plan) { return plan ? plan->workspace_bytes : 0; }

int wavepp_plan_get_info(const wavepp_plan* plan, wavepp_plan_info* info) {
  if (!plan || !info) return set_error(WAVEPP_EINVAL, "null argument");
  info->total_tokens = plan->total_tokens;
  info->num_items = int32_t(plan->items.size());
  info->num_real_items = plan->num_real_items;
  info->num_merge_items = int32_t(plan->merges.size());
  info->max_splits = plan->max_splits_used;
  info->rows_per_item = plan->rows_per_item;
  info->kv_tile = plan->kv_tile;
  info->partial_rows = plan->partial_rows;
  info->metadata_bytes = int64_t(plan->blob.size());
  info->workspace_bytes = int64_t(plan->workspace_bytes);
  return WAVEPP_OK;
}

int wavepp_plan_get_items(const wavepp_plan* plan, int32_t* items, int32_t capacity) {
  if (!plan || (!items && capacity > 0) || capacity < 0) return set_error(WAVEPP_EINVAL, "bad argument");
  const int32_t n = std::min<int32_t>(capacity, int32_t(plan->items.size()));
  for (int32_t i = 0; i < n; ++i) {
    const WorkItem& w = plan->items[i];
    const int32_t v[8] = {w.req, w.kv_head, w.row0, w.rows, w.kv_begin, w.kv_end, w.part, w.split};
    memcpy(items + 8 * int64_t(i), v, sizeof(v));
  }
  return n;
}

int wavepp_attn_plan_upload(const wavepp_plan* plan, void* workspace, size_t ws_bytes, hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(WAVEPP_EINVAL, "plan is NULL");
  int st = check_workspace(plan, workspace, ws_bytes);
  if (st) return st;
  st = stage_and_copy(plan->blob.data(), plan->blob.size(), workspace, stream);
  if (st) return st;
  note_upload(workspace, plan->serial);
  return WAVEPP_OK;
}

int wavepp_attn_append_kv(const wavepp_plan* plan, const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                          void* workspace, size_t ws_bytes, hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(WAVEPP_EINVAL, "plan is NULL");
  int st = check_workspace(plan, workspace, ws_bytes);
  if (st) return st;
  const bool shared = plan->shape.kv_shared != 0;
  if (plan->total_tokens == 0) return WAVEPP_OK;
  st = require_upload(workspace, plan->serial, "wavepp_attn_plan_upload");
  if (st) return st;
  if (!k_new || !k_pool) return set_error(WAVEPP_EINVAL, "k_new / k_pool is NULL");
  if (!shared && (!v_new || !v_pool)) return set_error(WAVEPP_EINVAL, "v_new / v_pool is NULL");
  if (shared && (v_new || v_pool)) return set_error(WAVEPP_EINVAL, "v_new / v_pool must be NULL for a latent cache");
  if (!aligned16(k_new) || !aligned16(k_pool) || (!shared && (!aligned16(v_new) || !aligned16(v_pool))))
    return set_error(WAVEPP_EINVAL, "device buffers must be 16-byte aligned");
  DevPlan d = make_dev(plan, workspace);
  hipError_t e = launch_append(d, k_new, v_new, k_pool, v_pool, stream);
  if (e != hipSuccess) return set_hip_error(e, "append_kv launch");
  return WAVEPP_OK;
}

int wavepp_attn_chunked_prefill(const wavepp_plan* plan, const void* q, const void* k_pool, const void* v_pool,
                                void* out, float* lse, void* workspace, size_t ws_bytes, hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(WAVEPP_EINVAL, "plan is NULL");
  int st = check_workspace(plan, workspace, ws_bytes);
  if (st) return st;
  const bool shared = plan->shape.kv_shared != 0;
  if (plan->total_tokens == 0) return WAVEPP_OK;
  st = require_upload(workspace, plan->serial, "wavepp_attn_plan_upload");
  if (st) return st;
  if (!q || !k_pool || !out) return set_error(WAVEPP_EINVAL, "q / k_pool / out is NULL");
  if (!shared && !v_pool) return set_error(WAVEPP_EINVAL, "v_pool is NULL");
  if (shared && v_pool) return set_error(WAVEPP_EINVAL, "v_pool must be NULL for a latent cache");
  if (!aligned16(q) || !aligned16(k_pool) || !aligned16(out) || (!shared && !aligned16(v_pool)) ||
      (reinterpret_cast<uintptr_t>(lse) & 3))
    return set_error(WAVEPP_EINVAL, "device buffers must be 16-byte aligned (lse 4-byte)");
  DevPlan d = make_dev(plan, workspace);
  hipError_t e = launch_attention(d, q, k_pool, v_pool, out, lse, stream);
  if (e != hipSuccess) return set_hip_error(e, "attention launch");
  if (!plan->merges.empty()) {
    e = launch_merge(d, out, lse, stream);
    if (e != hipSuccess) return set_hip_error(e, "merge launch");
  }
  return WAVEPP_OK;
}

int wavepp_attn_chunked_prefill_noalloc(const wavepp_plan* plan, const void* q, const void* k_new,
                                        const void* v_new, void* k_pool, void* v_pool, void* out, float* lse,
                                        hipStream_t stream) {
  clear_error();
  if (!plan) return set_error(WAVEPP_EINVAL, "plan is NULL");
  if (plan->workspace_bytes > kNoAllocScratchBytes)
    return set_error(WAVEPP_ENOSPACE, "plan needs %zu bytes of scratch, the static scratch holds %zu: plan the wave "
                     "with fewer key-range splits (max_splits) or call wavepp_attn_chunked_prefill with a workspace",
                     plan->workspace_bytes, kNoAllocScratchBytes);
  const bool shared = plan->shape.kv_shared != 0;
  if (plan->total_tokens == 0) return WAVEPP_OK;
  if (!q || !k_pool || !out) return set_error(WAVEPP_EINVAL, "q / k_pool / out is NULL");
  if (!shared && !v_pool) return set_error(WAVEPP_EINVAL, "v_pool is NULL");
  if (shared && (v_pool || v_new)) return set_error(WAVEPP_EINVAL, "v_pool / v_new must be NULL for a latent cache");
  if (k_new && !shared && !v_new) return set_error(WAVEPP_EINVAL, "v_new is NULL while k_new is given");
  if (!k_new && v_new) return set_error(WAVEPP_EINVAL, "v_new is given without k_new");
  if (!aligned16(q) || !aligned16(k_pool) || !aligned16(out) || (!shared && !aligned16(v_pool)) ||
      (k_new && !aligned16(k_new)) || (v_new && !aligned16(v_new)) || (reinterpret_cast<uintptr_t>(lse) & 3))
    return set_error(WAVEPP_EINVAL, "device buffers must be 16-byte aligned (lse 4-byte)");
  void* ws = nullptr;
  hipError_t e = noalloc_scratch(&ws);
  if (e != hipSuccess) return set_hip_error(e, "static scratch address");
  // the plan's metadata into the head of the scratch (from the plan's own host memory: no staging
  // buffer of the library's is involved), then the same kernels as the workspace entry points
  e = hipMemcpyAsync(ws, plan->blob.data(), plan->blob.size(), hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return set_hip_error(e, "metadata copy into the static scratch");
  DevPlan d = make_dev(plan, ws);
  if (k_new) {
    e = launch_append(d, k_new, v_new, k_pool, v_pool, stream);
    if (e != hipSuccess) return set_hip_error(e, "append_kv launch");
  }
  e = launch_attention(d, q, k_pool, v_pool, out, lse, stream);
  if (e != hipSuccess) return set_hip_error(e, "attention launch");
  if (!plan->merges.empty()) {
    e = launch_merge(d, out, lse, stream);
    if (e != hipSuccess) return set_hip_error(e, "merge launch");
  }
  return WAVEPP_OK;
}

void wavepp_plan_destroy(wavepp_plan* plan) { delete plan; }

}  // extern "C"
