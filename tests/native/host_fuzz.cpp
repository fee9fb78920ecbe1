// Seeded randomized driver of the host entry points, for builds under the address and
// undefined-behaviour sanitizers (and a plain build).  It makes no HIP call: the attention and KDA
// planners validate and plan, the kernel entry points are only driven into their host-side error
// paths (no upload into the workspace they are given), and the MPU planner and hint index are host
// objects.
//
// For every attention plan the validator accepts, the work list is checked: every visible
// (request, KV head, row, key) pair is covered exactly once, tiles start on the reported key tile,
// and split partial rows stay inside the workspace.  A status the validator returns is checked
// against an independent restatement of the rules (request order, then aliasing).
//
// Usage: host_fuzz [iterations] [seed]; exits non-zero on the first violation.
#include "wavepp_attn.h"
#include "wavepp_hints.h"
#include "wavepp_kda.h"
#include "wavepp_mpu.h"

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <vector>

namespace {

struct Rng {
  uint64_t s;
  explicit Rng(uint64_t seed) : s(seed * 0x9E3779B97F4A7C15ull + 1) {}
  uint64_t next() {
    s ^= s << 13;
    s ^= s >> 7;
    s ^= s << 17;
    return s;
  }
  int32_t range(int32_t lo, int32_t hi) { return lo + int32_t(next() % uint64_t(hi - lo + 1)); }   // [lo, hi]
  bool chance(int percent) { return int(next() % 100) < percent; }
};

int g_fail = 0;
int g_status_count[8] = {0};   // by -status
#define CHECK(cond, ...)                                  \
  do {                                                    \
    if (!(cond)) {                                        \
      fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      fprintf(stderr, __VA_ARGS__);                       \
      fprintf(stderr, "\n");                              \
      g_fail = 1;                                         \
      return;                                             \
    }                                                     \
  } while (0)

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool supported(const wavepp_attn_shape& s) {
  if (s.page_size != 16 && s.page_size != 64) return false;
  if (s.kv_shared) return s.head_dim_qk == 576 && s.head_dim_v == 512 && s.num_kv_heads == 1;
  return (s.head_dim_qk == 64 && s.head_dim_v == 64) || (s.head_dim_qk == 128 && s.head_dim_v == 128);
}

// The validation rules, restated: shape, then each request in order (lengths, span backed by the
// table, entries in the pool), then the aliasing of pages that receive appended tokens.
int expected_status(const wavepp_attn_shape& s, int R, const std::vector<int32_t>& pre,
                    const std::vector<int32_t>& chk, const std::vector<int32_t>& bt, int stride) {
  if (s.num_q_heads % s.num_kv_heads) return WAVEPP_EINVAL;
  if (!supported(s)) return WAVEPP_EUNSUPPORTED;
  const int B = s.page_size;
  std::vector<int> ref(s.num_pages, 0);
  for (int r = 0; r < R; ++r) {
    if (pre[r] < 0 || chk[r] < 0) return WAVEPP_EINVAL;
    const int64_t n = int64_t(pre[r]) + chk[r];
    if (n > int64_t(stride) * B) return WAVEPP_EPOSITION;
    for (int64_t b = 0; b < ceil_div(n, B); ++b) {
      const int32_t pg = bt[size_t(r) * stride + b];
      if (pg < 0 || pg >= s.num_pages) return WAVEPP_ERANGE;
      ref[pg]++;
    }
  }
  for (int r = 0; r < R; ++r) {
    if (chk[r] == 0) continue;
    for (int64_t b = pre[r] / B; b < ceil_div(int64_t(pre[r]) + chk[r], B); ++b)
      if (ref[bt[size_t(r) * stride + b]] != 1) return WAVEPP_EALIAS;
  }
  return WAVEPP_OK;
}

void check_plan(const wavepp_plan* plan, const wavepp_attn_shape& s, int R, const std::vector<int32_t>& pre,
                const std::vector<int32_t>& chk) {
  wavepp_plan_info info{};
  CHECK(wavepp_plan_get_info(plan, &info) == WAVEPP_OK, "get_info");
  std::vector<int32_t> items(size_t(std::max(info.num_items, 1)) * 8);
  const int got = wavepp_plan_get_items(plan, items.data(), info.num_items);
  CHECK(got == info.num_items, "get_items returned %d of %d", got, info.num_items);
  const int G = s.num_q_heads / s.num_kv_heads;
  const int KT = info.kv_tile;
  CHECK(KT > 0 && info.rows_per_item > 0, "tile %d rows %d", KT, info.rows_per_item);
  int64_t T = 0;
  for (int r = 0; r < R; ++r) T += chk[r];
  CHECK(info.total_tokens == T, "total tokens");
  // per (request, kv head, row): the key ranges covering it
  std::map<std::tuple<int, int, int>, std::vector<std::pair<int, int>>> seen;
  for (int i = 0; i < got; ++i) {
    const int32_t* w = &items[size_t(i) * 8];
    const int r = w[0], g = w[1], row0 = w[2], rows = w[3], kb = w[4], ke = w[5], part = w[6];
    if (rows == 0) continue;
    CHECK(r >= 0 && r < R && g >= 0 && g < s.num_kv_heads, "item %d request/head", i);
    CHECK(rows <= info.rows_per_item && row0 >= 0 && row0 + rows <= chk[r] * G, "item %d rows", i);
    CHECK(kb % KT == 0 && ke > kb && ke <= pre[r] + chk[r], "item %d keys [%d, %d) tile %d", i, kb, ke, KT);
    CHECK(part < 0 || int64_t(part) + rows <= info.partial_rows, "item %d partial rows", i);
    for (int row = row0; row < row0 + rows; ++row) seen[{r, g, row}].push_back({kb, ke});
  }
  for (int r = 0; r < R; ++r)
    for (int g = 0; g < s.num_kv_heads; ++g)
      for (int row = 0; row < chk[r] * G; ++row) {
        auto it = seen.find({r, g, row});
        CHECK(it != seen.end(), "row (%d, %d, %d) not covered", r, g, row);
        auto ranges = it->second;
        std::sort(ranges.begin(), ranges.end());
        int pos = 0;
        for (auto& kr : ranges) {
          CHECK(kr.first == pos, "row (%d, %d, %d): gap or overlap at key %d", r, g, row, pos);
          pos = kr.second;
        }
        CHECK(pos >= pre[r] + row / G + 1, "row (%d, %d, %d) misses visible keys", r, g, row);
        seen.erase(it);
      }
  CHECK(seen.empty(), "items cover rows that do not exist");
  CHECK(wavepp_plan_workspace_bytes(plan) % 256 == 0, "workspace alignment");
}

void fuzz_attention(Rng& rng) {
  wavepp_attn_shape s{};
  static const int dims[][2] = {{64, 64}, {128, 128}, {576, 512}, {96, 96}, {64, 128}};
  const int di = rng.chance(85) ? rng.range(0, 2) : rng.range(3, 4);
  s.head_dim_qk = dims[di][0];
  s.head_dim_v = dims[di][1];
  s.kv_shared = (di == 2) ? (rng.chance(90) ? 1 : 0) : (rng.chance(5) ? 1 : 0);
  s.num_kv_heads = s.kv_shared ? (rng.chance(95) ? 1 : 2) : rng.range(1, 4);
  s.num_q_heads = s.num_kv_heads * rng.range(1, 8) + (rng.chance(5) ? 1 : 0);
  s.page_size = rng.chance(90) ? (rng.chance(50) ? 16 : 64) : 32;
  s.num_pages = rng.range(1, 48);
  s.softmax_scale = 0.125f;
  const int R = rng.range(0, 5);
  const int stride = rng.range(1, 10);
  std::vector<int32_t> pre(R), chk(R), bt(size_t(std::max(R, 1)) * stride);
  for (int r = 0; r < R; ++r) {
    pre[r] = rng.chance(3) ? -rng.range(1, 5) : rng.range(0, 200);
    chk[r] = rng.chance(3) ? -1 : (rng.chance(15) ? 0 : rng.range(1, 150));
  }
  // tables: mostly distinct pages, sometimes a shared prefix page, an alias or an out-of-range entry
  for (auto& e : bt) e = rng.range(0, s.num_pages - 1);
  if (R > 0 && rng.chance(60)) {
    std::vector<int32_t> perm(s.num_pages);
    for (int i = 0; i < s.num_pages; ++i) perm[i] = i;
    for (int i = s.num_pages - 1; i > 0; --i) std::swap(perm[i], perm[rng.range(0, i)]);
    int k = 0;
    for (auto& e : bt) e = perm[(k++) % s.num_pages];
    if (R > 1 && rng.chance(40)) bt[stride] = bt[0];                 // second request shares page 0
  }
  if (!bt.empty() && rng.chance(10)) bt[rng.next() % bt.size()] = rng.chance(50) ? -1 : s.num_pages;
  wavepp_batch b{R, pre.data(), chk.data(), bt.data(), stride};
  wavepp_plan* plan = nullptr;
  const int splits = rng.chance(50) ? 0 : rng.range(1, 9);
  const int st = wavepp_attn_plan(&s, &b, splits, &plan);
  const int want = expected_status(s, R, pre, chk, bt, stride);
  if (st <= 0 && st > -8) g_status_count[-st]++;
  CHECK(st == want, "status %d, rules say %d (R=%d, P=%d, B=%d): %s", st, want, R, s.num_pages, s.page_size,
        wavepp_last_error());
  if (st != WAVEPP_OK) {
    CHECK(plan == nullptr, "plan set on error");
    return;
  }
  check_plan(plan, s, R, pre, chk);
  // kernel entry points refuse a workspace that was never given this plan, before any HIP call
  void* fake_ws = reinterpret_cast<void*>(uintptr_t(0x7f0000000000ull));
  const size_t wsb = wavepp_plan_workspace_bytes(plan) + 256;
  void* buf = reinterpret_cast<void*>(uintptr_t(0x7f0000100000ull));
  wavepp_plan_info info{};
  wavepp_plan_get_info(plan, &info);
  if (info.total_tokens > 0) {
    CHECK(wavepp_attn_chunked_prefill(plan, buf, buf, s.kv_shared ? nullptr : buf, buf, nullptr, fake_ws, wsb,
                                      nullptr) == WAVEPP_EINVAL, "prefill without upload");
    CHECK(wavepp_attn_append_kv(plan, buf, s.kv_shared ? nullptr : buf, buf, s.kv_shared ? nullptr : buf, fake_ws,
                                wsb, nullptr) == WAVEPP_EINVAL, "append without upload");
  }
  CHECK(wavepp_attn_chunked_prefill(plan, buf, buf, buf, buf, nullptr, fake_ws, 0, nullptr) == WAVEPP_ENOSPACE ||
            wavepp_plan_workspace_bytes(plan) == 0,
        "small workspace");
  wavepp_plan_destroy(plan);
}

void fuzz_kda(Rng& rng) {
  wavepp_kda_shape s{};
  s.num_heads = rng.range(0, 4);
  s.head_dim_k = rng.chance(90) ? 128 : 64;
  s.head_dim_v = rng.chance(90) ? 128 : 64;
  s.num_state_slots = rng.range(0, 8);
  const int R = rng.range(0, 6);
  std::vector<int32_t> c(R), si(R), so(R);
  for (int r = 0; r < R; ++r) {
    c[r] = rng.chance(5) ? -1 : rng.range(0, 300);
    si[r] = rng.range(-2, s.num_state_slots);
    so[r] = rng.range(-1, s.num_state_slots);
  }
  wavepp_kda_batch b{R, c.data(), si.data(), so.data()};
  wavepp_kda_plan_t* plan = nullptr;
  const int st = wavepp_kda_plan(&s, &b, &plan);
  if (st != WAVEPP_OK) {
    CHECK(plan == nullptr, "kda plan set on error");
    return;
  }
  wavepp_kda_info info{};
  CHECK(wavepp_kda_get_info(plan, &info) == WAVEPP_OK, "kda info");
  void* fake_ws = reinterpret_cast<void*>(uintptr_t(0x7f0000000000ull));
  void* buf = reinterpret_cast<void*>(uintptr_t(0x7f0000100000ull));
  if (info.num_items > 0)
    CHECK(wavepp_kda_chunked_prefill(plan, buf, buf, buf, (const float*)buf, (const float*)buf, (float*)buf, buf,
                                     fake_ws, wavepp_kda_workspace_bytes(plan), nullptr) == WAVEPP_EINVAL,
          "kda prefill without upload");
  wavepp_kda_destroy(plan);
}

void fuzz_mpu(Rng& rng) {
  wavepp_mpu_config cfg{};
  cfg.block = 64;
  cfg.max_budget = 64 * rng.range(1, 64);
  cfg.min_budget = 64 * rng.range(1, cfg.max_budget / 64);
  cfg.stages = rng.range(1, 4);
  cfg.fills = rng.range(1, 3);
  cfg.max_lanes = rng.range(1, 8);
  cfg.split_permille = rng.range(0, 1000);
  cfg.count_inflight = rng.range(0, 1);
  int32_t ladder[64];
  CHECK(wavepp_mpu_budget_ladder(&cfg, ladder, 64) > 0, "ladder");
  wavepp_mpu_t* m = nullptr;
  CHECK(wavepp_mpu_create(&cfg, &m) == WAVEPP_OK, "mpu create");
  std::vector<wavepp_span> spans(cfg.max_lanes);
  int next_id = 0;
  for (int step = 0; step < 200; ++step) {
    const int op = rng.range(0, 3);
    if (op == 0) {
      const int start = rng.range(0, 5000);
      wavepp_mpu_admit(m, next_id++, start, start + rng.range(0, 20000));
    } else if (op == 1) {
      int32_t budget = 0;
      const int n = wavepp_mpu_plan(m, rng.range(0, 1), spans.data(), cfg.max_lanes, &budget);
      CHECK(n >= 0 && n <= cfg.max_lanes, "mpu plan %d", n);
      if (n > 0 && rng.chance(80)) wavepp_mpu_commit(m, spans.data(), rng.chance(90) ? n : rng.range(0, n));
    } else if (op == 2) {
      wavepp_mpu_retire(m);
    } else {
      wavepp_mpu_state st{};
      CHECK(wavepp_mpu_get_state(m, &st) == WAVEPP_OK && st.ring >= 0, "mpu state");
    }
  }
  wavepp_mpu_destroy(m);
}

void fuzz_hints(Rng& rng) {
  const int block = rng.range(1, 32);
  const int n_tok = rng.range(0, 40 * block);
  std::vector<int32_t> tok(n_tok);
  for (auto& t : tok) t = rng.range(0, 50);
  const int nb = n_tok / block;
  std::vector<uint8_t> dig(size_t(std::max(nb, 1)) * 32);
  std::vector<uint64_t> keys(std::max(nb, 1));
  std::vector<int64_t> extra(std::max(nb, 1) * 2, 7);
  const uint8_t salt[3] = {1, 2, 3};
  const bool with_extra = rng.chance(50);
  const int64_t got = wavepp_block_hashes(tok.data(), n_tok, block, with_extra ? extra.data() : nullptr,
                                          with_extra ? 2 : 0, salt, rng.range(0, 3), dig.data(), keys.data());
  CHECK(got == nb, "hashes %lld of %d", (long long)got, nb);
  wavepp_hint_index_t* idx = nullptr;
  CHECK(wavepp_hint_index_create(rng.range(1, 16), &idx) == WAVEPP_OK, "index create");
  const int cut = nb ? rng.range(0, nb) : 0;
  wavepp_hint_index_add(idx, 1, keys.data(), cut);
  int64_t e = -1;
  int32_t probes = 0;
  CHECK(wavepp_hint_probe_prefix(idx, 1, keys.data(), nb, &e, &probes) == WAVEPP_OK && e >= cut && e <= nb,
        "prefix probe %lld (cut %d)", (long long)e, cut);
  int64_t e2 = -1;
  CHECK(wavepp_hint_probe_prefix_linear(idx, 1, keys.data(), nb, &e2, &probes) == WAVEPP_OK && e2 == e,
        "linear probe %lld vs %lld", (long long)e2, (long long)e);
  CHECK(wavepp_hint_probe_recurrent(idx, 1, keys.data(), nb ? rng.range(0, nb) : 0, &e, &probes) == WAVEPP_OK,
        "recurrent probe");
  if (cut) CHECK(wavepp_hint_index_detach(idx, 1, keys.data(), cut) == WAVEPP_OK, "detach");
  CHECK(wavepp_hint_index_size(idx) == 0, "index empty after detach");
  wavepp_hint_index_destroy(idx);
}

}  // namespace

int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 2000;
  const uint64_t seed = argc > 2 ? strtoull(argv[2], nullptr, 10) : 1;
  Rng rng(seed);
  int accepted = 0;
  for (int i = 0; i < iters && !g_fail; ++i) {
    fuzz_attention(rng);
    if (i % 4 == 0) fuzz_kda(rng);
    if (i % 20 == 0) fuzz_mpu(rng);
    if (i % 10 == 0) fuzz_hints(rng);
    accepted++;
  }
  if (g_fail) return 1;
  printf("host_fuzz ok: %d iterations, seed %llu; attention plan statuses 0..-7:", accepted,
         (unsigned long long)seed);
  for (int i = 0; i < 8; ++i) printf(" %d", g_status_count[i]);
  printf("\n");
  return 0;
}
