// Maximum Pipeline Utilization wave planner (Design of WavePP, "Pipeline Scheduling"): budget
// choice over the halving ladder (Eq. 6) from the estimate n(b) = max(W / b, N_{>b/2}) (Eq. 7),
// with the split limit and the hysteresis, and first-come-first-served packing of the admitted
// requests into waves.  All decisions are integer comparisons.
#include "wavepp_mpu.h"
#include "internal.h"

#include <algorithm>
#include <deque>
#include <new>
#include <unordered_map>
#include <vector>

using namespace wavepp;

namespace {

struct Req {
  int32_t id;
  int32_t pos;            // next unscheduled token
  int32_t end;
  int32_t last_len = 0;   // length of the most recent committed chunk
  int64_t last_wave = 0;  // its wave serial, 0 = none
};

int check_config(const wavepp_mpu_config* c) {
  if (!c) return set_error(WAVEPP_EINVAL, "config is NULL");
  if (c->block <= 0 || c->max_budget <= 0 || c->min_budget <= 0 || c->max_budget % c->block ||
      c->min_budget % c->block || c->min_budget < c->block || c->min_budget > c->max_budget)
    return set_error(WAVEPP_EINVAL, "need B | M, B | b_min and B <= b_min <= M (M=%d, b_min=%d, B=%d)",
                     c->max_budget, c->min_budget, c->block);
  if (c->stages < 1 || c->fills < 1 || c->max_lanes < 1) return set_error(WAVEPP_EINVAL, "stages, fills and max_lanes must be >= 1");
  if (c->split_permille < 0 || c->split_permille > 1000) return set_error(WAVEPP_EINVAL, "split_permille outside [0, 1000]");
  if (c->count_inflight != 0 && c->count_inflight != 1) return set_error(WAVEPP_EINVAL, "count_inflight must be 0 or 1");
  if (int64_t(c->stages) * (c->fills + 1) > (1 << 20)) return set_error(WAVEPP_EINVAL, "stages x fills too large");
  return WAVEPP_OK;
}

std::vector<int32_t> make_ladder(const wavepp_mpu_config& c) {
  std::vector<int32_t> l{c.max_budget};
  while (l.back() > c.min_budget) l.push_back(std::max(c.min_budget, (l.back() / 2) / c.block * c.block));
  return l;
}

}  // namespace

struct wavepp_mpu_s {
  wavepp_mpu_config cfg;
  std::vector<int32_t> ladder;
  int32_t R = 0, S = 0;
  std::vector<Req> reqs;                          // admission order
  std::unordered_map<int32_t, size_t> index;      // id -> position in reqs
  int64_t next_serial = 1;
  int64_t ring_first = 1;                         // serials in the ring: [ring_first, next_serial)
  int32_t budget = 0;
  int32_t up = 0, down = 0;
  bool waited = false;
  std::vector<int64_t> pieces;                    // scratch

  int32_t ring_size() const { return int32_t(next_serial - ring_first); }
  int64_t inflight(const Req& r) const {
    return (cfg.count_inflight && r.last_wave >= ring_first && r.last_wave > 0) ? r.last_len : 0;
  }
  int64_t gather_work() {
    int64_t W = 0;
    pieces.clear();
    for (const Req& r : reqs) {
      const int64_t rem = int64_t(r.end) - r.pos, inf = inflight(r);
      W += rem + inf;
      if (rem > 0) pieces.push_back(rem);
      if (inf > 0) pieces.push_back(inf);
    }
    return W;
  }
  int64_t big_pieces(int64_t b) const {
    int64_t n = 0;
    for (int64_t p : pieces) n += (2 * p > b);
    return n;
  }
  bool at_least(int64_t W, int64_t b, int64_t x) const { return W >= x * b || big_pieces(b) >= x; }
  bool at_most(int64_t W, int64_t b, int64_t x) const { return W <= x * b && big_pieces(b) <= x; }

  int32_t choose(int64_t W) const {
    for (size_t j = 0; j < ladder.size(); ++j) {
      const int64_t b = ladder[j];
      if (at_least(W, b, S)) return int32_t(b);
      if (j + 1 < ladder.size() && at_least(W, b, R)) {
        const int64_t nxt = ladder[j + 1];
        int64_t split = 0;
        for (int64_t p : pieces) split += (p > nxt && p <= b) ? p : 0;
        if (split * 1000 > int64_t(cfg.split_permille) * W) return int32_t(b);
      }
    }
    return ladder.back();
  }
  int ladder_pos(int32_t b) const { return int(std::find(ladder.begin(), ladder.end(), b) - ladder.begin()); }

  void update_budget(int32_t target, int64_t W) {
    if (budget == 0) {
      budget = target;
      return;
    }
    const int cur = ladder_pos(budget), tgt = ladder_pos(target);
    if (tgt == cur) {
      up = down = 0;
    } else if (tgt < cur) {
      down = 0;
      if (cur - tgt >= 2) {
        budget = target;
        up = 0;
      } else if (++up >= R / 2) {
        budget = target;
        up = 0;
      }
    } else {
      up = 0;
      ++down;
      if (down >= R && at_most(W, budget, S - 1)) {
        budget = target;
        down = 0;
      }
    }
  }

  void compact() {
    std::vector<Req> keep;
    keep.reserve(reqs.size());
    for (const Req& r : reqs)
      if (r.pos < r.end || inflight(r) > 0) keep.push_back(r);
    if (keep.size() == reqs.size()) return;
    reqs.swap(keep);
    index.clear();
    for (size_t i = 0; i < reqs.size(); ++i) index[reqs[i].id] = i;
  }
};

extern "C" {

int wavepp_mpu_budget_ladder(const wavepp_mpu_config* config, int32_t* out, int32_t capacity) {
  clear_error();
  int st = check_config(config);
  if (st) return st;
  if (capacity < 0 || (capacity > 0 && !out)) return set_error(WAVEPP_EINVAL, "bad output buffer");
  const std::vector<int32_t> l = make_ladder(*config);
  for (int32_t i = 0; i < std::min<int32_t>(capacity, int32_t(l.size())); ++i) out[i] = l[i];
  return int32_t(l.size());
}

int wavepp_mpu_create(const wavepp_mpu_config* config, wavepp_mpu_t** out) {
  clear_error();
  if (!out) return set_error(WAVEPP_EINVAL, "out is NULL");
  *out = nullptr;
  int st = check_config(config);
  if (st) return st;
  auto p = new (std::nothrow) wavepp_mpu_s();
  if (!p) return set_error(WAVEPP_EINVAL, "out of host memory");
  p->cfg = *config;
  p->ladder = make_ladder(*config);
  p->R = 2 * config->stages;
  p->S = p->R + (config->fills - 1) * config->stages;
  *out = p;
  return WAVEPP_OK;
}

int wavepp_mpu_admit(wavepp_mpu_t* p, int32_t request, int32_t start, int32_t end) {
  clear_error();
  if (!p) return set_error(WAVEPP_EINVAL, "planner is NULL");
  if (start < 0 || end <= start) return set_error(WAVEPP_EINVAL, "need 0 <= start < end (%d, %d)", start, end);
  if (p->index.count(request)) return set_error(WAVEPP_EINVAL, "request %d already admitted", request);
  p->index[request] = p->reqs.size();
  p->reqs.push_back(Req{request, start, end});
  return WAVEPP_OK;
}

int wavepp_mpu_plan(wavepp_mpu_t* p, int32_t admission_pending, wavepp_span* spans, int32_t capacity,
                    int32_t* budget) {
  clear_error();
  if (!p || !budget) return set_error(WAVEPP_EINVAL, "null argument");
  if (capacity < p->cfg.max_lanes || !spans) return set_error(WAVEPP_EINVAL, "span capacity below max_lanes");
  *budget = p->budget;
  if (p->ring_size() >= p->R) return 0;
  const int64_t W = p->gather_work();
  if (W == 0) return 0;
  p->update_budget(p->choose(W), W);
  const int32_t b = p->budget;
  *budget = b;
  const int64_t floor = std::max<int64_t>(p->cfg.min_budget, b / 2);
  int64_t space = b;
  int32_t n = 0;
  for (const Req& r : p->reqs) {
    const int64_t rem = int64_t(r.end) - r.pos;
    if (rem == 0) continue;
    if (n == p->cfg.max_lanes || space == 0) break;
    const int64_t take = std::min(rem, space);
    if (take < rem && take < floor) break;
    spans[n++] = wavepp_span{r.id, r.pos, int32_t(take)};
    space -= take;
  }
  if (n == 1 && 2 * int64_t(spans[0].length) < b && p->ring_size() > 0 && admission_pending && !p->waited) {
    p->waited = true;
    return 0;
  }
  return n;
}

int wavepp_mpu_commit(wavepp_mpu_t* p, const wavepp_span* spans, int32_t n) {
  clear_error();
  if (!p || (n > 0 && !spans) || n < 0) return set_error(WAVEPP_EINVAL, "bad arguments");
  if (p->ring_size() >= p->R) return set_error(WAVEPP_EINVAL, "ring full (%d waves)", p->R);
  std::vector<size_t> at(static_cast<size_t>(n), 0);
  for (int32_t i = 0; i < n; ++i) {
    auto f = p->index.find(spans[i].request);
    if (f == p->index.end()) return set_error(WAVEPP_EINVAL, "span %d: unknown request %d", i, spans[i].request);
    for (int32_t j = 0; j < i; ++j)
      if (spans[j].request == spans[i].request) return set_error(WAVEPP_EINVAL, "request %d appears twice", spans[i].request);
    const Req& r = p->reqs[f->second];
    if (spans[i].start != r.pos)
      return set_error(WAVEPP_EPOSITION, "request %d: span starts at %d, the request is at %d", r.id, spans[i].start, r.pos);
    if (spans[i].length <= 0 || spans[i].length > r.end - r.pos)
      return set_error(WAVEPP_EINVAL, "request %d: span length %d outside (0, %d]", r.id, spans[i].length, r.end - r.pos);
    at[size_t(i)] = f->second;
  }
  const int64_t serial = p->next_serial++;
  for (int32_t i = 0; i < n; ++i) {
    Req& r = p->reqs[at[size_t(i)]];
    r.pos += spans[i].length;
    r.last_len = spans[i].length;
    r.last_wave = serial;
  }
  p->waited = false;
  return int(serial);
}

int wavepp_mpu_retire(wavepp_mpu_t* p) {
  clear_error();
  if (!p) return set_error(WAVEPP_EINVAL, "planner is NULL");
  if (p->ring_size() == 0) return set_error(WAVEPP_EINVAL, "ring empty");
  ++p->ring_first;
  p->compact();
  return WAVEPP_OK;
}

int wavepp_mpu_get_state(const wavepp_mpu_t* p, wavepp_mpu_state* s) {
  if (!p || !s) return set_error(WAVEPP_EINVAL, "null argument");
  int64_t W = 0;
  for (const Req& r : p->reqs) W += int64_t(r.end) - r.pos + p->inflight(r);
  s->work = W;
  s->budget = p->budget;
  s->ring = p->ring_size();
  s->requests = int32_t(p->reqs.size());
  s->up_count = p->up;
  s->down_count = p->down;
  return WAVEPP_OK;
}

void wavepp_mpu_destroy(wavepp_mpu_t* p) { delete p; }

}  // extern "C"
