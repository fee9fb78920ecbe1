// Reuse hints (Design of WavePP, "Fast Reuse Hints"): chained block hashes (Eq. 5) with SHA-256,
// a sharded counted index of (window, key), and the dense-prefix (gallop + bisect) and recurrent
// (backward scan) probes.
#include "wavepp_hints.h"
#include "internal.h"

#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <unordered_map>
#include <vector>

using namespace wavepp;

namespace {

// ---------------------------------------------------------------------------------------------
// SHA-256 (FIPS 180-4).  The round constants are the first 32 bits of the fractional parts of
// the cube roots of the first 64 primes, and the initial state those of the square roots of the
// first 8 primes; both are derived here exactly with integer roots.
// ---------------------------------------------------------------------------------------------
typedef unsigned __int128 u128;

uint64_t iroot(u128 n, int k) {           // floor(n^(1/k)), k = 2 or 3, n < 2^110
  uint64_t lo = 0, hi = uint64_t(1) << 37;
  while (hi - lo > 1) {
    const uint64_t mid = lo + (hi - lo) / 2;
    u128 p = u128(mid) * mid;
    if (k == 3) p *= mid;
    if (p <= n) lo = mid; else hi = mid;
  }
  return lo;
}

struct ShaTables {
  uint32_t k[64];
  uint32_t h0[8];
  ShaTables() {
    int found = 0;
    for (uint32_t c = 2; found < 64; ++c) {
      bool prime = true;
      for (uint32_t d = 2; d * d <= c; ++d)
        if (c % d == 0) { prime = false; break; }
      if (!prime) continue;
      k[found] = uint32_t(iroot(u128(c) << 96, 3));          // frac(cbrt(c)) * 2^32, low 32 bits
      if (found < 8) h0[found] = uint32_t(iroot(u128(c) << 64, 2));
      ++found;
    }
  }
};

const ShaTables& sha_tables() {
  static const ShaTables t;
  return t;
}

inline uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

class Sha256 {
 public:
  Sha256() : t_(sha_tables()) { memcpy(h_, t_.h0, sizeof(h_)); }
  void update(const uint8_t* p, size_t n) {
    len_ += n;
    while (n) {
      const size_t take = std::min(n, size_t(64) - fill_);
      memcpy(buf_ + fill_, p, take);
      fill_ += take;
      p += take;
      n -= take;
      if (fill_ == 64) {
        block(buf_);
        fill_ = 0;
      }
    }
  }
  void finish(uint8_t out[32]) {
    const uint64_t bits = uint64_t(len_) * 8;
    const uint8_t one = 0x80, zero = 0;
    update(&one, 1);
    while (fill_ != 56) update(&zero, 1);
    uint8_t lenb[8];
    for (int i = 0; i < 8; ++i) lenb[i] = uint8_t(bits >> (56 - 8 * i));
    update(lenb, 8);
    for (int i = 0; i < 8; ++i)
      for (int j = 0; j < 4; ++j) out[4 * i + j] = uint8_t(h_[i] >> (24 - 8 * j));
  }

 private:
  void block(const uint8_t* b) {
    uint32_t w[64];
    for (int i = 0; i < 16; ++i)
      w[i] = (uint32_t(b[4 * i]) << 24) | (uint32_t(b[4 * i + 1]) << 16) | (uint32_t(b[4 * i + 2]) << 8) | b[4 * i + 3];
    for (int i = 16; i < 64; ++i) {
      const uint32_t s0 = rotr(w[i - 15], 7) ^ rotr(w[i - 15], 18) ^ (w[i - 15] >> 3);
      const uint32_t s1 = rotr(w[i - 2], 17) ^ rotr(w[i - 2], 19) ^ (w[i - 2] >> 10);
      w[i] = w[i - 16] + s0 + w[i - 7] + s1;
    }
    uint32_t a = h_[0], bb = h_[1], c = h_[2], d = h_[3], e = h_[4], f = h_[5], g = h_[6], h = h_[7];
    for (int i = 0; i < 64; ++i) {
      const uint32_t S1 = rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25);
      const uint32_t ch = (e & f) ^ (~e & g);
      const uint32_t t1 = h + S1 + ch + t_.k[i] + w[i];
      const uint32_t S0 = rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22);
      const uint32_t mj = (a & bb) ^ (a & c) ^ (bb & c);
      const uint32_t t2 = S0 + mj;
      h = g;
      g = f;
      f = e;
      e = d + t1;
      d = c;
      c = bb;
      bb = a;
      a = t1 + t2;
    }
    h_[0] += a;
    h_[1] += bb;
    h_[2] += c;
    h_[3] += d;
    h_[4] += e;
    h_[5] += f;
    h_[6] += g;
    h_[7] += h;
  }
  const ShaTables& t_;
  uint32_t h_[8];
  uint8_t buf_[64];
  size_t fill_ = 0;
  size_t len_ = 0;
};

void put_le32(uint8_t* p, uint32_t v) {
  for (int i = 0; i < 4; ++i) p[i] = uint8_t(v >> (8 * i));
}
void put_le64(uint8_t* p, uint64_t v) {
  for (int i = 0; i < 8; ++i) p[i] = uint8_t(v >> (8 * i));
}
uint64_t get_le64(const uint8_t* p) {
  uint64_t v = 0;
  for (int i = 0; i < 8; ++i) v |= uint64_t(p[i]) << (8 * i);
  return v;
}

// ---------------------------------------------------------------------------------------------
// Sharded counted index
// ---------------------------------------------------------------------------------------------
struct WKey {
  int32_t window;
  uint64_t key;
  bool operator==(const WKey& o) const { return window == o.window && key == o.key; }
};
struct WKeyHash {
  size_t operator()(const WKey& k) const { return size_t(k.key ^ (uint64_t(uint32_t(k.window)) * 0x9E3779B97F4A7C15ull)); }
};
struct Shard {
  std::mutex mu;
  std::unordered_map<WKey, int64_t, WKeyHash> count;
};

}  // namespace

struct wavepp_hint_index_s {
  std::vector<std::unique_ptr<Shard>> shards;
  Shard& shard_of(int32_t window, uint64_t key) {
    // the key is already a hash: its high bits choose the shard
    const uint64_t mixed = (key >> 32) ^ (key << 7) ^ uint64_t(uint32_t(window));
    return *shards[size_t(mixed % shards.size())];
  }
  bool contains(int32_t window, uint64_t key) {
    Shard& s = shard_of(window, key);
    std::lock_guard<std::mutex> lock(s.mu);
    return s.count.count(WKey{window, key}) != 0;
  }
};

extern "C" {

int64_t wavepp_block_hashes(const int32_t* tokens, int64_t n_tokens, int32_t block, const int64_t* extra_keys,
                            int32_t extra_per_block, const uint8_t* salt, int32_t salt_len, uint8_t* digests,
                            uint64_t* keys) {
  clear_error();
  if (block <= 0 || n_tokens < 0 || extra_per_block < 0 || salt_len < 0)
    return set_error(WAVEPP_EINVAL, "bad sizes (block=%d, n_tokens=%lld)", block, (long long)n_tokens);
  if ((n_tokens > 0 && !tokens) || (extra_per_block > 0 && !extra_keys) || (salt_len > 0 && !salt))
    return set_error(WAVEPP_EINVAL, "null input");
  const int64_t nb = n_tokens / block;
  uint8_t parent[32] = {0};
  std::vector<uint8_t> scratch(size_t(block) * 4 + size_t(extra_per_block) * 8);
  for (int64_t b = 0; b < nb; ++b) {
    Sha256 h;
    if (salt_len) h.update(salt, size_t(salt_len));
    h.update(parent, 32);
    uint8_t* q = scratch.data();
    for (int32_t j = 0; j < extra_per_block; ++j, q += 8) put_le64(q, uint64_t(extra_keys[b * extra_per_block + j]));
    for (int32_t j = 0; j < block; ++j, q += 4) put_le32(q, uint32_t(tokens[b * block + j]));
    h.update(scratch.data(), scratch.size());
    h.finish(parent);
    if (digests) memcpy(digests + 32 * b, parent, 32);
    if (keys) keys[b] = get_le64(parent);
  }
  return nb;
}

int wavepp_hint_index_create(int32_t num_shards, wavepp_hint_index_t** out) {
  clear_error();
  if (!out || num_shards < 1 || num_shards > 65536) return set_error(WAVEPP_EINVAL, "need 1 <= num_shards <= 65536");
  *out = nullptr;
  auto idx = new (std::nothrow) wavepp_hint_index_s();
  if (!idx) return set_error(WAVEPP_EINVAL, "out of host memory");
  for (int32_t i = 0; i < num_shards; ++i) idx->shards.emplace_back(new Shard());
  *out = idx;
  return WAVEPP_OK;
}

int wavepp_hint_index_add(wavepp_hint_index_t* idx, int32_t window, const uint64_t* keys, int64_t n) {
  clear_error();
  if (!idx || n < 0 || (n > 0 && !keys)) return set_error(WAVEPP_EINVAL, "bad arguments");
  for (int64_t i = 0; i < n; ++i) {
    Shard& s = idx->shard_of(window, keys[i]);
    std::lock_guard<std::mutex> lock(s.mu);
    ++s.count[WKey{window, keys[i]}];
  }
  return WAVEPP_OK;
}

int wavepp_hint_index_detach(wavepp_hint_index_t* idx, int32_t window, const uint64_t* keys, int64_t n) {
  clear_error();
  if (!idx || n < 0 || (n > 0 && !keys)) return set_error(WAVEPP_EINVAL, "bad arguments");
  for (int64_t i = 0; i < n; ++i) {
    Shard& s = idx->shard_of(window, keys[i]);
    std::lock_guard<std::mutex> lock(s.mu);
    auto it = s.count.find(WKey{window, keys[i]});
    if (it == s.count.end())
      return set_error(WAVEPP_EINVAL, "detach of key %016llx (window %d), which is not indexed",
                       (unsigned long long)keys[i], window);
    if (--it->second == 0) s.count.erase(it);
  }
  return WAVEPP_OK;
}

int64_t wavepp_hint_index_size(wavepp_hint_index_t* idx) {
  if (!idx) return set_error(WAVEPP_EINVAL, "index is NULL");
  int64_t n = 0;
  for (auto& s : idx->shards) {
    std::lock_guard<std::mutex> lock(s->mu);
    n += int64_t(s->count.size());
  }
  return n;
}

int wavepp_hint_probe_prefix(wavepp_hint_index_t* idx, int32_t window, const uint64_t* keys, int64_t n,
                             int64_t* endpoint, int32_t* probes) {
  clear_error();
  if (!idx || !endpoint || n < 0 || (n > 0 && !keys)) return set_error(WAVEPP_EINVAL, "bad arguments");
  int32_t np = 0;
  auto present = [&](int64_t depth) {     // are the first `depth` blocks reusable? (probe block depth - 1)
    ++np;
    return idx->contains(window, keys[depth - 1]);
  };
  int64_t good = 0, bad = n + 1;          // depth `good` is known present, `bad` known absent
  if (n > 0) {
    for (int64_t d = 1;; d *= 2) {
      const int64_t depth = d < n ? d : n;
      if (present(depth)) {
        good = depth;
        if (depth == n) break;
      } else {
        bad = depth;
        break;
      }
    }
    while (bad <= n && bad - good > 1) {
      const int64_t mid = good + (bad - good) / 2;
      if (present(mid)) good = mid; else bad = mid;
    }
  }
  *endpoint = good;
  if (probes) *probes = np;
  return WAVEPP_OK;
}

int wavepp_hint_probe_prefix_linear(wavepp_hint_index_t* idx, int32_t window, const uint64_t* keys, int64_t n,
                                    int64_t* endpoint, int32_t* probes) {
  clear_error();
  if (!idx || !endpoint || n < 0 || (n > 0 && !keys)) return set_error(WAVEPP_EINVAL, "bad arguments");
  int64_t e = 0;
  int32_t np = 0;
  while (e < n) {
    ++np;
    if (!idx->contains(window, keys[e])) break;
    ++e;
  }
  *endpoint = e;
  if (probes) *probes = np;
  return WAVEPP_OK;
}

int wavepp_hint_probe_recurrent(wavepp_hint_index_t* idx, int32_t window, const uint64_t* keys, int64_t limit,
                                int64_t* endpoint, int32_t* probes) {
  clear_error();
  if (!idx || !endpoint || limit < 0 || (limit > 0 && !keys)) return set_error(WAVEPP_EINVAL, "bad arguments");
  int64_t j = limit;
  int32_t np = 0;
  for (; j > 0; --j) {
    ++np;
    if (idx->contains(window, keys[j - 1])) break;
  }
  *endpoint = j;
  if (probes) *probes = np;
  return WAVEPP_OK;
}

void wavepp_hint_index_destroy(wavepp_hint_index_t* idx) { delete idx; }

}  // extern "C"
