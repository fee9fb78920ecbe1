// Concurrent use of the sharded hint index, for a build under the thread sanitizer (and a plain
// build): writer threads add and detach their own prompts' block keys while reader threads run the
// gallop/bisect and backward probes over the same keys.  At the end every writer's keys are added
// once more, and each prompt's dense prefix must be whole.
//
// Usage: hints_threads [rounds]; exits non-zero on a wrong result.
#include "wavepp_hints.h"

#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <vector>

int main(int argc, char** argv) {
  const int rounds = argc > 1 ? atoi(argv[1]) : 50;
  constexpr int kThreads = 4, kBlock = 16, kBlocks = 120;
  std::vector<std::vector<uint64_t>> keys(kThreads, std::vector<uint64_t>(kBlocks));
  for (int t = 0; t < kThreads; ++t) {
    std::vector<int32_t> tok(kBlock * kBlocks);
    uint32_t x = 2463534242u + 977u * t;
    for (auto& v : tok) {
      x ^= x << 13;
      x ^= x >> 17;
      x ^= x << 5;
      v = int32_t(x % 1000);
    }
    if (wavepp_block_hashes(tok.data(), int64_t(tok.size()), kBlock, nullptr, 0, nullptr, 0, nullptr,
                            keys[t].data()) != kBlocks)
      return 2;
  }
  wavepp_hint_index_t* idx = nullptr;
  if (wavepp_hint_index_create(8, &idx) != 0) return 2;
  std::atomic<int> bad{0};
  std::vector<std::thread> th;
  for (int t = 0; t < kThreads; ++t)
    th.emplace_back([&, t] {
      for (int r = 0; r < rounds; ++r) {
        if (wavepp_hint_index_add(idx, 0, keys[t].data(), kBlocks) != 0) bad++;
        if (wavepp_hint_index_detach(idx, 0, keys[t].data(), kBlocks) != 0) bad++;
      }
      if (wavepp_hint_index_add(idx, 0, keys[t].data(), kBlocks) != 0) bad++;
    });
  for (int t = 0; t < kThreads; ++t)
    th.emplace_back([&, t] {
      for (int r = 0; r < 4 * rounds; ++r) {
        int64_t e = -1;
        int32_t probes = 0;
        if (wavepp_hint_probe_prefix(idx, 0, keys[t].data(), kBlocks, &e, &probes) != 0 || e < 0 || e > kBlocks) bad++;
        if (wavepp_hint_probe_recurrent(idx, 0, keys[t].data(), kBlocks, &e, &probes) != 0 || e < 0 || e > kBlocks)
          bad++;
        (void)wavepp_hint_index_size(idx);
      }
    });
  for (auto& x : th) x.join();
  for (int t = 0; t < kThreads; ++t) {
    int64_t e = -1;
    int32_t probes = 0;
    if (wavepp_hint_probe_prefix(idx, 0, keys[t].data(), kBlocks, &e, &probes) != 0 || e != kBlocks) bad++;
  }
  wavepp_hint_index_destroy(idx);
  if (bad.load()) {
    fprintf(stderr, "hints_threads: %d wrong results\n", bad.load());
    return 1;
  }
  printf("hints_threads ok: %d threads x %d rounds\n", 2 * kThreads, rounds);
  return 0;
}
