// Host check of the staged fetch path's worker pool (built with ThreadSanitizer by
// tests/test_gather_pool.py): over many jobs of every size and grain, on all threads (run) and on
// the workers alone (start ... wait), every index is handed out exactly once, in whole grains.
#include "gather_pool.h"
#include <atomic>
#include <cstdio>
#include <vector>
int main() {
  using hisparse::GatherPool;
  const int T = GatherPool::host_threads(8);
  if (T < 1 || T > 8) { std::printf("bad threads %d\n", T); return 1; }
  GatherPool pool(T);
  for (int round = 0; round < 200; ++round) {
    const int64_t n = 1 + (round * 7919) % 5000, grain = 1 + round % 17;
    std::vector<std::atomic<int>> hits(n);
    for (auto& h : hits) h.store(0);
    std::atomic<int64_t> bad{0};
    const std::function<void(int64_t, int64_t)> fn = [&](int64_t b, int64_t e) {
      if (b % grain != 0 || e > n || e - b > grain || e <= b) bad.fetch_add(1);
      for (int64_t i = b; i < e; ++i) hits[i].fetch_add(1);
    };
    if (round % 2 && pool.threads() > 1) { pool.start(n, grain, fn); pool.wait(); }
    else pool.run(n, grain, fn);
    for (int64_t i = 0; i < n; ++i)
      if (hits[i].load() != 1) { std::printf("round %d index %lld hit %d times\n", round, (long long)i, hits[i].load()); return 1; }
    if (bad.load()) { std::printf("round %d: bad ranges\n", round); return 1; }
  }
  std::printf("ok %d threads\n", pool.threads());
  return 0;
}
