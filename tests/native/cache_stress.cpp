// The schedule cache (paper_2609_22755_amd/csrc/sched_cache.hpp) under
// concurrent use: threads cycle through many more distinct keys than the
// cache holds (a cache of 3 entries here, of 128 in the library), so entries
// are evicted while other threads still read them.
// Each entry owns a heap buffer filled with a pattern derived from its key;
// a thread reads its entry's whole buffer after get() returns, as a call
// reads its schedule until its kernels are enqueued.  Built with
// ThreadSanitizer or AddressSanitizer by tests/test_host_sanitizers.py: a
// buffer freed while still held shows as a use-after-free, a missing lock
// as a data race.  Prints "cache stress ok" and exits 0 on success.
#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <thread>
#include <vector>

#include "sched_cache.hpp"

namespace {

std::atomic<long> g_live{0};

struct Blob {
  std::vector<uint32_t> words;
  explicit Blob(uint32_t key) : words(256 + key % 512) {
    for (size_t i = 0; i < words.size(); ++i) words[i] = key * 2654435761u + (uint32_t)i;
    g_live.fetch_add(1);
  }
  ~Blob() {
    for (auto &w : words) w = 0xdeadbeef;   // a reader of a destroyed entry sees this
    g_live.fetch_sub(1);
  }
};

}  // namespace

int main() {
  constexpr int kThreads = 4, kKeys = 600, kIters = 6000, kCap = 3;
  nsp::LruCache<Blob> cache(kCap);
  std::atomic<int> bad{0}, builds{0};
  std::vector<std::thread> th;
  for (int t = 0; t < kThreads; ++t)
    th.emplace_back([&, t] {
      uint32_t x = 12345u + 977u * (uint32_t)t;
      for (int it = 0; it < kIters; ++it) {
        x = x * 1664525u + 1013904223u;
        const uint32_t key = (x >> 8) % kKeys;
        nsp::LruCache<Blob>::Ptr e;
        const int st = cache.get("k" + std::to_string(key), &e, [&](nsp::LruCache<Blob>::Ptr *made) {
          builds.fetch_add(1);
          *made = std::make_shared<Blob>(key);
          return 0;
        });
        if (st != 0 || !e) { bad.fetch_add(1); continue; }
        // read the entry twice, with other threads' evictions in between
        for (int pass = 0; pass < 2; ++pass) {
          for (size_t i = 0; i < e->words.size(); ++i)
            if (e->words[i] != key * 2654435761u + (uint32_t)i) { bad.fetch_add(1); break; }
          std::this_thread::yield();
        }
      }
    });
  for (auto &t : th) t.join();
  const size_t held = cache.size();
  if (bad.load() != 0 || held > (size_t)kCap || builds.load() <= kKeys) {
    std::fprintf(stderr, "cache stress failed: bad=%d held=%zu builds=%d\n", bad.load(), held, builds.load());
    return 1;
  }
  if (g_live.load() != (long)held) {
    std::fprintf(stderr, "cache stress failed: %ld live entries, %zu held\n", g_live.load(), held);
    return 1;
  }
  std::printf("cache stress ok (%d builds)\n", builds.load());
  return 0;
}
