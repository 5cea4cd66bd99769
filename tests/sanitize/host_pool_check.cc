// The host thread pool under the thread, address and undefined-behaviour
// sanitizers (built by tests/test_sanitizers.py): every index of every run is
// visited exactly once, for several pool sizes and chunk sizes.
#include "host_pool.h"
#include <cstdio>
#include <vector>
#include <atomic>
int main() {
  for (unsigned workers : {0u, 1u, 3u, 15u}) {
    lsm::HostPool pool(workers);
    for (int rep = 0; rep < 300; ++rep) {
      const uint64_t n = (rep * 7919) % 5000;
      std::vector<int> hits(n, 0);
      pool.run(n, 1 + rep % 64, [&](uint64_t i0, uint64_t i1) {
        for (uint64_t i = i0; i < i1; ++i) hits[i] += 1;
      });
      for (uint64_t i = 0; i < n; ++i)
        if (hits[i] != 1) { printf("index %lu covered %d times\n", (unsigned long)i, hits[i]); return 1; }
    }
  }
  printf("host pool ok\n");
  return 0;
}
