// Stress test of the staging copy pool: many sizes, offsets and concurrent
// callers; every copy is checked byte by byte.  Built with g++ (optionally
// with ThreadSanitizer) by tests/test_copy_pool.py.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <thread>
#include <vector>

#include "../../paper_2607_29678_amd/csrc/tt_copy.h"

static int run(int id, int iters) {
  std::mt19937_64 rng(0xC0FFEEu + id);
  std::vector<uint8_t> src(3 << 20), dst(3 << 20);
  for (auto& b : src) b = (uint8_t)rng();
  for (int it = 0; it < iters; ++it) {
    const size_t n = (it % 3 == 0) ? (size_t)(rng() % 4096) : (size_t)(rng() % (2 << 20));
    const size_t so = rng() % 4096, doff = rng() % 4096;
    std::memset(dst.data(), 0xA5, dst.size());
    if (it % 7 == 0) tt::host_copy_wake(n);
    tt::host_copy(dst.data() + doff, src.data() + so, n);
    if (std::memcmp(dst.data() + doff, src.data() + so, n) != 0) {
      std::printf("caller %d iteration %d: copy of %zu bytes differs\n", id, it, n);
      return 1;
    }
    for (size_t k = 0; k < doff; ++k)
      if (dst[k] != 0xA5) {
        std::printf("caller %d iteration %d: write before the destination\n", id, it);
        return 1;
      }
    for (size_t k = doff + n; k < dst.size(); ++k)
      if (dst[k] != 0xA5) {
        std::printf("caller %d iteration %d: write after the destination\n", id, it);
        return 1;
      }
    if (it % 50 == 49) std::this_thread::sleep_for(std::chrono::milliseconds(3));  // workers go to sleep
  }
  return 0;
}

int main(int argc, char** argv) {
  const int callers = argc > 1 ? std::atoi(argv[1]) : 3;
  const int iters = argc > 2 ? std::atoi(argv[2]) : 300;
  std::vector<int> rc(callers, 0);
  std::vector<std::thread> th;
  for (int c = 0; c < callers; ++c) th.emplace_back([&, c] { rc[c] = run(c, iters); });
  for (auto& t : th) t.join();
  for (int r : rc)
    if (r) return 1;
  std::printf("ok\n");
  return 0;
}
