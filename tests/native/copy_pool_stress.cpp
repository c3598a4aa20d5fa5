// Stress test of the staging copy pool: many sizes, offsets and concurrent
// callers, plain and widening (16- or 24-bit values into int32) copies; every
// copy is checked value by value, and the bytes around the destination must
// stay untouched.  Built with g++ (optionally with ThreadSanitizer) by
// tests/test_copy_pool.py.
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
    const bool wide = it % 3 == 1;  // a widening copy of n / 4 16-bit values into n bytes of int32
    size_t n_out = n;
    if (wide) {
      n_out = n & ~(size_t)3;
      const uint16_t* s16 = reinterpret_cast<const uint16_t*>(src.data() + (so & ~(size_t)1));
      // every second widening copy also takes bits 16..23 from a byte array
      const uint8_t* hi = (it / 3) % 2 ? src.data() + (2 << 20) + (so % 777) : nullptr;
      int32_t* d32 = reinterpret_cast<int32_t*>(dst.data() + (doff & ~(size_t)3));
      tt::host_widen(d32, s16, hi, n_out / 4);
      for (size_t i = 0; i < n_out / 4; ++i)
        if (d32[i] != (int32_t)((uint32_t)s16[i] | (hi ? (uint32_t)hi[i] << 16 : 0u))) {
          std::printf("caller %d iteration %d: widened value %zu of %zu differs\n", id, it, i, n_out / 4);
          return 1;
        }
    } else {
      tt::host_copy(dst.data() + doff, src.data() + so, n);
      if (std::memcmp(dst.data() + doff, src.data() + so, n) != 0) {
        std::printf("caller %d iteration %d: copy of %zu bytes differs\n", id, it, n);
        return 1;
      }
    }
    const size_t d0 = wide ? (doff & ~(size_t)3) : doff;
    for (size_t k = 0; k < d0; ++k)
      if (dst[k] != 0xA5) {
        std::printf("caller %d iteration %d: write before the destination\n", id, it);
        return 1;
      }
    for (size_t k = d0 + n_out; k < dst.size(); ++k)
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
