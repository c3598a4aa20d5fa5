// Parallel host copies for the staging of blocking calls.
//
// A request of a million characters moves about 1 MB into pinned staging and
// its IDs out of it (0.6 to 1.2 MB, with 2 to 4 bytes per staged ID, widened
// to 4 in the caller's array).  One core copies memory that is not in its caches
// at about 25 GB/s, so those two copies would take longer than the GPU's work
// on the request.  A few worker threads split each copy into chunks that they
// take from a shared counter together with the calling thread (the caller
// alone finishes a copy that no worker joins).  Workers spin for a short while
// after each copy and after a wake-up, then sleep on a condition variable, so
// that back-to-back requests find them awake and an idle process costs
// nothing.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

#include "tt_copy.h"

namespace tt {
namespace {

constexpr size_t PAR_MIN = 256 * 1024;   // smaller copies stay on the calling thread
constexpr size_t CHUNK = 64 * 1024;      // bytes per chunk
constexpr int MAX_WORKERS = 3;
constexpr auto SPIN_FOR = std::chrono::milliseconds(2);

class CopyPool {
 public:
  CopyPool() {
    const unsigned hc = std::thread::hardware_concurrency();
    const int n = std::min<int>(MAX_WORKERS, hc >= 8 ? (int)(hc / 4) : 0);
    for (int i = 0; i < n; ++i) threads_.emplace_back([this] { run(); });
  }
  ~CopyPool() {
    {
      std::lock_guard<std::mutex> g(m_);
      stop_.store(true);
    }
    cv_.notify_all();
    for (auto& t : threads_) t.join();
  }

  // Workers that sleep start spinning (a copy is coming soon).
  void wake() {
    if (sleeping_.load(std::memory_order_acquire) == 0) return;
    {
      std::lock_guard<std::mutex> g(m_);
      wake_gen_.fetch_add(1, std::memory_order_release);
    }
    cv_.notify_all();
  }

  // wide: src holds n / 4 16-bit values that dst receives as int32 (n bytes),
  // with bits 16..23 from hi when hi is set
  void copy(void* dst, const void* src, size_t n, bool wide = false, const uint8_t* hi = nullptr) {
    if (n < PAR_MIN || threads_.empty() || !job_mu_.try_lock()) {
      run_chunk(static_cast<uint8_t*>(dst), static_cast<const uint8_t*>(src), hi, 0, n, wide);
      return;
    }
    const uint64_t seq = seq_.load(std::memory_order_relaxed) + 1;
    // Chunk indices carry the copy's sequence number.  First no chunk can be
    // taken at all, then the fields change, then this copy's chunks open: a
    // worker still holding an earlier copy's sequence number takes nothing.
    next_.store((seq << 32) | 0xFFFFFFFFull, std::memory_order_seq_cst);
    dst_.store(static_cast<uint8_t*>(dst), std::memory_order_relaxed);
    src_.store(static_cast<const uint8_t*>(src), std::memory_order_relaxed);
    n_.store(n, std::memory_order_relaxed);
    wide_.store(wide, std::memory_order_relaxed);
    hi_.store(hi, std::memory_order_relaxed);
    n_chunks_.store((uint32_t)((n + CHUNK - 1) / CHUNK), std::memory_order_relaxed);
    done_.store(0, std::memory_order_relaxed);
    next_.store(seq << 32, std::memory_order_release);
    seq_.store(seq, std::memory_order_seq_cst);
    if (sleeping_.load(std::memory_order_seq_cst) != 0) cv_.notify_all();
    work(seq);
    const uint32_t total = n_chunks_.load(std::memory_order_relaxed);
    while (done_.load(std::memory_order_acquire) != total) __builtin_ia32_pause();
    job_mu_.unlock();
  }

 private:
  // Take and copy chunks of copy `seq` until none is left.  A chunk taken with
  // a successful exchange belongs to copy `seq`, whose fields stay put until
  // every chunk of it is done.
  void work(uint64_t seq) {
    for (;;) {
      uint64_t v = next_.load(std::memory_order_acquire);
      uint32_t i;
      do {
        if ((v >> 32) != seq) return;
        i = (uint32_t)v;
        if (i >= n_chunks_.load(std::memory_order_relaxed)) return;
      } while (!next_.compare_exchange_weak(v, v + 1, std::memory_order_acq_rel));
      const size_t n = n_.load(std::memory_order_relaxed);
      const size_t a = (size_t)i * CHUNK, b = std::min(n, a + CHUNK);
      run_chunk(dst_.load(std::memory_order_relaxed), src_.load(std::memory_order_relaxed),
                hi_.load(std::memory_order_relaxed), a, b, wide_.load(std::memory_order_relaxed));
      done_.fetch_add(1, std::memory_order_acq_rel);
    }
  }

  // Output bytes [a, b) of a copy (for a widening copy a and b are multiples
  // of 4: CHUNK is, and so is n).
  static void run_chunk(uint8_t* dst, const uint8_t* src, const uint8_t* hi, size_t a, size_t b, bool wide) {
    if (!wide) {
      std::memcpy(dst + a, src + a, b - a);
      return;
    }
    int32_t* d = reinterpret_cast<int32_t*>(dst);
    const uint16_t* s = reinterpret_cast<const uint16_t*>(src);
    if (hi == nullptr) {
      for (size_t i = a / 4; i < b / 4; ++i) d[i] = (int32_t)s[i];
    } else {
      for (size_t i = a / 4; i < b / 4; ++i) d[i] = (int32_t)((uint32_t)s[i] | ((uint32_t)hi[i] << 16));
    }
  }

  void run() {
    uint64_t seen = seq_.load(std::memory_order_acquire);
    uint64_t woke = wake_gen_.load(std::memory_order_acquire);
    for (;;) {
      auto since = std::chrono::steady_clock::now();
      for (uint32_t k = 0;; ++k) {
        const uint64_t s = seq_.load(std::memory_order_acquire);
        if (s != seen) {
          seen = s;
          work(s);
          since = std::chrono::steady_clock::now();
        }
        if (stop_.load(std::memory_order_relaxed)) return;
        if ((k & 255u) == 0u && std::chrono::steady_clock::now() - since > SPIN_FOR) break;
        __builtin_ia32_pause();
      }
      std::unique_lock<std::mutex> lk(m_);
      sleeping_.fetch_add(1, std::memory_order_seq_cst);
      cv_.wait(lk, [&] {
        return stop_.load() || seq_.load(std::memory_order_seq_cst) != seen ||
               wake_gen_.load(std::memory_order_acquire) != woke;
      });
      sleeping_.fetch_sub(1, std::memory_order_seq_cst);
      woke = wake_gen_.load(std::memory_order_acquire);
      if (stop_.load()) return;
    }
  }

  std::vector<std::thread> threads_;
  std::mutex job_mu_;  // one copy at a time; other callers copy alone
  std::mutex m_;
  std::condition_variable cv_;
  std::atomic<bool> stop_{false};
  std::atomic<int> sleeping_{0};
  std::atomic<uint64_t> wake_gen_{0};
  std::atomic<uint64_t> seq_{0};
  std::atomic<uint64_t> next_{0};
  std::atomic<uint32_t> done_{0};
  std::atomic<uint8_t*> dst_{nullptr};
  std::atomic<const uint8_t*> src_{nullptr};
  std::atomic<size_t> n_{0};
  std::atomic<bool> wide_{false};
  std::atomic<const uint8_t*> hi_{nullptr};
  std::atomic<uint32_t> n_chunks_{0};
};

CopyPool& pool() {
  static CopyPool p;
  return p;
}

}  // namespace

void host_copy_wake(size_t n) {
  if (n >= PAR_MIN) pool().wake();
}

void host_copy(void* dst, const void* src, size_t n) { pool().copy(dst, src, n); }

void host_widen(int32_t* dst, const uint16_t* lo, const uint8_t* hi, size_t count) {
  pool().copy(dst, lo, 4 * count, true, hi);
}

}  // namespace tt
