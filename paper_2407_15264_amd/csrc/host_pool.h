// A fork-join pool of host threads.  The cache uses it, when its backing store
// is pageable host memory (which the GPU cannot read), to copy the rows of a
// gather's misses and victim hits into a pinned bounce buffer.
#pragma once

#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace lsm {

class HostPool {
 public:
  // `workers` threads beside the calling thread, which also takes part in run().
  explicit HostPool(unsigned workers) {
    for (unsigned i = 0; i < workers; ++i) threads_.emplace_back([this] { loop(); });
  }

  ~HostPool() {
    {
      std::lock_guard<std::mutex> lock(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    for (std::thread &t : threads_) t.join();
  }

  HostPool(const HostPool &) = delete;
  HostPool &operator=(const HostPool &) = delete;

  // Calls body(i0, i1) for consecutive chunks [i0, i1) covering [0, n), spread
  // over the workers and the calling thread; returns once every chunk is done.
  // Not reentrant: one run at a time.
  void run(uint64_t n, uint64_t chunk, const std::function<void(uint64_t, uint64_t)> &body) {
    if (n == 0) return;
    if (chunk == 0) chunk = 1;
    {
      std::lock_guard<std::mutex> lock(mu_);
      body_ = &body;
      n_ = n;
      chunk_ = chunk;
      next_.store(0, std::memory_order_relaxed);
      active_ = (unsigned)threads_.size();
      ++generation_;
    }
    cv_.notify_all();
    work();
    std::unique_lock<std::mutex> lock(mu_);
    done_cv_.wait(lock, [this] { return active_ == 0; });
    body_ = nullptr;
  }

 private:
  void work() {
    for (;;) {
      const uint64_t i0 = next_.fetch_add(chunk_, std::memory_order_relaxed);
      if (i0 >= n_) return;
      const uint64_t i1 = i0 + chunk_ < n_ ? i0 + chunk_ : n_;
      (*body_)(i0, i1);
    }
  }

  void loop() {
    uint64_t seen = 0;
    for (;;) {
      {
        std::unique_lock<std::mutex> lock(mu_);
        cv_.wait(lock, [&] { return stop_ || generation_ != seen; });
        if (stop_) return;
        seen = generation_;
      }
      work();
      {
        std::lock_guard<std::mutex> lock(mu_);
        --active_;
      }
      done_cv_.notify_one();
    }
  }

  std::vector<std::thread> threads_;
  std::mutex mu_;
  std::condition_variable cv_, done_cv_;
  const std::function<void(uint64_t, uint64_t)> *body_ = nullptr;
  uint64_t n_ = 0, chunk_ = 1;
  std::atomic<uint64_t> next_{0};
  unsigned active_ = 0;
  uint64_t generation_ = 0;
  bool stop_ = false;
};

}  // namespace lsm
