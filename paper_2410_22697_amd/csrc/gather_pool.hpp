// Host threads that copy rows of the pinned halo store into pinned staging
// memory: the host half of the staged link mode. The DMA engines then move
// the staged rows to the device, so that no kernel reads host memory (such
// reads hold shared memory-system resources for the whole link latency and
// slow every kernel running beside them).
#pragma once

#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

namespace ms {

class GatherPool {
 public:
  // `threads` gathering threads in all: the caller of gather() and
  // threads - 1 helpers
  explicit GatherPool(int threads) {
    try {
      for (int i = 1; i < threads; ++i) helpers_.emplace_back([this, i] { loop(i); });
    } catch (...) {  // a thread could not start: end the others before passing it on
      stop();
      throw;
    }
  }
  ~GatherPool() { stop(); }
  GatherPool(const GatherPool&) = delete;
  GatherPool& operator=(const GatherPool&) = delete;

  // dst row i = src row rows[i] (rb bytes each) for i < n; a row id outside
  // [0, nrows) gives a zero row instead of a read outside the store
  void gather(const uint8_t* src, int64_t nrows, int64_t rb, const int32_t* rows, int64_t n, uint8_t* dst) {
    if (n <= 0) return;
    const int parts = (int)helpers_.size() + 1;
    {
      std::lock_guard<std::mutex> lk(mu_);
      src_ = src;
      nrows_ = nrows;
      rb_ = rb;
      rows_ = rows;
      n_ = n;
      dst_ = dst;
      busy_ = parts - 1;
      ++gen_;
    }
    go_.notify_all();
    part(0, parts);
    std::unique_lock<std::mutex> lk(mu_);
    done_.wait(lk, [this] { return busy_ == 0; });
  }

 private:
  void stop() {
    {
      std::lock_guard<std::mutex> lk(mu_);
      stop_ = true;
    }
    go_.notify_all();
    for (auto& t : helpers_) t.join();
    helpers_.clear();
  }
  void part(int p, int parts) {
    const int64_t lo = n_ * p / parts, hi = n_ * (p + 1) / parts;
    constexpr int64_t kAhead = 8;  // rows prefetched ahead of the copy
    for (int64_t i = lo; i < hi; ++i) {
      if (i + kAhead < hi) {
        const int32_t f = rows_[i + kAhead];
        if (f >= 0 && f < nrows_) __builtin_prefetch(src_ + (int64_t)f * rb_);
      }
      const int32_t r = rows_[i];
      uint8_t* d = dst_ + i * rb_;
      if (r >= 0 && r < nrows_)
        std::memcpy(d, src_ + (int64_t)r * rb_, (size_t)rb_);
      else
        std::memset(d, 0, (size_t)rb_);
    }
  }
  void loop(int id) {
    uint64_t seen = 0;
    for (;;) {
      int parts;
      {
        std::unique_lock<std::mutex> lk(mu_);
        go_.wait(lk, [&] { return stop_ || gen_ != seen; });
        if (stop_) return;
        seen = gen_;
        parts = (int)helpers_.size() + 1;
      }
      part(id, parts);
      {
        std::lock_guard<std::mutex> lk(mu_);
        if (--busy_ == 0) done_.notify_one();
      }
    }
  }

  std::vector<std::thread> helpers_;
  std::mutex mu_;
  std::condition_variable go_, done_;
  uint64_t gen_ = 0;
  int busy_ = 0;
  bool stop_ = false;
  const uint8_t* src_ = nullptr;
  int64_t nrows_ = 0, rb_ = 0;
  const int32_t* rows_ = nullptr;
  int64_t n_ = 0;
  uint8_t* dst_ = nullptr;
};

}  // namespace ms
