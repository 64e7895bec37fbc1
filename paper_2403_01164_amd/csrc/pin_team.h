// Pin team of the hybrid pin || transfer path (HeteGen Sec. 4.2, Fig. 5c: pageable
// weights are copied into pinned buffers by host threads while earlier chunks cross the
// link).  Host code only, no device calls, so it also builds alone (the ThreadSanitizer
// check of the host threads).
#pragma once
#include <string.h>

#include <algorithm>
#include <condition_variable>
#include <mutex>
#include <thread>
#include <vector>

namespace hg {

// Fork-join team for large host copies: the calling thread takes the first part,
// helpers the others (page-aligned contiguous parts).
class PinTeam {
 public:
  ~PinTeam() { shutdown(); }
  bool started() const { return parts_ > 0; }
  bool start(int threads) {
    parts_ = std::max(1, threads);
    try {
      for (int i = 1; i < parts_; ++i) th_.emplace_back([this, i] { work(i); });
    } catch (...) {
      shutdown();
      return false;
    }
    return true;
  }
  void copy(char* dst, const char* src, size_t n) {
    if (parts_ <= 1 || n < ((size_t)1 << 20)) {
      memcpy(dst, src, n);
      return;
    }
    {
      std::lock_guard<std::mutex> lk(m_);
      dst_ = dst;
      src_ = src;
      n_ = n;
      pending_ = parts_ - 1;
      ++gen_;
    }
    cv_.notify_all();
    part(dst, src, n, 0);
    std::unique_lock<std::mutex> lk(m_);
    done_.wait(lk, [&] { return pending_ == 0; });
  }
  void shutdown() {
    {
      std::lock_guard<std::mutex> lk(m_);
      stop_ = true;
    }
    cv_.notify_all();
    for (auto& t : th_) t.join();
    th_.clear();
    parts_ = 0;
    stop_ = false;
  }

 private:
  void part(char* dst, const char* src, size_t n, int i) const {
    const size_t per = (n / parts_ + 4095) & ~(size_t)4095;
    const size_t b = per * i;
    if (b >= n) return;
    memcpy(dst + b, src + b, std::min(n, b + per) - b);
  }
  void work(int i) {
    long long seen = 0;
    std::unique_lock<std::mutex> lk(m_);
    for (;;) {
      cv_.wait(lk, [&] { return stop_ || gen_ != seen; });
      if (stop_) return;
      seen = gen_;
      char* d = dst_;
      const char* s = src_;
      const size_t n = n_;
      lk.unlock();
      part(d, s, n, i);
      lk.lock();
      if (--pending_ == 0) done_.notify_one();
    }
  }
  std::vector<std::thread> th_;
  std::mutex m_;
  std::condition_variable cv_, done_;
  long long gen_ = 0;
  int pending_ = 0, parts_ = 0;
  bool stop_ = false;
  char* dst_ = nullptr;
  const char* src_ = nullptr;
  size_t n_ = 0;
};

}  // namespace hg
