// Fork-join thread pool of the host suffix: run(n, fn) calls fn(i) for every
// i in [0, n) exactly once, on the pool's threads and the calling thread, and
// returns when all calls have returned.  One run at a time per pool.
#pragma once

#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace vla {
namespace host {

// Indices of a run are handed out from one 64-bit ticket: the run's number
// in the high 32 bits, the next index in the low 32.  A thread claims an index
// only by a compare-and-swap that still sees its own run's number, so a thread
// that fell asleep at the end of one run can never take an index of the next
// one.  (A plain counter with a separate bound cannot promise that: a thread
// whose claim overshot one run can be preempted before its bound check, see
// the next run's larger bound after the counter was reset, and run an index
// that the new run hands out again, so the completion count overshoots and
// the caller waits for ever.)
class Pool {
 public:
  explicit Pool(int n) : n_(std::max(1, n)) {
    for (int i = 1; i < n_; ++i) th_.emplace_back([this] { worker(); });
  }
  ~Pool() {
    {
      std::lock_guard<std::mutex> g(mu_);
      stop_ = true;
      ++gen_;
    }
    cv_.notify_all();
    for (auto& t : th_) t.join();
  }
  int size() const { return n_; }
  // fn(i) for i in [0, n), on the pool and the calling thread; returns when all ran
  void run(int n, const std::function<void(int)>& fn) {
    if (n <= 0) return;
    if (n == 1 || n_ == 1) {
      for (int i = 0; i < n; ++i) fn(i);
      return;
    }
    uint32_t g;
    {
      std::lock_guard<std::mutex> lk(mu_);
      g = (uint32_t)++gen_;
      fn_ = &fn;
      ntask_ = n;
      done_ = 0;
      ticket_.store((uint64_t)g << 32, std::memory_order_relaxed);
    }
    cv_.notify_all();
    const int did = drain(g, n, fn);
    std::unique_lock<std::mutex> lk(mu_);
    done_ += did;
    done_cv_.wait(lk, [&] { return done_ == ntask_; });
    fn_ = nullptr;
  }

 private:
  // runs the indices of run g this thread manages to claim; returns how many.
  // A run cannot finish while a claimed index is unaccounted for, so fn stays
  // alive for every index claimed here.
  int drain(uint32_t g, int n, const std::function<void(int)>& fn) {
    int did = 0;
    uint64_t t = ticket_.load(std::memory_order_relaxed);
    for (;;) {
      if ((uint32_t)(t >> 32) != g || (int)(uint32_t)t >= n) break;
      if (!ticket_.compare_exchange_weak(t, t + 1, std::memory_order_acq_rel, std::memory_order_relaxed))
        continue;  // t now holds the current ticket
      fn((int)(uint32_t)t);
      ++did;
      t = ticket_.load(std::memory_order_relaxed);
    }
    return did;
  }
  void worker() {
    uint64_t seen = 0;
    for (;;) {
      uint32_t g;
      int n;
      const std::function<void(int)>* fn;
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return gen_ != seen; });
        seen = gen_;
        if (stop_) return;
        if (!fn_) continue;
        g = (uint32_t)gen_;
        n = ntask_;
        fn = fn_;
      }
      const int did = drain(g, n, *fn);
      if (did) {
        std::lock_guard<std::mutex> lk(mu_);
        done_ += did;
        if (done_ == ntask_) done_cv_.notify_all();
      }
    }
  }
  int n_;
  std::vector<std::thread> th_;
  std::mutex mu_;
  std::condition_variable cv_, done_cv_;
  const std::function<void(int)>* fn_ = nullptr;
  std::atomic<uint64_t> ticket_{0};
  int ntask_ = 0, done_ = 0;
  uint64_t gen_ = 0;
  bool stop_ = false;
};

}  // namespace host
}  // namespace vla
