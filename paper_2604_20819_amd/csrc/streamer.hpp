// Host-side pieces of the task streamer shared by the forward and backward
// drivers (internal): host worker threads, the in-order host merge queue, and
// the split of a task's staging into host copies and reuse of the previously
// staged task's rows.
#pragma once

#include <algorithm>
#include <condition_variable>
#include <deque>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include "plan.hpp"

namespace cqsa {

inline int host_threads() {
  unsigned n = std::thread::hardware_concurrency();
  if (n == 0) n = 4;
  return int(std::min(16u, n));
}

// Runs f(lo, hi) over [0, n) split across up to host_threads() threads.
template <typename F>
void parallel_rows(int64_t n, F f) {
  const int nt = int(std::min<int64_t>(host_threads(), std::max<int64_t>(1, n / 256)));
  if (nt <= 1) {
    f(int64_t(0), n);
    return;
  }
  std::vector<std::thread> th;
  for (int i = 0; i < nt; ++i) {
    const int64_t a = n * i / nt, b = n * (i + 1) / nt;
    th.emplace_back([=] { f(a, b); });
  }
  for (auto& t : th) t.join();
}

// One consumer thread that runs host merges strictly in submission order
// (merges of different tasks touch shared rows).
class HostMerger {
 public:
  ~HostMerger() { finish(); }
  // Queues a job; returns its sequence number.
  int64_t push(std::function<bool()> job) {
    std::unique_lock<std::mutex> g(mu_);
    if (!th_.joinable()) th_ = std::thread([this] { run(); });
    q_.push_back(std::move(job));
    cv_.notify_all();
    return pushed_++;
  }
  // Blocks until job `id` (and all before it) finished; false on failure.
  bool wait_done(int64_t id) {
    std::unique_lock<std::mutex> g(mu_);
    cv_.wait(g, [&] { return done_ > id || !ok_; });
    return ok_;
  }
  bool finish() {
    {
      std::unique_lock<std::mutex> g(mu_);
      stop_ = true;
      cv_.notify_all();
    }
    if (th_.joinable()) th_.join();
    return ok_;
  }

 private:
  void run() {
    for (;;) {
      std::function<bool()> job;
      {
        std::unique_lock<std::mutex> g(mu_);
        cv_.wait(g, [&] { return !q_.empty() || stop_; });
        if (q_.empty()) return;
        job = std::move(q_.front());
        q_.pop_front();
      }
      const bool ok = ok_ && job();
      std::unique_lock<std::mutex> g(mu_);
      if (!ok) ok_ = false;
      ++done_;
      cv_.notify_all();
    }
  }
  std::mutex mu_;
  std::condition_variable cv_;
  std::deque<std::function<bool()>> q_;
  std::thread th_;
  int64_t pushed_ = 0, done_ = 0;
  bool stop_ = false, ok_ = true;
};

// One piece of a task's staging: local rows [dst, dst + length) of the task
// come either from the host tensors at global row `src`, or, when the task
// staged just before holds the same tokens, from its staged rows at its local
// row `src` (device to device).
struct StagePiece {
  int64_t dst, src, length;
  bool reuse;
};

// Splits `cur`'s runs against the runs of the previously staged task `prev`
// (both ascending in global order): overlapping tokens are reused, the rest
// comes from the host.  Consecutive tasks in quorum order share chunks (at
// depth 1 with I = (0, 1, 3), task q + 1 holds chunk q + 1 of task q).
std::vector<StagePiece> stage_pieces(const Task& cur, const Task* prev);

}  // namespace cqsa
