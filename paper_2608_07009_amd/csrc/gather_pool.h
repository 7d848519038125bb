// Host worker threads of the staged fetch path (HISPARSE_FETCH_STAGED): the records of a miss
// plan are gathered from the pinned host pool into a pinned staging buffer by all threads at
// once, ahead of one host-to-device copy.
#pragma once

#include <sched.h>

#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace hisparse {

class GatherPool {
 public:
  // The process's cores (its CPU affinity), at most `cap`; the calling thread is one of them.
  static int host_threads(int cap) {
    cpu_set_t set;
    int n = 1;
    if (sched_getaffinity(0, sizeof(set), &set) == 0) n = CPU_COUNT(&set);
    return std::max(1, std::min(n, cap));
  }

  explicit GatherPool(int threads) {
    for (int i = 1; i < threads; ++i) workers_.emplace_back([this] { loop(); });
  }
  ~GatherPool() {
    {
      std::lock_guard<std::mutex> lock(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    for (auto& t : workers_) t.join();
  }
  GatherPool(const GatherPool&) = delete;
  GatherPool& operator=(const GatherPool&) = delete;

  int threads() const { return (int)workers_.size() + 1; }

  // fn(begin, end) over [0, n) in pieces of `grain` (begin a multiple of grain), handed out in
  // increasing order; on every thread (run), or on the worker threads only while the caller
  // does something else (start ... wait, with at least one worker). fn must outlive the job.
  void run(int64_t n, int64_t grain, const std::function<void(int64_t, int64_t)>& fn) {
    if (!start(n, grain, fn)) return;
    work();
    wait();
  }
  bool start(int64_t n, int64_t grain, const std::function<void(int64_t, int64_t)>& fn) {
    if (n <= 0) return false;
    {
      std::lock_guard<std::mutex> lock(mu_);
      fn_ = &fn;
      n_ = n;
      grain_ = std::max<int64_t>(1, grain);
      next_.store(0);
      busy_ = (int)workers_.size();
      ++gen_;
    }
    cv_.notify_all();
    return true;
  }
  void wait() {
    std::unique_lock<std::mutex> lock(mu_);
    done_cv_.wait(lock, [this] { return busy_ == 0; });
    fn_ = nullptr;
  }

 private:
  void work() {
    for (;;) {
      const int64_t b = next_.fetch_add(grain_);
      if (b >= n_) break;
      (*fn_)(b, std::min(n_, b + grain_));
    }
  }
  void loop() {
    uint64_t seen = 0;
    for (;;) {
      {
        std::unique_lock<std::mutex> lock(mu_);
        cv_.wait(lock, [&] { return stop_ || gen_ != seen; });
        if (stop_) return;
        seen = gen_;
      }
      work();
      {
        std::lock_guard<std::mutex> lock(mu_);
        --busy_;
      }
      done_cv_.notify_one();
    }
  }

  std::vector<std::thread> workers_;
  std::mutex mu_;
  std::condition_variable cv_, done_cv_;
  bool stop_ = false;
  uint64_t gen_ = 0;
  int busy_ = 0;
  std::atomic<int64_t> next_{0};
  int64_t n_ = 0, grain_ = 1;
  const std::function<void(int64_t, int64_t)>* fn_ = nullptr;
};

}  // namespace hisparse
