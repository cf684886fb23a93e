// A small persistent pool of host threads for the library's host-side steps
// (hyperparameter search, forest training).  Work is cut into a fixed number
// of chunks that does not depend on the thread count, and callers reduce the
// chunks' partial results in chunk order, so results are identical whatever
// the number of threads.
//
// A likelihood evaluation is a dozen short parallel steps, so waking the
// workers dominates if they sleep between steps (measured: 23 us per empty
// step with 8 threads).  Idle workers and a waiting caller therefore spin on
// atomic mirrors of the job state for a bounded time before they block on the
// condition variables; the state itself still changes only under the mutex.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdlib>
#include <exception>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include "internal.h"

namespace scoot {

namespace {

class Pool {
 public:
  Pool() {
    int want = 0;
    if (const char* e = std::getenv("SCOOT_HOST_THREADS")) want = std::atoi(e);
    if (want <= 0) want = std::min(16, (int)std::max(1u, std::thread::hardware_concurrency()));
    for (int t = 1; t < want; ++t) workers_.emplace_back([this] { loop(); });
  }
  ~Pool() {
    {
      std::lock_guard<std::mutex> lk(mu_);
      stop_ = true;
      stop_seen_.store(true);
    }
    cv_.notify_all();
    for (auto& w : workers_) w.join();
  }

  void run(int n_chunks, const std::function<void(int)>& fn) {
    if (n_chunks <= 0) return;
    if (workers_.empty() || n_chunks == 1) {
      for (int c = 0; c < n_chunks; ++c) fn(c);
      return;
    }
    std::lock_guard<std::mutex> one_job(job_mu_);  // one job at a time
    {
      // The job's fields change only while no thread is inside work().
      std::unique_lock<std::mutex> lk(mu_);
      cv_done_.wait(lk, [&] { return active_ == 0; });
      fn_ = &fn;
      n_ = n_chunks;
      next_.store(0);
      done_ = 0;
      ++active_;  // the calling thread takes part
      active_seen_.store(active_, std::memory_order_relaxed);
      gen_.fetch_add(1, std::memory_order_release);
    }
    cv_.notify_all();
    work();
    spin_until([&] { return active_seen_.load(std::memory_order_acquire) == 0; });
    std::unique_lock<std::mutex> lk(mu_);
    cv_done_.wait(lk, [&] { return done_ == n_ && active_ == 0; });
    fn_ = nullptr;
    if (error_) {  // a chunk threw: report it to the caller
      std::exception_ptr e = error_;
      error_ = nullptr;
      std::rethrow_exception(e);
    }
  }

 private:
  // Entered with active_ counting this thread; claims chunks until none is
  // left, then reports them and leaves.
  void work() {
    int ran = 0;
    std::exception_ptr err;
    for (int c; (c = next_.fetch_add(1)) < n_;) {
      try {
        (*fn_)(c);
      } catch (...) {
        if (!err) err = std::current_exception();
      }
      ++ran;
    }
    std::lock_guard<std::mutex> lk(mu_);
    if (err && !error_) error_ = err;
    done_ += ran;
    --active_;
    active_seen_.store(active_, std::memory_order_release);
    cv_done_.notify_all();
  }
  void loop() {
    unsigned long seen = 0;
    for (;;) {
      spin_until([&] { return gen_.load(std::memory_order_acquire) != seen || stop_seen_.load(); });
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return stop_ || gen_.load() != seen; });
        if (stop_) return;
        seen = gen_.load();
        ++active_;
        active_seen_.store(active_, std::memory_order_relaxed);
      }
      work();
    }
  }
  // Polls cond for up to kSpin before the caller falls back to blocking.
  template <typename F>
  static void spin_until(F&& cond) {
    constexpr auto kSpin = std::chrono::microseconds(200);
    const auto t0 = std::chrono::steady_clock::now();
    for (int k = 0; !cond(); ++k)
      if ((k & 255) == 255 && std::chrono::steady_clock::now() - t0 > kSpin) return;
  }

  std::vector<std::thread> workers_;
  std::mutex mu_, job_mu_;
  std::condition_variable cv_, cv_done_;
  const std::function<void(int)>* fn_ = nullptr;
  std::atomic<int> next_{0};
  int n_ = 0, done_ = 0, active_ = 0;
  std::atomic<unsigned long> gen_{0};
  bool stop_ = false;
  // lock-free mirrors of active_ and stop_ for the spinning waits
  std::atomic<int> active_seen_{0};
  std::atomic<bool> stop_seen_{false};
  std::exception_ptr error_;
};

Pool& pool() {
  static Pool p;
  return p;
}

}  // namespace

void parallel_chunks(int n_chunks, const std::function<void(int)>& fn) { pool().run(n_chunks, fn); }

}  // namespace scoot
