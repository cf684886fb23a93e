// A small persistent pool of host threads for the library's host-side steps
// (hyperparameter search, forest training).  Work is cut into a fixed number
// of chunks that does not depend on the thread count, and callers reduce the
// chunks' partial results in chunk order, so results are identical whatever
// the number of threads.
//
// A likelihood evaluation is a few dozen short parallel steps, so the cost of
// handing out a step matters.  Each step is a job object shared by reference
// count: threads claim its chunks from an atomic counter and count finished
// chunks atomically, so no lock is taken on the way.  Idle workers and the
// waiting caller spin for a bounded time before they sleep on a condition
// variable; the mutex serves only that sleeping and waking.  A worker that
// arrives after the last chunk was claimed finds the counter exhausted and
// never calls the job's function, which may then no longer exist.  Up to
// kSlots callers (say, the hyperparameter searches of several objectives) may
// run jobs at the same time; idle threads take chunks from any of them.  A
// caller may cap the number of workers that join its jobs (PoolHelpers), to
// leave cores to other threads of its own; the results do not change.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdlib>
#include <exception>
#include <functional>
#include <memory>
#include <mutex>
#include <thread>
#include <vector>

#include "internal.h"

namespace scoot {

extern thread_local int t_max_helpers;  // this thread's cap on the workers that join its jobs

namespace {

struct Job {
  const std::function<void(int)>* fn;
  int n;
  int max_helpers = -1;  // workers that may join, besides the caller (-1: any)
  std::atomic<int> next{0}, done{0}, helpers{0};
  std::mutex err_mu;
  std::exception_ptr error;
};

// Polls cond for up to 200 us; the caller blocks afterwards if it is still false.
template <typename F>
void spin_until(F&& cond) {
  constexpr auto kSpin = std::chrono::microseconds(200);
  const auto t0 = std::chrono::steady_clock::now();
  for (int k = 0; !cond(); ++k)
    if ((k & 255) == 255 && std::chrono::steady_clock::now() - t0 > kSpin) return;
}

class Pool {
 public:
  Pool() {
    int want = 0;
    if (const char* e = std::getenv("SCOOT_HOST_THREADS")) want = std::atoi(e);
    if (want <= 0) want = std::min(16, (int)std::max(1u, std::thread::hardware_concurrency()));
    for (int t = 1; t < want; ++t) workers_.emplace_back([this] { loop(); });
  }
  ~Pool() {
    stop_.store(true);
    { std::lock_guard<std::mutex> lk(mu_); }
    cv_.notify_all();
    for (auto& w : workers_) w.join();
  }

  int threads() const { return (int)workers_.size() + 1; }

  void run(int n_chunks, const std::function<void(int)>& fn) {
    if (n_chunks <= 0) return;
    if (workers_.empty() || n_chunks == 1) {
      for (int c = 0; c < n_chunks; ++c) fn(c);
      return;
    }
    auto job = std::make_shared<Job>();
    job->fn = &fn;
    job->n = n_chunks;
    job->max_helpers = t_max_helpers;
    int slot = -1;
    {
      std::unique_lock<std::mutex> lk(slots_mu_);
      slot_free_.wait(lk, [&] {
        for (int k = 0; k < kSlots; ++k)
          if (!busy_[k]) return true;
        return false;
      });
      for (int k = 0; k < kSlots && slot < 0; ++k)
        if (!busy_[k]) slot = k;
      busy_[slot] = true;
    }
    std::atomic_store(&slots_[slot], job);
    gen_.fetch_add(1);
    if (sleepers_.load() > 0) {
      { std::lock_guard<std::mutex> lk(mu_); }  // a worker may be between its check and its wait
      cv_.notify_all();
    }
    work(*job);  // the calling thread takes part
    auto finished = [&] { return job->done.load(std::memory_order_acquire) == n_chunks; };
    spin_until(finished);
    if (!finished()) {
      std::unique_lock<std::mutex> lk(mu_);
      cv_done_.wait(lk, finished);
    }
    std::atomic_store(&slots_[slot], std::shared_ptr<Job>());
    {
      std::lock_guard<std::mutex> lk(slots_mu_);
      busy_[slot] = false;
    }
    slot_free_.notify_one();
    if (job->error) std::rethrow_exception(job->error);  // a chunk threw: report it to the caller
  }

 private:
  // Claims chunks of job until none is left; whether it ran any.
  bool work(Job& job) {
    bool ran = false;
    for (int c; (c = job.next.fetch_add(1)) < job.n; ran = true) {
      try {
        (*job.fn)(c);
      } catch (...) {
        std::lock_guard<std::mutex> lk(job.err_mu);
        if (!job.error) job.error = std::current_exception();
      }
      if (job.done.fetch_add(1, std::memory_order_acq_rel) + 1 == job.n) {
        { std::lock_guard<std::mutex> lk(mu_); }  // the caller may be between its check and its wait
        cv_done_.notify_all();
      }
    }
    return ran;
  }
  void loop() {
    unsigned long seen = 0;
    auto wake = [&] { return gen_.load() != seen || stop_.load(); };
    for (;;) {
      spin_until(wake);
      if (!wake()) {
        std::unique_lock<std::mutex> lk(mu_);
        sleepers_.fetch_add(1);
        cv_.wait(lk, wake);
        sleepers_.fetch_sub(1);
      }
      if (stop_.load()) return;
      // every slot until a whole round finds nothing to do; a job published
      // meanwhile moves gen_ past seen, so it is not missed
      seen = gen_.load();
      for (bool any = true; any;) {
        any = false;
        for (int k = 0; k < kSlots; ++k) {
          std::shared_ptr<Job> job = std::atomic_load(&slots_[k]);
          if (job && (job->max_helpers < 0 || job->helpers.fetch_add(1) < job->max_helpers) && work(*job))
            any = true;
        }
      }
    }
  }

  static constexpr int kSlots = 4;
  std::vector<std::thread> workers_;
  std::mutex mu_, slots_mu_;
  std::condition_variable cv_, cv_done_, slot_free_;
  std::shared_ptr<Job> slots_[kSlots];  // read and written with std::atomic_load / std::atomic_store
  bool busy_[kSlots] = {};              // under slots_mu_
  std::atomic<unsigned long> gen_{0};
  std::atomic<int> sleepers_{0};
  std::atomic<bool> stop_{false};
};

Pool& pool() {
  static Pool p;
  return p;
}

}  // namespace

thread_local int t_max_helpers = -1;

void parallel_chunks(int n_chunks, const std::function<void(int)>& fn) { pool().run(n_chunks, fn); }

int pool_threads() { return pool().threads(); }

PoolHelpers::PoolHelpers(int n) : prev_(t_max_helpers) { t_max_helpers = n < 0 ? -1 : n; }
PoolHelpers::~PoolHelpers() { t_max_helpers = prev_; }

}  // namespace scoot
