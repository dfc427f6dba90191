// Small host thread helpers shared by the runtime and the fusion.
#pragma once
#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace eahr {

inline int host_threads() {
    unsigned n = std::thread::hardware_concurrency();
    if (n == 0) n = 1;
    return static_cast<int>(std::min(n, 16u));
}

// Persistent worker threads for parallel_for: one job at a time; a caller
// that finds the pool busy (another thread's job) is told so and uses its
// own threads instead.
class WorkerPool {
public:
    static WorkerPool& get() {
        static WorkerPool pool(host_threads() - 1);
        return pool;
    }
    // Runs work() on the caller and up to `extra` workers; false when busy.
    bool run(int extra, const std::function<void()>& work) {
        bool idle = false;
        if (!busy_.compare_exchange_strong(idle, true, std::memory_order_acquire)) return false;
        extra = std::max(0, std::min<int>(extra, static_cast<int>(workers_.size())));
        {
            std::lock_guard<std::mutex> lk(mu_);
            fn_ = &work;
            want_ = extra;
            pending_ = extra;
            ++gen_;
        }
        if (extra > 0) cv_.notify_all();
        work();
        {
            std::unique_lock<std::mutex> lk(mu_);
            done_.wait(lk, [&] { return pending_ == 0; });
            fn_ = nullptr;
        }
        busy_.store(false, std::memory_order_release);
        return true;
    }
    ~WorkerPool() {
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
            ++gen_;
        }
        cv_.notify_all();
        for (auto& t : workers_) t.join();
    }

private:
    explicit WorkerPool(int n) {
        for (int i = 0; i < n; ++i) workers_.emplace_back([this, i] { loop(i); });
    }
    void loop(int id) {
        uint64_t seen = 0;
        for (;;) {
            const std::function<void()>* f = nullptr;
            {
                std::unique_lock<std::mutex> lk(mu_);
                cv_.wait(lk, [&] { return stop_ || gen_ != seen; });
                if (stop_) return;
                seen = gen_;
                if (id >= want_) continue;   // not needed for this job
                f = fn_;
            }
            (*f)();
            std::lock_guard<std::mutex> lk(mu_);
            if (--pending_ == 0) done_.notify_one();
        }
    }
    std::atomic<bool> busy_{false};         // a job is running (nested calls see it too)
    std::mutex mu_;
    std::condition_variable cv_, done_;
    std::vector<std::thread> workers_;
    const std::function<void()>* fn_ = nullptr;
    uint64_t gen_ = 0;
    int want_ = 0, pending_ = 0;
    bool stop_ = false;
};

// f(i) for i in [0, n) on up to `threads` threads (the caller is one of them).
template <typename F>
void parallel_for(int64_t n, int threads, F&& f) {
    if (n <= 0) return;
    if (threads <= 1 || n == 1) {
        for (int64_t i = 0; i < n; ++i) f(i);
        return;
    }
    std::atomic<int64_t> next{0};
    const std::function<void()> work = [&]() {
        for (int64_t i = next.fetch_add(1); i < n; i = next.fetch_add(1)) f(i);
    };
    const int extra = static_cast<int>(std::min<int64_t>(threads, n)) - 1;
    if (WorkerPool::get().run(extra, work)) return;
    std::vector<std::thread> pool;
    pool.reserve(extra);
    for (int t = 0; t < extra; ++t) pool.emplace_back(work);
    work();
    for (auto& t : pool) t.join();
}

}  // namespace eahr
