// Small host thread helpers shared by the runtime and the fusion.
#pragma once
#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <functional>
#include <memory>
#include <mutex>
#include <thread>
#include <utility>
#include <vector>

namespace eahr {

inline int host_threads() {
    unsigned n = std::thread::hardware_concurrency();
    if (n == 0) n = 1;
    return static_cast<int>(std::min(n, 16u));
}

// Persistent worker threads shared by every parallel_for of the process.
// A call posts a job (items [0, n), at most `extra` helpers) and works on it
// itself; idle workers join open jobs.  Calls may run concurrently and may
// nest (a job's item may post a job): a caller only ever waits for items
// that are already running, so every wait ends.
class WorkerPool {
public:
    static WorkerPool& get() {
        static WorkerPool pool(host_threads() - 1);
        return pool;
    }

    void run(int64_t n, int extra, const std::function<void(int64_t)>& f) {
        Job job;
        job.f = &f;
        job.n = n;
        job.helpers = std::max(0, extra);
        if (job.helpers > 0 && !workers_.empty()) {
            {
                std::lock_guard<std::mutex> lk(mu_);
                jobs_.push_back(&job);
            }
            cv_.notify_all();
        }
        work_on(job);
        {
            // no new helper may join once the job is withdrawn
            std::lock_guard<std::mutex> lk(mu_);
            jobs_.erase(std::remove(jobs_.begin(), jobs_.end(), &job), jobs_.end());
        }
        std::unique_lock<std::mutex> lk(job.mu);
        job.cv.wait(lk, [&] { return job.active == 0; });
    }

    ~WorkerPool() {
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
        }
        cv_.notify_all();
        for (auto& t : workers_) t.join();
    }

private:
    struct Job {
        const std::function<void(int64_t)>* f = nullptr;
        int64_t n = 0;
        int helpers = 0;                    // helpers still allowed to join
        std::atomic<int64_t> next{0};
        std::mutex mu;
        std::condition_variable cv;
        int active = 0;                     // helpers inside work_on
    };

    explicit WorkerPool(int n) {
        for (int i = 0; i < n; ++i) workers_.emplace_back([this] { loop(); });
    }

    static void work_on(Job& job) {
        for (int64_t i = job.next.fetch_add(1); i < job.n; i = job.next.fetch_add(1)) (*job.f)(i);
    }

    void loop() {
        for (;;) {
            Job* job = nullptr;
            {
                std::unique_lock<std::mutex> lk(mu_);
                // the job is picked inside the wait: items are taken without
                // the pool lock, so a second look could find none left
                cv_.wait(lk, [&] {
                    if (stop_) return true;
                    for (Job* j : jobs_)
                        if (j->helpers > 0 && j->next.load(std::memory_order_relaxed) < j->n) {
                            job = j;
                            return true;
                        }
                    return false;
                });
                if (stop_) return;
                --job->helpers;
                std::lock_guard<std::mutex> jl(job->mu);   // registered before the pool lock is released
                ++job->active;
            }
            work_on(*job);
            std::lock_guard<std::mutex> jl(job->mu);
            if (--job->active == 0) job->cv.notify_all();
        }
    }

    std::mutex mu_;
    std::condition_variable cv_;
    std::vector<Job*> jobs_;
    std::vector<std::thread> workers_;
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
    const std::function<void(int64_t)> work = [&](int64_t i) { f(i); };
    const int extra = static_cast<int>(std::min<int64_t>(threads, n)) - 1;
    WorkerPool::get().run(n, extra, work);
}

// One long-lived thread that runs one job at a time for its owner, started
// on first use: the owner posts a job, goes on with its own work and waits
// for the job later (cheaper than a thread per job when jobs are short).
class Helper {
public:
    Helper() = default;
    Helper(const Helper&) = delete;
    Helper& operator=(const Helper&) = delete;
    ~Helper() {
        {
            std::lock_guard<std::mutex> lk(mu_);
            stop_ = true;
        }
        cv_.notify_all();
        if (t_.joinable()) t_.join();
    }
    // Starts f; the previous job must have been waited for.
    void post(std::function<void()> f) {
        {
            std::lock_guard<std::mutex> lk(mu_);
            if (!t_.joinable()) t_ = std::thread([this] { loop(); });
            job_ = std::move(f);
            state_ = 1;
        }
        cv_.notify_all();
    }
    // Waits for the posted job to finish (returns at once if none is).
    void wait() {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return state_ != 1 && state_ != 2; });
        state_ = 0;
    }

private:
    void loop() {
        std::unique_lock<std::mutex> lk(mu_);
        for (;;) {
            cv_.wait(lk, [&] { return state_ == 1 || stop_; });
            if (stop_) return;
            state_ = 2;
            std::function<void()> f = std::move(job_);
            lk.unlock();
            f();
            lk.lock();
            state_ = 3;
            cv_.notify_all();
        }
    }
    std::mutex mu_;
    std::condition_variable cv_;
    std::thread t_;
    std::function<void()> job_;
    int state_ = 0;   // 0 idle, 1 posted, 2 running, 3 done
    bool stop_ = false;
};

// Allocator that leaves new elements of a vector uninitialised on resize
// (for buffers written right after, in parallel when long).
template <typename T>
struct NoInit : std::allocator<T> {
    template <typename U>
    struct rebind {
        using other = NoInit<U>;
    };
    NoInit() = default;
    template <typename U>
    NoInit(const NoInit<U>&) noexcept {}
    template <typename U>
    void construct(U* p) noexcept {
        ::new (static_cast<void*>(p)) U;
    }
    template <typename U, typename... A>
    void construct(U* p, A&&... a) {
        ::new (static_cast<void*>(p)) U(std::forward<A>(a)...);
    }
};

// f(i, lo, hi) over [0, n[i]) of every item i, cut into pieces of at most
// `piece` elements that run on up to `threads` threads: a few long items
// use every thread, many short ones one each.
template <typename F>
void parallel_pieces(const std::vector<int64_t>& n, int64_t piece, int threads, F&& f) {
    struct Piece {
        int64_t i, lo, hi;
    };
    std::vector<Piece> ps;
    for (int64_t i = 0; i < static_cast<int64_t>(n.size()); ++i)
        for (int64_t lo = 0; lo < n[i]; lo += piece) ps.push_back(Piece{i, lo, std::min(n[i], lo + piece)});
    parallel_for(static_cast<int64_t>(ps.size()), threads, [&](int64_t k) { f(ps[k].i, ps[k].lo, ps[k].hi); });
}

}  // namespace eahr
