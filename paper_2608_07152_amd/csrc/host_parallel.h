// Small host thread helpers shared by the runtime and the fusion.
#pragma once
#include <algorithm>
#include <atomic>
#include <cstdint>
#include <thread>
#include <vector>

namespace eahr {

inline int host_threads() {
    unsigned n = std::thread::hardware_concurrency();
    if (n == 0) n = 1;
    return static_cast<int>(std::min(n, 16u));
}

// f(i) for i in [0, n) on up to `threads` threads (the caller is one of them).
template <typename F>
void parallel_for(int64_t n, int threads, F&& f) {
    if (n <= 0) return;
    if (threads <= 1 || n == 1) {
        for (int64_t i = 0; i < n; ++i) f(i);
        return;
    }
    std::atomic<int64_t> next{0};
    auto work = [&]() {
        for (int64_t i = next.fetch_add(1); i < n; i = next.fetch_add(1)) f(i);
    };
    const int extra = static_cast<int>(std::min<int64_t>(threads, n)) - 1;
    std::vector<std::thread> pool;
    pool.reserve(extra);
    for (int t = 0; t < extra; ++t) pool.emplace_back(work);
    work();
    for (auto& t : pool) t.join();
}

}  // namespace eahr
