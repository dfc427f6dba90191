// Stress test of the host worker pool: several threads post jobs of random
// sizes and thread counts at once, and items post nested jobs.  Every item
// must run exactly once and every call must return.  The same work also runs
// as jobs of long-lived helper threads (posted, overlapped with the poster's
// own work, waited for), as the fusion runs its sparse channel.
#include <atomic>
#include <cstdio>
#include <random>
#include <thread>
#include <vector>

#include "host_parallel.h"

static std::atomic<long> g_items{0};
static long g_expected_check = 0;

static long work(int depth, unsigned seed) {
    std::mt19937 rng(seed);
    const int n = 1 + static_cast<int>(rng() % 50);
    const int threads = 1 + static_cast<int>(rng() % 16);
    std::vector<std::atomic<int>> hits(n);
    for (auto& h : hits) h = 0;
    std::atomic<long> nested{0};
    eahr::parallel_for(n, threads, [&](int64_t i) {
        hits[i] += 1;
        g_items += 1;
        if (depth < 2 && i % 7 == 0) nested += work(depth + 1, seed * 31u + static_cast<unsigned>(i));
    });
    for (auto& h : hits)
        if (h != 1) {
            std::printf("item ran %d times\n", h.load());
            std::exit(1);
        }
    return n + nested;
}

int main(int argc, char** argv) {
    const int reps = argc > 1 ? std::atoi(argv[1]) : 100;
    long want = 0;
    for (int rep = 0; rep < reps; ++rep) {
        std::vector<std::thread> ts;
        std::vector<long> got(4);
        for (int t = 0; t < 4; ++t) ts.emplace_back([rep, t, &got] { got[t] = work(0, rep * 10u + t); });
        for (auto& t : ts) t.join();
        for (long g : got) want += g;
    }
    // helpers: each of 4 threads owns one and posts a job per round
    {
        std::vector<std::thread> ts;
        std::vector<long> got(4, 0);
        for (int t = 0; t < 4; ++t)
            ts.emplace_back([reps, t, &got] {
                eahr::Helper h;
                for (int rep = 0; rep < reps; ++rep) {
                    long side = 0;
                    h.post([&] { side = work(0, 7000u + rep * 10u + t); });
                    const long mine = work(0, 9000u + rep * 10u + t);
                    h.wait();
                    got[t] += side + mine;
                }
                h.wait();   // nothing posted: returns at once
            });
        for (auto& t : ts) t.join();
        for (long g : got) want += g;
    }
    if (want != g_items) {
        std::printf("items %ld, expected %ld\n", g_items.load(), want);
        return 1;
    }
    (void)g_expected_check;
    std::printf("ok %ld\n", want);
    return 0;
}
