// eahr_topk and eahr_fuse_lists: the depth-round driver of exact adaptive
// weighted-RRF fusion (Sec. 2.1, 2.2).  Every Open list with positive weight
// advances to cumulative depth depth0 * growth^j; after each round the
// positions are certified (fusion.h).  Exhausted lists contribute their
// complete rankings, so a request either resolves early or at exhaustion.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <tuple>
#include <vector>

#include "common.h"
#include "eahr.h"
#include "fusion.h"
#include "host_parallel.h"
#include "pbm_internal.h"
#include "pvs_internal.h"
#include "schedule.h"

namespace {

using ::eahr::Fusion;
using ::eahr::Params;

int check_params(const eahr_params& ep) {
    if (ep.K < 0 || ep.depth0 < 1 || ep.growth < 2 || ep.k_rrf < 1 || ep.k_rrf > (1 << 20) ||
        ep.w_dense < 0 || ep.w_dense > 1024 || ep.w_sparse < 0 || ep.w_sparse > 1024 ||
        (ep.dense_generator != EAHR_GEN_INTERVALS && ep.dense_generator != EAHR_GEN_FULL_SCAN) ||
        (ep.schedule != EAHR_SCHED_DOUBLING && ep.schedule != EAHR_SCHED_FROZEN) ||
        (ep.sparse_generator != EAHR_SPARSE_PBM && ep.sparse_generator != EAHR_SPARSE_COMPLETE &&
         ep.sparse_generator != EAHR_SPARSE_PBM_GPU))
        EAHR_FAIL(EAHR_E_INVALID, "eahr: parameters out of range");
    return EAHR_OK;
}

using ::eahr::host_threads;
using ::eahr::parallel_for;

// Dense work-ahead while a round's sparse channel runs: never past this depth
// per query, nor past this many ranks summed over the round's dense queries.
// A further level starts only while its estimated time (ranks it may certify
// times the measured time per certified rank of earlier work-ahead) fits in
// the sparse channel's estimated remaining time (elapsed time scaled by the
// share of its queries still to finish).
constexpr int64_t kFillMaxDepth = int64_t(1) << 17;
constexpr int64_t kFillBudget = int64_t(1) << 25;

// Rates measured by earlier calls on the same pair of indexes and sparse
// generator: time per posting of a first sparse round (which scores about
// all of its queries' postings), per host thread it could use (one per
// query, up to the pool's size; the GPU generator counts as one), and dense
// time per rank certified ahead.
// With both known, the first round certifies ahead in one scan, to the
// deepest depth level whose estimated time fits in kAheadSlack times the
// sparse channel's expected time, instead of in steps of one level (a scan
// each) while it runs.  Entries are a few bytes and live as long as the
// process; an index allocated where a freed one was starts from that one's
// rates, which only sizes work.
struct Rates {
    double sparse_ms_per_posting = 0.0;   // times the threads the round could use
    double dense_ms_per_rank = 0.0;
};
constexpr double kAheadSlack = 1.25;
// Sparse rounds shorter than this (as the previous one was) run inline.
constexpr double kInlineSparseMs = 0.1;
std::mutex g_rates_mu;
std::map<std::tuple<const void*, const void*, int32_t>, Rates> g_rates;

double ms_since(std::chrono::steady_clock::time_point t0) {
    return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
}

template <typename T>
struct RawBuf {   // uninitialised growable host buffer
    std::unique_ptr<T[]> p;
    size_t n = 0;
    T* get(size_t want) {
        if (want > n) {
            p.reset(new T[want]);
            n = want;
        }
        return p.get();
    }
};

// Per-call buffers of eahr_topk (fusion states, the rounds' dense and sparse
// ranks), kept between calls so that their memory is reused rather than
// faulted in again; concurrent calls each take their own.
struct TopkWork {
    ::eahr::Helper sparse;   // runs each round's sparse channel beside the dense one
    std::vector<Fusion> F;
    RawBuf<int64_t> dids;
    RawBuf<float> dscores;
    std::vector<std::vector<int64_t>> sids;
    std::vector<std::vector<float>> sscores;
};

std::mutex g_work_mu;
std::vector<std::unique_ptr<TopkWork>> g_work;

// eahr_set_rank_observer
std::mutex g_obs_mu;
eahr_rank_observer g_obs = nullptr;
void* g_obs_user = nullptr;

struct WorkLease {
    std::unique_ptr<TopkWork> w;
    WorkLease() {
        std::lock_guard<std::mutex> lk(g_work_mu);
        if (!g_work.empty()) {
            w = std::move(g_work.back());
            g_work.pop_back();
        }
        if (!w) w.reset(new TopkWork());
    }
    ~WorkLease() {
        std::lock_guard<std::mutex> lk(g_work_mu);
        if (g_work.size() < 4) g_work.push_back(std::move(w));
    }
};

}  // namespace

// The dense channel is either a pvs_state opened here on `dense` or, when
// `merged` is given, a caller-opened merged ranking (Segments / Shards).
static int topk_impl(const pvs_index* dense, int64_t epoch, pvs_merge* merged,
                     const pbm_index* sparse, const float* q_dense, int32_t q_ptr_kind,
                     const eahr_sparse_query* q_sparse, int32_t B, const eahr_params* params,
                     int64_t* out_ids, int32_t* out_count, int32_t* out_status,
                     eahr_query_stats* stats) {
    if (!params || B <= 0 || !out_ids || !out_count || !out_status)
        EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: bad arguments");
    const eahr_params& ep = *params;
    EAHR_TRY(check_params(ep));
    const bool use_dense = ep.w_dense > 0, use_sparse = ep.w_sparse > 0;
    if (use_dense && !merged && (!dense || !q_dense)) EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: dense channel missing");
    if (use_dense && merged && eahr_merge_batch(merged) != B)
        EAHR_FAIL(EAHR_E_INVALID, "eahr_topk_merged: the merge was opened for another batch size");
    if (use_sparse && (!sparse || !q_sparse)) EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: sparse channel missing");
    const Params P{ep.K, ep.k_rrf, {ep.w_dense, ep.w_sparse}};
    const auto t_call = std::chrono::steady_clock::now();
    const int threads = host_threads();
    eahr_rank_observer obs = nullptr;
    void* obs_user = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_obs_mu);
        obs = g_obs;
        obs_user = g_obs_user;
    }
    std::vector<int64_t> nobs[2];   // ranks passed to the observer per list and query
    nobs[0].assign(B, 0);
    nobs[1].assign(B, 0);
    auto observe = [&](int32_t b, int list, const int64_t* ids, const float* sc, int64_t n) {
        if (!obs || n <= 0) return;
        obs(obs_user, b, list, nobs[list][b], ids, sc, n);
        nobs[list][b] += n;
    };
    const bool prof = pvs_profile_on();
    double t_dense = 0, t_sparse = 0, t_fuse = 0;

    WorkLease lease;
    TopkWork& W = *lease.w;
    if (W.F.size() < static_cast<size_t>(B)) W.F.resize(B);
    for (int32_t b = 0; b < B; ++b) W.F[b].reset();
    Fusion* F = W.F.data();
    std::vector<int32_t> dstat(B, EAHR_LIST_EXHAUSTED), sstat(B, EAHR_LIST_EXHAUSTED);
    std::vector<int32_t> rounds(B, 0);
    std::vector<uint8_t> failed(B, 0);
    // Under the frozen scheduler appends stay small (at most a check's gap)
    // while lists grow deep, so deep queries switch the fusion to direct rank
    // arrays over the channels' id range (dense rows, sparse documents).
    // Depth doubling appends as many ranks as a list already holds, so its
    // merges into the id order cost O(depth) in all and the arrays (8 bytes
    // per id of the range) would cost more than they save.
    int64_t universe = 0;
    if (ep.schedule == EAHR_SCHED_FROZEN && !merged) {
        if (use_dense) {
            int64_t rows = 0;
            EAHR_TRY(pvs_info(dense, epoch, &rows, nullptr, nullptr));
            universe = rows;
        }
        if (use_sparse) universe = std::max<int64_t>(universe, sparse->n_docs);
    }
    for (int32_t b = 0; b < B; ++b) {
        F[b].P = &P;
        F[b].universe = universe;
        F[b].L[0].open = use_dense;
        F[b].L[1].open = use_sparse;
        if (use_dense) dstat[b] = EAHR_LIST_OPEN;
        if (use_sparse) sstat[b] = EAHR_LIST_OPEN;
        if (ep.K == 0) F[b].resolved = true;
    }
    struct Cleanup {
        pvs_state* st = nullptr;
        std::vector<pbm_state*> sp;
        pbm_gpu_state* gsp = nullptr;   // the batch's GPU sparse states
        ~Cleanup() {
            if (st) pvs_close(st);
            for (auto* s : sp)
                if (s) pbm_close(s);
            if (gsp) pbm_gpu_close(gsp);
        }
    } cl;
    const auto t_open = std::chrono::steady_clock::now();
    if (use_dense && !merged)
        EAHR_TRY(pvs_open_gen(dense, epoch, q_dense, B, q_ptr_kind, ep.dense_generator, &cl.st));
    const double open_dense_ms = ms_since(t_open);
    // sparse states are opened by the sparse workers, at a query's first
    // call; the queries are checked here
    if (use_sparse) {
        for (int32_t b = 0; b < B; ++b) EAHR_TRY(pbm_check_query(sparse, &q_sparse[b]));
        cl.sp.assign(B, nullptr);
    }
    if (::eahr::trace_on()) std::fprintf(stderr, "eahr open dense_ms=%.2f\n", open_dense_ms);
    RawBuf<int64_t>& dids = W.dids;
    RawBuf<float>& dscores = W.dscores;
    std::vector<int32_t> dcnt(B, 0), dsts(B);
    std::vector<uint8_t> dact(B, 0);
    if (W.sids.size() < static_cast<size_t>(B)) {
        W.sids.resize(B);
        W.sscores.resize(B);
    }
    auto& sids = W.sids;
    auto& sscores = W.sscores;
    std::vector<int32_t> scnt(B, 0), ssts(B, EAHR_LIST_OPEN);
    std::vector<uint8_t> sact(B, 0);
    std::vector<int> sparse_rc(B, EAHR_OK);
    // error messages are per thread: a sparse worker's first one is carried
    // back to the caller
    std::mutex sparse_err_mu;
    std::string sparse_err;
    auto note_sparse_error = [&](int rc) {
        if (rc == EAHR_OK) return;
        std::lock_guard<std::mutex> lk(sparse_err_mu);
        if (sparse_err.empty()) sparse_err = eahr_last_error();
    };
    // sparse work order: the queries with the most postings first, so that
    // the last ones a round waits for are short (their first call scores
    // about their postings)
    std::vector<int32_t> sorder(B);
    for (int32_t b = 0; b < B; ++b) sorder[b] = b;
    std::vector<int64_t> cost(B, 1);
    if (use_sparse) {
        for (int32_t b = 0; b < B; ++b)
            for (int32_t i = 0; i < q_sparse[b].n_terms; ++i) {
                const int32_t t = q_sparse[b].terms[i];
                if (t >= 0 && t < sparse->vocab) cost[b] += sparse->term_ptr[t + 1] - sparse->term_ptr[t];
            }
        std::stable_sort(sorder.begin(), sorder.end(), [&](int32_t a, int32_t c) { return cost[a] > cost[c]; });
    }
    // GPU sparse generator: one batched call serves every query that wants
    // ranks (want[b] > 0) into sids / sscores; the batch's states are opened
    // at the first call
    const bool gpu_sparse = use_sparse && ep.sparse_generator == EAHR_SPARSE_PBM_GPU;
    std::vector<int32_t> gwant(B, 0);
    std::vector<int64_t*> gids(B, nullptr);
    std::vector<float*> gsc(B, nullptr);
    auto gpu_sparse_next = [&](const std::vector<int64_t>& want) -> int {
        if (!cl.gsp) EAHR_TRY(pbm_gpu_open(sparse, q_sparse, B, &cl.gsp));
        for (int32_t b = 0; b < B; ++b) {
            gwant[b] = static_cast<int32_t>(std::min<int64_t>(std::max<int64_t>(want[b], 0), 1LL << 30));
            sids[b].resize(static_cast<size_t>(gwant[b]));
            sscores[b].resize(static_cast<size_t>(gwant[b]));
            gids[b] = sids[b].data();
            gsc[b] = sscores[b].data();
            if (gwant[b] == 0) scnt[b] = 0;
        }
        return pbm_gpu_next(cl.gsp, gwant.data(), gids.data(), gsc.data(), scnt.data(), ssts.data());
    };
    if (ep.schedule == EAHR_SCHED_FROZEN) {
        // Frozen scheduler: ranks are read ahead into per-query pending
        // buffers (dense batched, sparse per query), and every check appends
        // exactly the ranks the schedule has reached and certifies.
        const int64_t H = ::eahr::FrozenSchedule::kHorizon;
        std::vector<::eahr::FrozenSchedule> Sch(B);
        std::vector<std::vector<int64_t>> pend[2];
        std::vector<int64_t> head[2];
        std::vector<uint8_t> exh[2];
        for (int i = 0; i < 2; ++i) {
            pend[i].assign(B, {});
            head[i].assign(B, 0);
            exh[i].assign(B, 0);
        }
        auto live = [&](int32_t b) { return !F[b].resolved && !failed[b]; };
        auto have = [&](int i, int32_t b) { return static_cast<int64_t>(pend[i][b].size()) - head[i][b]; };
        for (;;) {
            bool any = false;
            for (int32_t b = 0; b < B; ++b) any |= live(b);
            if (!any) break;
            const auto t0 = std::chrono::steady_clock::now();
            if (use_dense) {
                int64_t m = 0;
                for (int32_t b = 0; b < B; ++b) {
                    dact[b] = live(b) && !exh[0][b] && have(0, b) < H;
                    if (dact[b]) m = std::max<int64_t>(m, 2 * H - have(0, b));
                }
                if (m > 0) {
                    int64_t* ids = dids.get(static_cast<size_t>(B) * m);
                    float* sc = dscores.get(static_cast<size_t>(B) * m);
                    EAHR_TRY(pvs_next(cl.st, static_cast<int32_t>(m), dact.data(), ids, sc, dcnt.data(),
                                      dsts.data()));
                    for (int32_t b = 0; b < B; ++b) {
                        if (!dact[b]) continue;
                        if (dsts[b] == EAHR_LIST_FAILED) {
                            failed[b] = 1;
                            dstat[b] = EAHR_LIST_FAILED;
                            continue;
                        }
                        const int64_t* p = ids + static_cast<size_t>(b) * m;
                        observe(b, 0, p, sc + static_cast<size_t>(b) * m, dcnt[b]);
                        pend[0][b].insert(pend[0][b].end(), p, p + dcnt[b]);
                        if (dsts[b] == EAHR_LIST_EXHAUSTED) exh[0][b] = 1;
                    }
                }
            }
            t_dense += ms_since(t0);
            const auto t1 = std::chrono::steady_clock::now();
            if (gpu_sparse) {
                std::vector<int64_t> want(B, 0);
                for (int32_t b = 0; b < B; ++b)
                    if (live(b) && !exh[1][b] && have(1, b) < H) want[b] = 2 * H - have(1, b);
                EAHR_TRY(gpu_sparse_next(want));
                for (int32_t b = 0; b < B; ++b) {
                    if (want[b] == 0) continue;
                    if (ssts[b] == EAHR_LIST_FAILED) {
                        failed[b] = 1;
                        sstat[b] = EAHR_LIST_FAILED;
                        continue;
                    }
                    observe(b, 1, sids[b].data(), sscores[b].data(), scnt[b]);
                    pend[1][b].insert(pend[1][b].end(), sids[b].begin(), sids[b].begin() + scnt[b]);
                    if (ssts[b] == EAHR_LIST_EXHAUSTED) exh[1][b] = 1;
                }
            } else if (use_sparse) {
                std::vector<uint8_t> sread(B, 0);
                parallel_for(B, threads, [&](int64_t b) {
                    if (!live(static_cast<int32_t>(b)) || exh[1][b] || have(1, b) >= H) return;
                    if (!cl.sp[b]) {
                        sparse_rc[b] = pbm_open_gen(sparse, &q_sparse[b], ep.sparse_generator, &cl.sp[b]);
                        if (sparse_rc[b] != EAHR_OK) {
                            note_sparse_error(sparse_rc[b]);
                            return;
                        }
                    }
                    const int64_t need = 2 * H - have(1, b);
                    sids[b].resize(static_cast<size_t>(need));
                    sscores[b].resize(static_cast<size_t>(need));
                    sparse_rc[b] = pbm_next(cl.sp[b], static_cast<int32_t>(need), sids[b].data(),
                                            sscores[b].data(), &scnt[b], &ssts[b]);
                    if (sparse_rc[b] != EAHR_OK) {
                        note_sparse_error(sparse_rc[b]);
                        return;
                    }
                    if (ssts[b] == EAHR_LIST_FAILED) {
                        failed[b] = 1;
                        sstat[b] = EAHR_LIST_FAILED;
                        return;
                    }
                    pend[1][b].insert(pend[1][b].end(), sids[b].begin(), sids[b].begin() + scnt[b]);
                    sread[b] = 1;
                    if (ssts[b] == EAHR_LIST_EXHAUSTED) exh[1][b] = 1;
                });
                for (int32_t b = 0; b < B; ++b)
                    if (sread[b]) observe(b, 1, sids[b].data(), sscores[b].data(), scnt[b]);
                for (int32_t b = 0; b < B; ++b)
                    if (sparse_rc[b] != EAHR_OK) {
                        ::eahr::set_error("%s", sparse_err.c_str());
                        return sparse_rc[b];
                    }
            }
            t_sparse += ms_since(t1);
            const auto t2 = std::chrono::steady_clock::now();
            parallel_for(B, threads, [&](int64_t bb) {
                const int32_t b = static_cast<int32_t>(bb);
                if (!live(b)) return;
                auto& S = Sch[b];
                const int64_t avail[2] = {S.d[0] + have(0, b), S.d[1] + have(1, b)};
                const bool done[2] = {exh[0][b] != 0, exh[1][b] != 0};
                const bool use[2] = {use_dense, use_sparse};
                S.advance(P, avail, done, use);
                for (int i = 0; i < 2; ++i) {
                    const int64_t n = S.d[i] - static_cast<int64_t>(F[b].L[i].size());
                    if (n > 0) {
                        F[b].append(i, pend[i][b].data() + head[i][b], n);
                        head[i][b] += n;
                    }
                    if (done[i] && S.d[i] == avail[i] && F[b].L[i].open) {
                        F[b].L[i].open = false;
                        (i == 0 ? dstat : sstat)[b] = EAHR_LIST_EXHAUSTED;
                    }
                    if (head[i][b] > (1 << 16) && 2 * head[i][b] > static_cast<int64_t>(pend[i][b].size())) {
                        pend[i][b].erase(pend[i][b].begin(), pend[i][b].begin() + head[i][b]);
                        head[i][b] = 0;
                    }
                }
                if (F[b].dup) {
                    failed[b] = 1;
                    return;
                }
                rounds[b] += 1;
                F[b].certify();
                // both lists complete and still unresolved: not rankings
                if (!F[b].resolved && !F[b].L[0].open && !F[b].L[1].open) failed[b] = 1;
            });
            t_fuse += ms_since(t2);
        }
    }
    int64_t depth = ep.depth0;
    double fill_ms = 0.0;            // measured cost of dense work-ahead
    int64_t fill_ranks = 0;
    const std::tuple<const void*, const void*, int32_t> rates_key{dense, sparse, ep.sparse_generator};
    Rates rates;
    {
        std::lock_guard<std::mutex> lk(g_rates_mu);
        const auto it = g_rates.find(rates_key);
        if (it != g_rates.end()) rates = it->second;
    }
    double first_sparse_ms = -1.0;   // the first round's sparse time, postings and threads
    int64_t first_sparse_cost = 0;
    int64_t first_sparse_par = 1;
    bool first_round = true;
    std::vector<uint8_t> retired(B, 0);
    double last_sparse_ms = -1.0;    // the previous round's sparse time
    for (bool doubling = ep.schedule == EAHR_SCHED_DOUBLING; doubling;) {
        bool any = false;
        for (int32_t b = 0; b < B; ++b) any |= !F[b].resolved && !failed[b];
        if (!any) break;
        // requests of this round: every Open list of an unresolved query to `depth`
        int64_t m = 0;
        for (int32_t b = 0; b < B; ++b) {
            const bool live = !F[b].resolved && !failed[b];
            dact[b] = live && use_dense && F[b].L[0].open &&
                      static_cast<int64_t>(F[b].L[0].size()) < depth;
            sact[b] = live && use_sparse && F[b].L[1].open &&
                      static_cast<int64_t>(F[b].L[1].size()) < depth;
            dcnt[b] = 0;
            scnt[b] = 0;
            if (dact[b]) m = std::max<int64_t>(m, depth - static_cast<int64_t>(F[b].L[0].size()));
        }
        if (m > (1LL << 30)) m = 1LL << 30;
        const auto t_round = std::chrono::steady_clock::now();
        double r_dense = 0, r_sparse = 0;
        // sparse channel on worker threads while the dense channel runs on the GPU
        bool sparse_running = false;
        struct WaitSparse {   // the job refers to this round's locals
            ::eahr::Helper& h;
            bool& running;
            ~WaitSparse() {
                if (running) h.wait();
            }
        } wait_sparse{W.sparse, sparse_running};
        std::atomic<bool> sparse_done{false};
        std::atomic<int64_t> sparse_cost_done{0};   // postings of the queries finished
        int64_t sparse_cost = 0, sparse_queries = 0;
        for (int32_t b = 0; b < B; ++b)
            if (sact[b]) {
                sparse_cost += cost[b];
                sparse_queries += 1;
            }
        // threads the round's sparse work can use (one per query)
        const int64_t sparse_par =
            gpu_sparse ? 1 : std::max<int64_t>(1, std::min<int64_t>(std::max(1, threads - 1), sparse_queries));
        const auto t_sparse0 = std::chrono::steady_clock::now();
        auto sparse_work = [&]() {
            const auto t0 = std::chrono::steady_clock::now();
            if (gpu_sparse) {
                std::vector<int64_t> want(B, 0);
                for (int32_t b = 0; b < B; ++b)
                    if (sact[b]) want[b] = depth - static_cast<int64_t>(F[b].L[1].size());
                const int rc = gpu_sparse_next(want);
                if (rc != EAHR_OK) {
                    note_sparse_error(rc);
                    for (int32_t b = 0; b < B; ++b)
                        if (sact[b]) sparse_rc[b] = rc;
                }
                sparse_cost_done.store(sparse_cost, std::memory_order_relaxed);
                r_sparse = ms_since(t0);
                t_sparse += r_sparse;
                sparse_done.store(true, std::memory_order_release);
                return;
            }
            parallel_for(B, std::max(1, threads - 1), [&](int64_t i) {
                const int32_t b = sorder[i];
                if (!sact[b]) return;
                if (!cl.sp[b]) {
                    sparse_rc[b] = pbm_open_gen(sparse, &q_sparse[b], ep.sparse_generator, &cl.sp[b]);
                    if (sparse_rc[b] != EAHR_OK) {
                        note_sparse_error(sparse_rc[b]);
                        sparse_cost_done.fetch_add(cost[b], std::memory_order_relaxed);
                        return;
                    }
                }
                const int64_t need = std::min<int64_t>(depth - static_cast<int64_t>(F[b].L[1].size()), 1LL << 30);
                sids[b].resize(static_cast<size_t>(need));
                sscores[b].resize(static_cast<size_t>(need));
                sparse_rc[b] = pbm_next(cl.sp[b], static_cast<int32_t>(need), sids[b].data(),
                                        sscores[b].data(), &scnt[b], &ssts[b]);
                note_sparse_error(sparse_rc[b]);
                sparse_cost_done.fetch_add(cost[b], std::memory_order_relaxed);
            });
            r_sparse = ms_since(t0);
            t_sparse += r_sparse;
            sparse_done.store(true, std::memory_order_release);
        };
        bool any_sparse = false;
        for (int32_t b = 0; b < B; ++b) any_sparse |= sact[b] != 0;
        // A short sparse round beside dense ranks that are already certified
        // runs on this thread after them: handing it to the helper thread and
        // back costs more than the overlap saves.
        const bool sparse_inline = any_sparse && !gpu_sparse && !merged && last_sparse_ms >= 0.0 &&
                                   last_sparse_ms < kInlineSparseMs &&
                                   (m == 0 || pvs_covered(cl.st, m, dact.data()));
        if (any_sparse && !sparse_inline) {
            W.sparse.post(sparse_work);
            sparse_running = true;
        }
        int dense_rc = EAHR_OK;
        if (m > 0) {
            const auto t0 = std::chrono::steady_clock::now();
            int64_t nd = 0;
            for (int32_t b = 0; b < B; ++b) nd += dact[b];
            const int64_t cap = std::min<int64_t>(kFillMaxDepth, kFillBudget / std::max<int64_t>(nd, 1));
            if (first_round && !merged && sparse_running && rates.sparse_ms_per_posting > 0.0 &&
                rates.dense_ms_per_rank > 0.0) {
                // certify ahead, in one scan, to the deepest level the sparse
                // channel's expected time pays for; worth a scan of its own
                // only beyond what a first scan certifies anyway
                const double expect = rates.sparse_ms_per_posting * static_cast<double>(sparse_cost) /
                                      static_cast<double>(sparse_par);
                const double per_level = rates.dense_ms_per_rank * static_cast<double>(nd);
                const int64_t first_scan = std::max(pvs::kSpecFloor, pvs::kSpecFloorBudget / std::max<int64_t>(nd, 1));
                int64_t ahead = 0;
                for (int64_t l = depth; l <= cap && per_level * static_cast<double>(l) <= kAheadSlack * expect;
                     l *= ep.growth)
                    ahead = l;
                if (ahead > std::max(depth * ep.growth, first_scan)) {
                    int64_t added = 0;
                    dense_rc = pvs_fill_exact(cl.st, ahead, dact.data(), &added);
                    if (added > 0) {
                        fill_ms += ms_since(t0);
                        fill_ranks += added;
                    }
                    if (::eahr::trace_on())
                        std::fprintf(stderr, "eahr ahead depth=%lld expected_sparse_ms=%.2f added=%lld fill_ms=%.2f\n",
                                     static_cast<long long>(ahead), expect, static_cast<long long>(added),
                                     ms_since(t0));
                }
            }
            int64_t* ids = dids.get(static_cast<size_t>(B) * m);
            float* sc = dscores.get(static_cast<size_t>(B) * m);
            if (dense_rc == EAHR_OK)
                dense_rc = merged ? pvs_merge_next(merged, static_cast<int32_t>(m), dact.data(), ids, sc,
                                                   dcnt.data(), dsts.data())
                                  : obs ? pvs_next(cl.st, static_cast<int32_t>(m), dact.data(), ids, sc,
                                                   dcnt.data(), dsts.data())
                                        // the fusion needs the ids only
                                        : pvs_next_ids(cl.st, static_cast<int32_t>(m), dact.data(), ids,
                                                       dcnt.data(), dsts.data());
            // While the sparse channel is still busy, certify the dense ranks
            // of the next depths ahead (they are served from the cache later;
            // the output does not depend on it).
            int64_t ahead = depth;
            while (dense_rc == EAHR_OK && !merged && sparse_running && ahead <= cap / ep.growth &&
                   !sparse_done.load(std::memory_order_acquire)) {
                // remaining sparse time: from the share of postings of the
                // finished queries (a first call scores about its postings),
                // or (none finished yet) at least the time it has run so far
                const int64_t fin = sparse_cost_done.load(std::memory_order_relaxed);
                const double run = ms_since(t_sparse0);
                const double left = fin > 0 ? run * static_cast<double>(sparse_cost - fin) / fin : run;
                const double rate = fill_ranks > 0 ? fill_ms / static_cast<double>(fill_ranks) : 0.0;
                const double est = rate * static_cast<double>((ahead * ep.growth - ahead) * nd);
                if (est > left) break;
                ahead *= ep.growth;
                const auto tf = std::chrono::steady_clock::now();
                int64_t added = 0;
                dense_rc = pvs_fill(cl.st, ahead, dact.data(), &added);
                if (added > 0) {
                    fill_ms += ms_since(tf);
                    fill_ranks += added;
                }
                if (::eahr::trace_on())
                    std::fprintf(stderr,
                                 "eahr fill depth=%lld sparse_postings_done=%lld/%lld sparse_left_ms=%.2f "
                                 "est_ms=%.2f added=%lld fill_ms=%.2f\n",
                                 static_cast<long long>(ahead), static_cast<long long>(fin),
                                 static_cast<long long>(sparse_cost), left, est,
                                 static_cast<long long>(added), ms_since(tf));
            }
            r_dense = ms_since(t0);
            t_dense += r_dense;
        }
        if (sparse_inline) sparse_work();
        if (sparse_running) {
            W.sparse.wait();
            sparse_running = false;
            if (first_round) {
                first_sparse_ms = r_sparse;
                first_sparse_cost = sparse_cost;
                first_sparse_par = sparse_par;
            }
        }
        if (any_sparse) last_sparse_ms = r_sparse;
        first_round = false;
        EAHR_TRY(dense_rc);
        for (int32_t b = 0; b < B; ++b)
            if (sparse_rc[b] != EAHR_OK) {
                ::eahr::set_error("%s", sparse_err.c_str());
                return sparse_rc[b];
            }
        if (obs)
            for (int32_t b = 0; b < B; ++b) {
                if (F[b].resolved || failed[b]) continue;
                if (dact[b] && dsts[b] != EAHR_LIST_FAILED)
                    observe(b, 0, dids.p.get() + static_cast<size_t>(b) * m,
                            dscores.p.get() + static_cast<size_t>(b) * m, dcnt[b]);
                if (sact[b] && ssts[b] != EAHR_LIST_FAILED)
                    observe(b, 1, sids[b].data(), sscores[b].data(), scnt[b]);
            }
        // merge this round's ranks and certify
        const auto t0 = std::chrono::steady_clock::now();
        int64_t busy = 0;
        for (int32_t b = 0; b < B; ++b) busy += !F[b].resolved && !failed[b] && (dact[b] || sact[b]);
        // one query per task; a long append of one of few queries takes the
        // threads the others leave
        for (int32_t b = 0; b < B; ++b) F[b].threads = std::max<int>(1, threads / std::max<int64_t>(busy, 1));
        auto certify_one = [&](int64_t b) {
            if (F[b].resolved || failed[b]) return;
            if (dact[b]) {
                if (dsts[b] == EAHR_LIST_FAILED) {
                    failed[b] = 1;
                    dstat[b] = EAHR_LIST_FAILED;
                    return;
                }
                F[b].append(0, dids.p.get() + static_cast<size_t>(b) * m, dcnt[b]);
                if (dsts[b] == EAHR_LIST_EXHAUSTED) {
                    F[b].L[0].open = false;
                    dstat[b] = EAHR_LIST_EXHAUSTED;
                }
            }
            if (sact[b]) {
                if (ssts[b] == EAHR_LIST_FAILED) {
                    failed[b] = 1;
                    sstat[b] = EAHR_LIST_FAILED;
                    return;
                }
                F[b].append(1, sids[b].data(), scnt[b]);
                if (ssts[b] == EAHR_LIST_EXHAUSTED) {
                    F[b].L[1].open = false;
                    sstat[b] = EAHR_LIST_EXHAUSTED;
                }
            }
            if (F[b].dup) {   // a channel repeated an id: its list is not a ranking
                failed[b] = 1;
                return;
            }
            rounds[b] += 1;
            F[b].certify();
        };
        parallel_for(B, threads, certify_one);
        // settled queries read no further dense ranks
        if (cl.st)
            for (int32_t b = 0; b < B; ++b)
                if ((F[b].resolved || failed[b]) && !retired[b]) {
                    pvs_retire(cl.st, b);
                    retired[b] = 1;
                }
        const double r_fuse = ms_since(t0);
        t_fuse += r_fuse;
        if (::eahr::trace_on()) {
            int64_t nd = 0, ns = 0, open_q = 0;
            for (int32_t b = 0; b < B; ++b) {
                nd += dact[b];
                ns += sact[b];
                open_q += !F[b].resolved && !failed[b];
            }
            std::fprintf(stderr,
                         "eahr round depth=%lld dense_q=%lld sparse_q=%lld dense_ms=%.2f sparse_ms=%.2f "
                         "certify_ms=%.2f round_ms=%.2f unresolved_after=%lld\n",
                         static_cast<long long>(depth), static_cast<long long>(nd),
                         static_cast<long long>(ns), r_dense, r_sparse, r_fuse, ms_since(t_round),
                         static_cast<long long>(open_q));
        }
        depth = (depth > (INT64_MAX / ep.growth)) ? INT64_MAX : depth * ep.growth;
    }
    if (!merged && (fill_ranks > 0 || (first_sparse_ms > 0.0 && first_sparse_cost > 0))) {
        std::lock_guard<std::mutex> lk(g_rates_mu);
        Rates& r = g_rates[rates_key];
        if (fill_ranks > 0) r.dense_ms_per_rank = fill_ms / static_cast<double>(fill_ranks);
        if (first_sparse_ms > 0.0 && first_sparse_cost > 0)
            r.sparse_ms_per_posting =
                first_sparse_ms * static_cast<double>(first_sparse_par) / static_cast<double>(first_sparse_cost);
    }
    // a rescored score outside its interval fails its query even when the
    // failure came from work-ahead that no pvs_next has reported yet
    // (App. A.1: PVS fails the request)
    if (cl.st)
        for (int32_t b = 0; b < B; ++b)
            if (!failed[b] && pvs_query_failed(cl.st, b)) {
                failed[b] = 1;
                dstat[b] = EAHR_LIST_FAILED;
            }
    if (prof) pvs_profile_add_host(t_dense, t_sparse, t_fuse);
    std::vector<int64_t> d_evals(B, 0), s_posts(B, 0), s_scored(B, 0);
    for (int32_t b = 0; b < B; ++b) {
        if (cl.st) d_evals[b] = pvs_query_evals(cl.st, b);
        if (!cl.sp.empty() && cl.sp[b]) {
            s_posts[b] = cl.sp[b]->postings_visited;
            s_scored[b] = cl.sp[b]->items_scored;
        }
        if (cl.gsp) {
            int64_t c[3];
            if (pbm_gpu_counters(cl.gsp, b, c) == EAHR_OK) {
                s_posts[b] = c[0];
                s_scored[b] = c[1];
            }
        }
    }
    if (::eahr::trace_on()) {
        const auto tc = std::chrono::steady_clock::now();
        if (cl.st) pvs_close(cl.st);
        cl.st = nullptr;
        const double cd = ms_since(tc);
        for (auto*& sp : cl.sp) {
            if (sp) pbm_close(sp);
            sp = nullptr;
        }
        if (cl.gsp) pbm_gpu_close(cl.gsp);
        cl.gsp = nullptr;
        std::fprintf(stderr, "eahr close dense_ms=%.2f sparse_ms=%.2f call_ms=%.2f\n", cd,
                     ms_since(tc) - cd, ms_since(t_call));
    }
    bool any_failed = false;
    for (int32_t b = 0; b < B; ++b) {
        const auto& f = F[b];
        const int64_t q = failed[b] ? 0 : static_cast<int64_t>(f.A.size());
        for (int64_t j = 0; j < ep.K; ++j) out_ids[static_cast<int64_t>(b) * ep.K + j] = (j < q) ? f.A[j] : -1;
        out_count[b] = static_cast<int32_t>(q);
        out_status[b] = failed[b] ? EAHR_LIST_FAILED : 0;
        any_failed |= failed[b] != 0;
        if (stats) {
            eahr_query_stats& s = stats[b];
            s.dense_depth = static_cast<int64_t>(f.L[0].size());
            s.sparse_depth = static_cast<int64_t>(f.L[1].size());
            s.dense_len = (dstat[b] == EAHR_LIST_EXHAUSTED) ? s.dense_depth : -1;
            s.sparse_len = (sstat[b] == EAHR_LIST_EXHAUSTED) ? s.sparse_depth : -1;
            s.dense_status = dstat[b];
            s.sparse_status = sstat[b];
            s.rounds = rounds[b];
            s.resolved = f.resolved ? 1 : 0;
            s.dense_evals = d_evals[b];
            s.sparse_postings = s_posts[b];
            s.sparse_scored = s_scored[b];
        }
    }
    if (any_failed) EAHR_FAIL(EAHR_E_FAILED, "eahr_topk: a ranked list failed");
    return EAHR_OK;
}

extern "C" int eahr_topk(const pvs_index* dense, int64_t epoch, const pbm_index* sparse,
                         const float* q_dense, int32_t q_ptr_kind,
                         const eahr_sparse_query* q_sparse, int32_t B, const eahr_params* params,
                         int64_t* out_ids, int32_t* out_count, int32_t* out_status,
                         eahr_query_stats* stats) {
    return topk_impl(dense, epoch, nullptr, sparse, q_dense, q_ptr_kind, q_sparse, B, params, out_ids,
                     out_count, out_status, stats);
}

extern "C" int eahr_topk_merged(pvs_merge* dense, const pbm_index* sparse,
                                const eahr_sparse_query* q_sparse, int32_t B,
                                const eahr_params* params, int64_t* out_ids, int32_t* out_count,
                                int32_t* out_status, eahr_query_stats* stats) {
    if (params && params->w_dense > 0 && !dense)
        EAHR_FAIL(EAHR_E_INVALID, "eahr_topk_merged: dense channel missing");
    if (params && params->dense_generator != EAHR_GEN_INTERVALS)
        EAHR_FAIL(EAHR_E_INVALID, "eahr_topk_merged: the merged channel uses interval scans");
    if (params && params->w_dense > 0 && !eahr_merge_unread(dense))
        EAHR_FAIL(EAHR_E_INVALID, "eahr_topk_merged: the merge has already been read");
    return topk_impl(nullptr, 0, dense, sparse, nullptr, EAHR_PTR_HOST, q_sparse, B, params, out_ids,
                     out_count, out_status, stats);
}

extern "C" int eahr_set_rank_observer(eahr_rank_observer fn, void* user) {
    std::lock_guard<std::mutex> lk(g_obs_mu);
    g_obs = fn;
    g_obs_user = user;
    return EAHR_OK;
}

extern "C" int eahr_fuse_lists(const int64_t* list_d, int64_t n_d, const int64_t* list_s,
                               int64_t n_s, const eahr_params* params, int32_t step,
                               int64_t* out_ids, int32_t* out_count, eahr_query_stats* stats) {
    if (!params || !out_ids || !out_count || n_d < 0 || n_s < 0 || step < 0 ||
        (n_d > 0 && !list_d) || (n_s > 0 && !list_s))
        EAHR_FAIL(EAHR_E_INVALID, "eahr_fuse_lists: bad arguments");
    const eahr_params& ep = *params;
    EAHR_TRY(check_params(ep));
    if (n_d >= (1LL << 31) || n_s >= (1LL << 31)) EAHR_FAIL(EAHR_E_RANGE, "eahr_fuse_lists: lists too long");
    for (int64_t j = 0; j < n_d; ++j)
        if (list_d[j] < 0 || list_d[j] >= (1LL << 31)) EAHR_FAIL(EAHR_E_RANGE, "eahr_fuse_lists: id outside [0, 2^31)");
    for (int64_t j = 0; j < n_s; ++j)
        if (list_s[j] < 0 || list_s[j] >= (1LL << 31)) EAHR_FAIL(EAHR_E_RANGE, "eahr_fuse_lists: id outside [0, 2^31)");
    const Params P{ep.K, ep.k_rrf, {ep.w_dense, ep.w_sparse}};
    Fusion f;
    f.P = &P;
    f.threads = host_threads();
    for (int64_t j = 0; j < n_d; ++j) f.universe = std::max(f.universe, list_d[j] + 1);
    for (int64_t j = 0; j < n_s; ++j) f.universe = std::max(f.universe, list_s[j] + 1);
    // both lists are given whole, so their id range is exact: direct rank
    // arrays from the start keep small steps linear in the depth
    f.enter_direct_mode();
    const int64_t* lists[2] = {list_d, list_s};
    const int64_t lens[2] = {n_d, n_s};
    for (int i = 0; i < 2; ++i) f.L[i].open = P.w[i] > 0 && lens[i] > 0;
    if (ep.K == 0) f.resolved = true;
    int32_t rounds = 0;
    if (ep.schedule == EAHR_SCHED_FROZEN) {
        ::eahr::FrozenSchedule S;
        const bool use[2] = {f.L[0].open, f.L[1].open};
        const int64_t avail[2] = {use[0] ? lens[0] : 0, use[1] ? lens[1] : 0};
        const bool done[2] = {true, true};
        while (!f.resolved) {
            const bool stepped = S.advance(P, avail, done, use);
            for (int i = 0; i < 2; ++i) {
                const int64_t have = static_cast<int64_t>(f.L[i].size());
                if (S.d[i] > have) f.append(i, lists[i] + have, S.d[i] - have);
                if (f.L[i].open && static_cast<int64_t>(f.L[i].size()) == avail[i]) f.L[i].open = false;
            }
            if (f.dup) EAHR_FAIL(EAHR_E_INVALID, "eahr_fuse_lists: a list repeats an id");
            rounds += 1;
            f.certify();
            if (!f.resolved && !stepped)
                EAHR_FAIL(EAHR_E_INVALID, "eahr_fuse_lists: lists hold duplicate ids");
        }
    }
    int64_t depth = step > 0 ? step : ep.depth0;
    while (!f.resolved) {
        for (int i = 0; i < 2; ++i) {
            if (!f.L[i].open) continue;
            const int64_t have = static_cast<int64_t>(f.L[i].size());
            const int64_t upto = std::min(depth, lens[i]);
            if (upto > have) f.append(i, lists[i] + have, upto - have);
            if (static_cast<int64_t>(f.L[i].size()) == lens[i]) f.L[i].open = false;
        }
        if (f.dup) EAHR_FAIL(EAHR_E_INVALID, "eahr_fuse_lists: a list repeats an id");
        rounds += 1;
        f.certify();
        if (step > 0) depth += step;
        else depth = (depth > INT64_MAX / ep.growth) ? INT64_MAX : depth * ep.growth;
        if (!f.resolved && !f.L[0].open && !f.L[1].open) {
            f.certify();   // both complete: certification resolves every position
            if (!f.resolved) EAHR_FAIL(EAHR_E_INVALID, "eahr_fuse_lists: lists hold duplicate ids");
        }
    }
    const int64_t q = static_cast<int64_t>(f.A.size());
    for (int64_t j = 0; j < ep.K; ++j) out_ids[j] = (j < q) ? f.A[j] : -1;
    *out_count = static_cast<int32_t>(q);
    if (stats) {
        stats->dense_depth = static_cast<int64_t>(f.L[0].size());
        stats->sparse_depth = static_cast<int64_t>(f.L[1].size());
        stats->dense_len = f.L[0].open ? -1 : stats->dense_depth;
        stats->sparse_len = f.L[1].open ? -1 : stats->sparse_depth;
        stats->dense_status = f.L[0].open ? EAHR_LIST_OPEN : EAHR_LIST_EXHAUSTED;
        stats->sparse_status = f.L[1].open ? EAHR_LIST_OPEN : EAHR_LIST_EXHAUSTED;
        stats->rounds = rounds;
        stats->resolved = f.resolved ? 1 : 0;
        stats->dense_evals = 0;
        stats->sparse_postings = 0;
        stats->sparse_scored = 0;
    }
    return EAHR_OK;
}
