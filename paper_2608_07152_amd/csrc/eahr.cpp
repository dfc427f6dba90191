// Exact adaptive weighted-RRF fusion of the dense (PVS) and sparse (PBM)
// channels (Sec. 2.1, Sec. 2.2).
//
// g_i(r) = 1 / (r / w_i + k - 1) = w_i / (r + w_i (k - 1)) with integer k and
// w_i, so every bound is a sum of at most two unit terms w / D and compares
// exactly as a fraction (numerators < 2^43, denominators < 2^64, products
// < 2^107 in unsigned 128-bit integers).
//
// Certification: after every depth round the remaining observed items fall
// into three groups: seen by both lists (L = U = F), seen by the dense list
// only (L = g_d(r_d), U = L + u_s), seen by the sparse list only.  Inside a
// single-list group L and U strictly decrease with the rank, so the group's
// best L and best U belong to its first unfixed member; the both-seen group
// is a binary heap on (F desc, id asc), whose best two items are the root and
// the better child.  x_dag and its strongest competitor y are therefore among
// at most six items, and each position is decided as in Sec. 2.2:
// (L(x_dag), x_dag) must precede (U(y), y) for every other remaining y, and
// L(x_dag) > B strictly.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstring>
#include <memory>
#include <new>
#include <thread>
#include <vector>

#include "common.h"
#include "eahr.h"
#include "host_parallel.h"
#include "pvs_internal.h"

namespace {

typedef unsigned __int128 u128;

struct Frac {
    u128 num = 0;
    u128 den = 1;
};

inline int cmp(const Frac& a, const Frac& b) {
    const u128 l = a.num * b.den, r = b.num * a.den;
    return (l < r) ? -1 : (l > r) ? 1 : 0;
}
inline Frac add(const Frac& a, const Frac& b) {
    if (a.num == 0) return b;
    if (b.num == 0) return a;
    return Frac{a.num * b.den + b.num * a.den, a.den * b.den};
}

struct Params {
    int64_t K, k, w[2];
};

// g_i(r), 1-based r; 0 when w_i = 0.
inline Frac g(const Params& P, int i, int64_t r) {
    if (P.w[i] == 0) return Frac{0, 1};
    return Frac{static_cast<u128>(P.w[i]), static_cast<u128>(r + P.w[i] * (P.k - 1))};
}

// (a, x) precedes (b, y): a > b, or a == b and x < y.
inline bool precedes(const Frac& a, int64_t x, const Frac& b, int64_t y) {
    const int c = cmp(a, b);
    return c > 0 || (c == 0 && x < y);
}

// Open-addressing map id -> (rank in dense, rank in sparse, fixed flag).
struct ItemMap {
    struct Slot {
        int64_t id;
        int32_t rank[2];
        int32_t fixed;
    };
    std::vector<Slot> slots;
    size_t used = 0;
    ItemMap() { slots.assign(64, Slot{-1, {0, 0}, 0}); }
    static size_t hash(int64_t id) {
        const uint64_t x = static_cast<uint64_t>(id) * 0x9E3779B97F4A7C15ull;
        return static_cast<size_t>(x ^ (x >> 29));
    }
    Slot* find(int64_t id) {
        const size_t mask = slots.size() - 1;
        for (size_t h = hash(id) & mask;; h = (h + 1) & mask) {
            if (slots[h].id == id) return &slots[h];
            if (slots[h].id < 0) return nullptr;
        }
    }
    Slot* get(int64_t id) {
        if ((used + 1) * 2 > slots.size()) rehash(slots.size() * 2);
        const size_t mask = slots.size() - 1;
        for (size_t h = hash(id) & mask;; h = (h + 1) & mask) {
            if (slots[h].id == id) return &slots[h];
            if (slots[h].id < 0) {
                slots[h] = Slot{id, {0, 0}, 0};
                ++used;
                return &slots[h];
            }
        }
    }
    void reserve(size_t n) {
        size_t want = 64;
        while (want < 2 * n + 2) want *= 2;
        if (want > slots.size()) rehash(want);
    }
    void rehash(size_t n) {
        std::vector<Slot> old;
        old.swap(slots);
        slots.assign(n, Slot{-1, {0, 0}, 0});
        used = 0;
        const size_t mask = n - 1;
        for (const Slot& s : old) {
            if (s.id < 0) continue;
            size_t h = hash(s.id) & mask;
            while (slots[h].id >= 0) h = (h + 1) & mask;
            slots[h] = s;
            ++used;
        }
    }
};

struct Scored {
    Frac F;
    int64_t id;
};
// heap order: a below b when b precedes a
struct HeapLess {
    bool operator()(const Scored& a, const Scored& b) const { return precedes(b.F, b.id, a.F, a.id); }
};

struct Fusion {
    const Params* P = nullptr;
    std::vector<int64_t> list[2];   // exact prefixes read so far
    bool open[2] = {true, true};
    int64_t cursor[2] = {0, 0};     // first possibly single-list unfixed item
    ItemMap items;
    std::vector<Scored> both;       // binary heap of unfixed both-seen items
    std::vector<int64_t> A;
    bool resolved = false;

    void append(int i, const int64_t* ids, int64_t n) {
        items.reserve(items.used + static_cast<size_t>(n));
        list[i].reserve(list[i].size() + static_cast<size_t>(n));
        for (int64_t j = 0; j < n; ++j) {
            const int64_t x = ids[j];
            list[i].push_back(x);
            ItemMap::Slot* s = items.get(x);
            s->rank[i] = static_cast<int32_t>(list[i].size());
            if (!s->fixed && s->rank[1 - i] > 0) {
                both.push_back(Scored{add(g(*P, 0, s->rank[0]), g(*P, 1, s->rank[1])), x});
                std::push_heap(both.begin(), both.end(), HeapLess());
            }
        }
    }

    // first unfixed item of list i, at or after position p, seen only by i
    int64_t single_from(int i, int64_t p) {
        for (; p < static_cast<int64_t>(list[i].size()); ++p) {
            const ItemMap::Slot* s = items.find(list[i][p]);
            if (!s->fixed && s->rank[1 - i] == 0) return p;
        }
        return -1;
    }

    Frac u(int i) const {
        return open[i] ? g(*P, i, static_cast<int64_t>(list[i].size()) + 1) : Frac{0, 1};
    }

    void certify() {
        if (resolved) return;
        const Frac ui[2] = {u(0), u(1)};
        const Frac B = add(ui[0], ui[1]);
        while (static_cast<int64_t>(A.size()) < P->K) {
            struct Cand {
                int64_t id;
                Frac L, U;
                int kind;        // 0: both, 1: dense only, 2: sparse only
                int64_t pos;     // list position for single-list items
            };
            Cand c[3];
            int nc = 0;
            if (!both.empty()) c[nc++] = Cand{both[0].id, both[0].F, both[0].F, 0, -1};
            for (int i = 0; i < 2; ++i) {
                const int64_t p = single_from(i, cursor[i]);
                if (p >= 0) {
                    cursor[i] = p;
                    const Frac L = g(*P, i, p + 1);
                    c[nc++] = Cand{list[i][p], L, add(L, ui[1 - i]), 1 + i, p};
                } else {
                    cursor[i] = static_cast<int64_t>(list[i].size());
                }
            }
            if (nc == 0) break;
            int xd = 0;
            for (int j = 1; j < nc; ++j)
                if (precedes(c[j].L, c[j].id, c[xd].L, c[xd].id)) xd = j;
            const Cand& X = c[xd];
            bool ok = cmp(X.L, B) > 0;
            // strongest remaining competitor of each group, x_dag excluded
            for (int j = 0; ok && j < nc; ++j) {
                if (j != xd) {
                    ok = precedes(X.L, X.id, c[j].U, c[j].id);
                    continue;
                }
                if (X.kind == 0) {
                    const size_t n = both.size();
                    int64_t second = -1;
                    if (n > 1) second = 1;
                    if (n > 2 && HeapLess()(both[1], both[2])) second = 2;
                    if (second >= 0) ok = precedes(X.L, X.id, both[second].F, both[second].id);
                } else {
                    const int i = X.kind - 1;
                    const int64_t p = single_from(i, X.pos + 1);
                    if (p >= 0) {
                        const Frac L = g(*P, i, p + 1);
                        ok = precedes(X.L, X.id, add(L, ui[1 - i]), list[i][p]);
                    }
                }
            }
            if (!ok) break;
            A.push_back(X.id);
            items.find(X.id)->fixed = 1;
            if (X.kind == 0) {
                std::pop_heap(both.begin(), both.end(), HeapLess());
                both.pop_back();
            }
        }
        if (static_cast<int64_t>(A.size()) >= P->K) {
            resolved = true;
        } else if (B.num == 0 && both.empty() && single_from(0, cursor[0]) < 0 &&
                   single_from(1, cursor[1]) < 0) {
            resolved = true;   // nothing unseen or remaining can score: q_K = |A|
        }
    }
};

int check_params(const eahr_params& ep) {
    if (ep.K < 0 || ep.depth0 < 1 || ep.growth < 2 || ep.k_rrf < 1 || ep.k_rrf > (1 << 20) ||
        ep.w_dense < 0 || ep.w_dense > 1024 || ep.w_sparse < 0 || ep.w_sparse > 1024)
        EAHR_FAIL(EAHR_E_INVALID, "eahr: parameters out of range");
    return EAHR_OK;
}

using ::eahr::host_threads;
using ::eahr::parallel_for;

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

}  // namespace

extern "C" int eahr_topk(const pvs_index* dense, int64_t epoch, const pbm_index* sparse,
                         const float* q_dense, int32_t q_ptr_kind,
                         const eahr_sparse_query* q_sparse, int32_t B, const eahr_params* params,
                         int64_t* out_ids, int32_t* out_count, int32_t* out_status,
                         eahr_query_stats* stats) {
    if (!params || B <= 0 || !out_ids || !out_count || !out_status)
        EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: bad arguments");
    const eahr_params& ep = *params;
    EAHR_TRY(check_params(ep));
    const bool use_dense = ep.w_dense > 0, use_sparse = ep.w_sparse > 0;
    if (use_dense && (!dense || !q_dense)) EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: dense channel missing");
    if (use_sparse && (!sparse || !q_sparse)) EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: sparse channel missing");
    const Params P{ep.K, ep.k_rrf, {ep.w_dense, ep.w_sparse}};
    const int threads = host_threads();
    const bool prof = pvs_profile_on();
    double t_dense = 0, t_sparse = 0, t_fuse = 0;

    std::vector<Fusion> F(B);
    std::vector<int32_t> dstat(B, EAHR_LIST_EXHAUSTED), sstat(B, EAHR_LIST_EXHAUSTED);
    std::vector<int32_t> rounds(B, 0);
    std::vector<uint8_t> failed(B, 0);
    for (int32_t b = 0; b < B; ++b) {
        F[b].P = &P;
        F[b].open[0] = use_dense;
        F[b].open[1] = use_sparse;
        if (use_dense) dstat[b] = EAHR_LIST_OPEN;
        if (use_sparse) sstat[b] = EAHR_LIST_OPEN;
        if (ep.K == 0) F[b].resolved = true;
    }
    struct Cleanup {
        pvs_state* st = nullptr;
        std::vector<pbm_state*> sp;
        ~Cleanup() {
            if (st) pvs_close(st);
            for (auto* s : sp)
                if (s) pbm_close(s);
        }
    } cl;
    if (use_dense) EAHR_TRY(pvs_open(dense, epoch, q_dense, B, q_ptr_kind, &cl.st));
    if (use_sparse) {
        cl.sp.assign(B, nullptr);
        for (int32_t b = 0; b < B; ++b) EAHR_TRY(pbm_open(sparse, &q_sparse[b], &cl.sp[b]));
    }
    RawBuf<int64_t> dids;
    RawBuf<float> dscores;
    std::vector<int32_t> dcnt(B, 0), dsts(B);
    std::vector<uint8_t> dact(B, 0);
    std::vector<std::vector<int64_t>> sids(B);
    std::vector<std::vector<float>> sscores(B);
    std::vector<int32_t> scnt(B, 0), ssts(B, EAHR_LIST_OPEN);
    std::vector<uint8_t> sact(B, 0);
    std::vector<int> sparse_rc(B, EAHR_OK);
    int64_t depth = ep.depth0;
    for (;;) {
        bool any = false;
        for (int32_t b = 0; b < B; ++b) any |= !F[b].resolved && !failed[b];
        if (!any) break;
        // requests of this round: every Open list of an unresolved query to `depth`
        int64_t m = 0;
        for (int32_t b = 0; b < B; ++b) {
            const bool live = !F[b].resolved && !failed[b];
            dact[b] = live && use_dense && F[b].open[0] &&
                      static_cast<int64_t>(F[b].list[0].size()) < depth;
            sact[b] = live && use_sparse && F[b].open[1] &&
                      static_cast<int64_t>(F[b].list[1].size()) < depth;
            dcnt[b] = 0;
            scnt[b] = 0;
            if (dact[b]) m = std::max<int64_t>(m, depth - static_cast<int64_t>(F[b].list[0].size()));
        }
        if (m > (1LL << 30)) m = 1LL << 30;
        // sparse channel on worker threads while the dense channel runs on the GPU
        std::thread sparse_thread;
        auto t_round = std::chrono::steady_clock::now();
        auto sparse_work = [&]() {
            const auto t0 = std::chrono::steady_clock::now();
            parallel_for(B, std::max(1, threads - 1), [&](int64_t b) {
                if (!sact[b]) return;
                const int64_t need = std::min<int64_t>(depth - static_cast<int64_t>(F[b].list[1].size()), 1LL << 30);
                sids[b].resize(static_cast<size_t>(need));
                sscores[b].resize(static_cast<size_t>(need));
                sparse_rc[b] = pbm_next(cl.sp[b], static_cast<int32_t>(need), sids[b].data(),
                                        sscores[b].data(), &scnt[b], &ssts[b]);
            });
            t_sparse += ms_since(t0);
        };
        bool any_sparse = false;
        for (int32_t b = 0; b < B; ++b) any_sparse |= sact[b] != 0;
        if (any_sparse) sparse_thread = std::thread(sparse_work);
        int dense_rc = EAHR_OK;
        if (m > 0) {
            const auto t0 = std::chrono::steady_clock::now();
            int64_t* ids = dids.get(static_cast<size_t>(B) * m);
            float* sc = dscores.get(static_cast<size_t>(B) * m);
            dense_rc = pvs_next(cl.st, static_cast<int32_t>(m), dact.data(), ids, sc, dcnt.data(), dsts.data());
            t_dense += ms_since(t0);
        }
        if (sparse_thread.joinable()) sparse_thread.join();
        (void)t_round;
        EAHR_TRY(dense_rc);
        for (int32_t b = 0; b < B; ++b) EAHR_TRY(sparse_rc[b]);
        // merge this round's ranks and certify, one query per task
        const auto t0 = std::chrono::steady_clock::now();
        parallel_for(B, threads, [&](int64_t b) {
            if (F[b].resolved || failed[b]) return;
            if (dact[b]) {
                if (dsts[b] == EAHR_LIST_FAILED) {
                    failed[b] = 1;
                    dstat[b] = EAHR_LIST_FAILED;
                    return;
                }
                F[b].append(0, dids.p.get() + static_cast<size_t>(b) * m, dcnt[b]);
                if (dsts[b] == EAHR_LIST_EXHAUSTED) {
                    F[b].open[0] = false;
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
                    F[b].open[1] = false;
                    sstat[b] = EAHR_LIST_EXHAUSTED;
                }
            }
            rounds[b] += 1;
            F[b].certify();
        });
        t_fuse += ms_since(t0);
        depth = (depth > (INT64_MAX / ep.growth)) ? INT64_MAX : depth * ep.growth;
    }
    if (prof) pvs_profile_add_host(t_dense, t_sparse, t_fuse);
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
            s.dense_depth = static_cast<int64_t>(f.list[0].size());
            s.sparse_depth = static_cast<int64_t>(f.list[1].size());
            s.dense_len = (dstat[b] == EAHR_LIST_EXHAUSTED) ? s.dense_depth : -1;
            s.sparse_len = (sstat[b] == EAHR_LIST_EXHAUSTED) ? s.sparse_depth : -1;
            s.dense_status = dstat[b];
            s.sparse_status = sstat[b];
            s.rounds = rounds[b];
            s.resolved = f.resolved ? 1 : 0;
        }
    }
    if (any_failed) EAHR_FAIL(EAHR_E_FAILED, "eahr_topk: a ranked list failed");
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
    const Params P{ep.K, ep.k_rrf, {ep.w_dense, ep.w_sparse}};
    Fusion f;
    f.P = &P;
    const int64_t* lists[2] = {list_d, list_s};
    const int64_t lens[2] = {n_d, n_s};
    for (int i = 0; i < 2; ++i) f.open[i] = P.w[i] > 0 && lens[i] > 0;
    if (ep.K == 0) f.resolved = true;
    int32_t rounds = 0;
    int64_t depth = step > 0 ? step : ep.depth0;
    while (!f.resolved) {
        for (int i = 0; i < 2; ++i) {
            if (!f.open[i]) continue;
            const int64_t have = static_cast<int64_t>(f.list[i].size());
            const int64_t upto = std::min(depth, lens[i]);
            if (upto > have) f.append(i, lists[i] + have, upto - have);
            if (static_cast<int64_t>(f.list[i].size()) == lens[i]) f.open[i] = false;
        }
        rounds += 1;
        f.certify();
        if (step > 0) depth += step;
        else depth = (depth > INT64_MAX / ep.growth) ? INT64_MAX : depth * ep.growth;
        if (!f.resolved && !f.open[0] && !f.open[1]) {
            f.certify();   // both complete: certification resolves every position
            if (!f.resolved) EAHR_FAIL(EAHR_E_INVALID, "eahr_fuse_lists: lists hold duplicate ids");
        }
    }
    const int64_t q = static_cast<int64_t>(f.A.size());
    for (int64_t j = 0; j < ep.K; ++j) out_ids[j] = (j < q) ? f.A[j] : -1;
    *out_count = static_cast<int32_t>(q);
    if (stats) {
        stats->dense_depth = static_cast<int64_t>(f.list[0].size());
        stats->sparse_depth = static_cast<int64_t>(f.list[1].size());
        stats->dense_len = f.open[0] ? -1 : stats->dense_depth;
        stats->sparse_len = f.open[1] ? -1 : stats->sparse_depth;
        stats->dense_status = f.open[0] ? EAHR_LIST_OPEN : EAHR_LIST_EXHAUSTED;
        stats->sparse_status = f.open[1] ? EAHR_LIST_OPEN : EAHR_LIST_EXHAUSTED;
        stats->rounds = rounds;
        stats->resolved = f.resolved ? 1 : 0;
    }
    return EAHR_OK;
}
