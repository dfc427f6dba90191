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
// is kept ordered by (F desc, id asc).  x_dag and the strongest competitor
// y are therefore among at most six items, and each position is decided as
// in Sec. 2.2: (L(x_dag), x_dag) must precede (U(y), y) for every other
// remaining y, and L(x_dag) > B strictly.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <memory>
#include <new>
#include <set>
#include <vector>

#include "common.h"
#include "eahr.h"

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
        uint64_t x = static_cast<uint64_t>(id) * 0x9E3779B97F4A7C15ull;
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

struct BothOrder {   // (F desc, id asc)
    bool operator()(const std::pair<Frac, int64_t>& a, const std::pair<Frac, int64_t>& b) const {
        const int c = cmp(a.first, b.first);
        if (c != 0) return c > 0;
        return a.second < b.second;
    }
};

struct Fusion {
    const Params* P = nullptr;
    std::vector<int64_t> list[2];   // exact prefixes read so far
    bool open[2] = {true, true};
    int64_t cursor[2] = {0, 0};     // first possibly single-list unfixed item
    ItemMap items;
    std::set<std::pair<Frac, int64_t>, BothOrder> both;
    std::vector<int64_t> A;
    bool resolved = false;

    Frac F_both(const ItemMap::Slot* s) const {
        return add(g(*P, 0, s->rank[0]), g(*P, 1, s->rank[1]));
    }

    void append(int i, const int64_t* ids, int32_t n) {
        for (int32_t j = 0; j < n; ++j) {
            const int64_t x = ids[j];
            list[i].push_back(x);
            ItemMap::Slot* s = items.get(x);
            s->rank[i] = static_cast<int32_t>(list[i].size());
            if (!s->fixed && s->rank[1 - i] > 0) both.insert({F_both(s), x});
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
            if (!both.empty()) {
                const auto& top = *both.begin();
                c[nc++] = Cand{top.second, top.first, top.first, 0, -1};
            }
            for (int i = 0; i < 2; ++i) {
                cursor[i] = std::max<int64_t>(cursor[i], 0);
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
                    auto it = both.begin();
                    ++it;
                    if (it != both.end()) ok = precedes(X.L, X.id, it->first, it->second);
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
            ItemMap::Slot* s = items.find(X.id);
            s->fixed = 1;
            if (X.kind == 0) both.erase(both.begin());
        }
        if (static_cast<int64_t>(A.size()) >= P->K) {
            resolved = true;
        } else if (B.num == 0 && both.empty() && single_from(0, cursor[0]) < 0 &&
                   single_from(1, cursor[1]) < 0) {
            resolved = true;   // nothing unseen or remaining can score: q_K = |A|
        }
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
    if (ep.K < 0 || ep.depth0 < 1 || ep.growth < 2 || ep.k_rrf < 1 || ep.k_rrf > (1 << 20) ||
        ep.w_dense < 0 || ep.w_dense > 1024 || ep.w_sparse < 0 || ep.w_sparse > 1024)
        EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: parameters out of range");
    const bool use_dense = ep.w_dense > 0, use_sparse = ep.w_sparse > 0;
    if (use_dense && (!dense || !q_dense)) EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: dense channel missing");
    if (use_sparse && (!sparse || !q_sparse)) EAHR_FAIL(EAHR_E_INVALID, "eahr_topk: sparse channel missing");
    Params P{ep.K, ep.k_rrf, {ep.w_dense, ep.w_sparse}};

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
    if (ep.K == 0) {
        for (int32_t b = 0; b < B; ++b) F[b].resolved = true;
    }
    std::vector<int64_t> ids;
    std::vector<float> scores;
    std::vector<int32_t> cnt(B), sts(B);
    std::vector<uint8_t> active(B);
    int64_t depth = ep.depth0;
    for (;;) {
        bool any = false;
        for (int32_t b = 0; b < B; ++b) any |= !F[b].resolved && !failed[b];
        if (!any) break;
        // dense channel: one batched call for every query still needing ranks
        if (use_dense) {
            int64_t m = 0;
            for (int32_t b = 0; b < B; ++b) {
                active[b] = !F[b].resolved && !failed[b] && F[b].open[0] &&
                            static_cast<int64_t>(F[b].list[0].size()) < depth;
                if (active[b]) m = std::max<int64_t>(m, depth - static_cast<int64_t>(F[b].list[0].size()));
            }
            if (m > 0) {
                if (m > (1LL << 30)) m = 1LL << 30;
                ids.resize(static_cast<size_t>(B) * m);
                scores.resize(static_cast<size_t>(B) * m);
                EAHR_TRY(pvs_next(cl.st, static_cast<int32_t>(m), active.data(), ids.data(),
                                  scores.data(), cnt.data(), sts.data()));
                for (int32_t b = 0; b < B; ++b) {
                    if (!active[b]) continue;
                    if (sts[b] == EAHR_LIST_FAILED) {
                        failed[b] = 1;
                        dstat[b] = EAHR_LIST_FAILED;
                        continue;
                    }
                    F[b].append(0, ids.data() + static_cast<size_t>(b) * m, cnt[b]);
                    if (sts[b] == EAHR_LIST_EXHAUSTED) {
                        F[b].open[0] = false;
                        dstat[b] = EAHR_LIST_EXHAUSTED;
                    }
                }
            }
        }
        if (use_sparse) {
            for (int32_t b = 0; b < B; ++b) {
                if (F[b].resolved || failed[b] || !F[b].open[1]) continue;
                const int64_t need = depth - static_cast<int64_t>(F[b].list[1].size());
                if (need <= 0) continue;
                const int32_t m = static_cast<int32_t>(std::min<int64_t>(need, 1LL << 30));
                ids.resize(m);
                scores.resize(m);
                int32_t c = 0, s = 0;
                EAHR_TRY(pbm_next(cl.sp[b], m, ids.data(), scores.data(), &c, &s));
                if (s == EAHR_LIST_FAILED) {
                    failed[b] = 1;
                    sstat[b] = EAHR_LIST_FAILED;
                    continue;
                }
                F[b].append(1, ids.data(), c);
                if (s == EAHR_LIST_EXHAUSTED) {
                    F[b].open[1] = false;
                    sstat[b] = EAHR_LIST_EXHAUSTED;
                }
            }
        }
        for (int32_t b = 0; b < B; ++b) {
            if (F[b].resolved || failed[b]) continue;
            rounds[b] += 1;
            F[b].certify();
        }
        depth = (depth > (INT64_MAX / ep.growth)) ? INT64_MAX : depth * ep.growth;
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
    if (ep.K < 0 || ep.depth0 < 1 || ep.growth < 2 || ep.k_rrf < 1 || ep.k_rrf > (1 << 20) ||
        ep.w_dense < 0 || ep.w_dense > 1024 || ep.w_sparse < 0 || ep.w_sparse > 1024)
        EAHR_FAIL(EAHR_E_INVALID, "eahr_fuse_lists: parameters out of range");
    if (n_d >= (1LL << 31) || n_s >= (1LL << 31)) EAHR_FAIL(EAHR_E_RANGE, "eahr_fuse_lists: lists too long");
    Params P{ep.K, ep.k_rrf, {ep.w_dense, ep.w_sparse}};
    Fusion f;
    f.P = &P;
    const int64_t* lists[2] = {list_d, list_s};
    const int64_t lens[2] = {n_d, n_s};
    for (int i = 0; i < 2; ++i) {
        f.open[i] = P.w[i] > 0;
        if (f.open[i] && lens[i] == 0) f.open[i] = false;
    }
    if (ep.K == 0) f.resolved = true;
    int32_t rounds = 0;
    int64_t depth = step > 0 ? step : ep.depth0;
    while (!f.resolved) {
        for (int i = 0; i < 2; ++i) {
            if (!f.open[i]) continue;
            const int64_t have = static_cast<int64_t>(f.list[i].size());
            const int64_t upto = std::min(depth, lens[i]);
            if (upto > have) f.append(i, lists[i] + have, static_cast<int32_t>(upto - have));
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
