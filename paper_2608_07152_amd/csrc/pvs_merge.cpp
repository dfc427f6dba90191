// Hierarchical merging of exact dense rankings (Sec. 2.4): Segment rankings
// are merged inside a Shard, Shard rankings across Shards, each time by
// (score descending, global id ascending), giving one resumable request-level
// ranking with the same exact-prefix contract as pvs_next (Sec. 2.1).
//
// A Segment is a pvs_index with a map from its rows to global item ids
// (strictly ascending, so its own (score, row) order is the global (score,
// id) order) and a version per row.  The merge is a host layer over the
// public dense-channel calls: every source is read in chunks through
// pvs_next (or a child merge), and the next merged rank is taken only when
// every source that is still Open has a buffered head, so no unread rank of
// any source can precede it.
//
// An item held by several sources (an id visible in more than one of them)
// is emitted once: a later copy with the same score and version is dropped.
// Copies that disagree invalidate the request whatever depth it reaches
// (Sec. 2.4), so they are found when a merge is opened: every id visible in
// more than one source is compared across its copies (versions for all
// queries, authoritative scores per query), and each query with a
// disagreeing copy is Failed from the start (sticky), as is a query whose
// source fails.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <memory>
#include <new>
#include <unordered_map>
#include <vector>

#include "common.h"
#include "pvs_internal.h"

namespace {

struct Item {
    int64_t id;
    float score;
    int64_t version;
};

// A visible copy of an item: its global id, the Segment state holding it,
// its row there and its version.
struct Copy {
    int64_t gid;
    pvs_state* st;
    int64_t row;
    int64_t version;
};

// (score, id) precedes: higher score, then lower id.  Scores are finite and
// -0 == +0 under IEEE comparison.
inline bool precedes(const Item& a, const Item& b) {
    return a.score > b.score || (a.score == b.score && a.id < b.id);
}

}  // namespace

struct pvs_merge {
    struct Source {
        // exactly one of these is set
        pvs_state* st = nullptr;         // a Segment's dense state
        pvs_merge* child = nullptr;      // a Shard (a merge of Segments)
        std::vector<int64_t> gid;        // Segment: row -> global id
        std::vector<int64_t> version;    // Segment: row -> version (empty: 0)
        // per query: buffered ranks not yet merged, and the source's state
        std::vector<std::vector<Item>> buf;
        std::vector<size_t> pos;
        std::vector<int32_t> status;
    };
    int32_t B = 0;
    std::vector<Source> src;
    std::vector<Copy> copies;                  // every visible copy below this merge, by gid
    std::unordered_map<int64_t, int> shared;   // ids visible in more than one source
    struct Query {
        bool failed = false;
        bool has_last = false;
        Item last{};                           // last emitted rank
        std::unordered_map<int64_t, Item> seen;   // emitted shared ids
        int64_t emitted = 0;
    };
    std::vector<Query> q;
    bool owns_children = false;
    ~pvs_merge();
};

pvs_merge::~pvs_merge() {
    for (auto& s : src) {
        if (s.st) pvs_close(s.st);
        if (s.child && owns_children) delete s.child;
    }
}

namespace {

// Sorts the visible copies of every source of mg (already in mg->copies) by
// global id, records the ids visible in more than one copy and fails up
// front every query for which two copies of one id disagree: a different
// version fails every query, a different authoritative float32 score the
// query it differs for (the copies are scored with pvs_scores, the same
// arithmetic that ranks them).
int find_conflicts(pvs_merge* mg) {
    auto& cp = mg->copies;
    std::stable_sort(cp.begin(), cp.end(), [](const Copy& a, const Copy& b) { return a.gid < b.gid; });
    std::vector<std::pair<size_t, size_t>> runs;   // [first, last) of ids with several copies
    for (size_t i = 0; i < cp.size();) {
        size_t j = i + 1;
        while (j < cp.size() && cp[j].gid == cp[i].gid) ++j;
        if (j - i > 1) {
            runs.emplace_back(i, j);
            mg->shared[cp[i].gid] = 1;
        }
        i = j;
    }
    if (runs.empty()) return EAHR_OK;
    bool version_conflict = false;
    for (const auto& r : runs)
        for (size_t k = r.first + 1; k < r.second; ++k) version_conflict |= cp[k].version != cp[r.first].version;
    if (version_conflict) {
        for (auto& Q : mg->q) Q.failed = true;
        return EAHR_OK;
    }
    // scores of every shared copy, per query: one pvs_scores call per
    // (Segment state, query) over that state's shared rows
    std::vector<pvs_state*> states;
    for (const auto& r : runs)
        for (size_t k = r.first; k < r.second; ++k) states.push_back(cp[k].st);
    std::sort(states.begin(), states.end());
    states.erase(std::unique(states.begin(), states.end()), states.end());
    std::vector<std::vector<int64_t>> rows(states.size());
    std::vector<size_t> slot(cp.size(), 0);   // copy k -> its index in its state's row list
    for (const auto& r : runs)
        for (size_t k = r.first; k < r.second; ++k) {
            const size_t s = std::lower_bound(states.begin(), states.end(), cp[k].st) - states.begin();
            slot[k] = rows[s].size();
            rows[s].push_back(cp[k].row);
        }
    std::vector<std::vector<float>> sc(states.size());
    for (int32_t b = 0; b < mg->B; ++b) {
        if (mg->q[b].failed) continue;
        for (size_t s = 0; s < states.size(); ++s) {
            sc[s].resize(rows[s].size());
            EAHR_TRY(pvs_scores(states[s], b, rows[s].data(), static_cast<int64_t>(rows[s].size()),
                                sc[s].data()));
        }
        auto score_of = [&](size_t k) {
            const size_t s = std::lower_bound(states.begin(), states.end(), cp[k].st) - states.begin();
            return sc[s][slot[k]];
        };
        for (const auto& r : runs) {
            const float s0 = score_of(r.first);
            for (size_t k = r.first + 1; k < r.second; ++k)
                if (!(score_of(k) == s0)) mg->q[b].failed = true;
        }
    }
    return EAHR_OK;
}

int merge_next_items(pvs_merge* mg, int32_t m, const uint8_t* active, std::vector<std::vector<Item>>& out,
                     std::vector<int32_t>& status);

// Refill the empty buffers of source s for the queries in `need` (flags).
int refill(pvs_merge* mg, size_t s, const std::vector<uint8_t>& need, int32_t chunk) {
    auto& S = mg->src[s];
    const int32_t B = mg->B;
    if (S.st) {
        std::vector<int64_t> ids(static_cast<size_t>(B) * chunk);
        std::vector<float> sc(static_cast<size_t>(B) * chunk);
        std::vector<int32_t> cnt(B, 0), stt(B, EAHR_LIST_OPEN);
        EAHR_TRY(pvs_next(S.st, chunk, need.data(), ids.data(), sc.data(), cnt.data(), stt.data()));
        for (int32_t b = 0; b < B; ++b) {
            if (!need[b]) continue;
            auto& bf = S.buf[b];
            bf.clear();
            S.pos[b] = 0;
            for (int32_t j = 0; j < cnt[b]; ++j) {
                const int64_t row = ids[static_cast<size_t>(b) * chunk + j];
                if (row < 0 || row >= static_cast<int64_t>(S.gid.size()))
                    EAHR_FAIL(EAHR_E_INVALID, "pvs_merge: a segment emitted a row outside its id map");
                bf.push_back(Item{S.gid[row], sc[static_cast<size_t>(b) * chunk + j],
                                  S.version.empty() ? 0 : S.version[row]});
            }
            S.status[b] = stt[b];
        }
    } else {
        std::vector<std::vector<Item>> items(B);
        std::vector<int32_t> stt(B, EAHR_LIST_OPEN);
        EAHR_TRY(merge_next_items(S.child, chunk, need.data(), items, stt));
        for (int32_t b = 0; b < B; ++b) {
            if (!need[b]) continue;
            S.buf[b].swap(items[b]);
            S.pos[b] = 0;
            S.status[b] = stt[b];
        }
    }
    return EAHR_OK;
}

// Up to m next merged ranks of every active query into out[b]; status[b]
// as pvs_next.
int merge_next_items(pvs_merge* mg, int32_t m, const uint8_t* active, std::vector<std::vector<Item>>& out,
                     std::vector<int32_t>& status) {
    const int32_t B = mg->B;
    const size_t ns = mg->src.size();
    // ranks read from a source per refill: at least the request, within
    // 2^24 buffered entries per call over the batch
    const int32_t chunk = std::max<int32_t>(
        256, std::min<int32_t>(std::min<int32_t>(m, 1 << 20), static_cast<int32_t>((1 << 24) / std::max(B, 1))));
    std::vector<uint8_t> want(B, 0);
    for (int32_t b = 0; b < B; ++b) {
        out[b].clear();
        want[b] = (!active || active[b]) && !mg->q[b].failed && m > 0;
    }
    for (int guard = 0;; ++guard) {
        if (guard > (1 << 24)) EAHR_FAIL(EAHR_E_INVALID, "pvs_merge: merge did not converge");
        // sources whose head is missing for a query that still wants ranks
        for (size_t s = 0; s < ns; ++s) {
            auto& S = mg->src[s];
            std::vector<uint8_t> need(B, 0);
            bool some = false;
            for (int32_t b = 0; b < B; ++b) {
                if (!want[b] || mg->q[b].failed) continue;
                if (S.status[b] == EAHR_LIST_FAILED) {
                    mg->q[b].failed = true;
                    continue;
                }
                if (S.pos[b] >= S.buf[b].size() && S.status[b] == EAHR_LIST_OPEN) {
                    need[b] = 1;
                    some = true;
                }
            }
            if (some) {
                EAHR_TRY(refill(mg, s, need, chunk));
                for (int32_t b = 0; b < B; ++b)
                    if (need[b] && S.status[b] == EAHR_LIST_FAILED) mg->q[b].failed = true;
            }
        }
        // merge while every Open source has a head
        bool progress_needed = false;
        for (int32_t b = 0; b < B; ++b) {
            auto& Q = mg->q[b];
            if (!want[b] || Q.failed) continue;
            while (static_cast<int32_t>(out[b].size()) < m) {
                int best = -1;
                bool blocked = false;
                for (size_t s = 0; s < ns; ++s) {
                    const auto& S = mg->src[s];
                    if (S.pos[b] < S.buf[b].size()) {
                        const Item& h = S.buf[b][S.pos[b]];
                        if (best < 0 || precedes(h, mg->src[best].buf[b][mg->src[best].pos[b]]))
                            best = static_cast<int>(s);
                    } else if (S.status[b] == EAHR_LIST_OPEN) {
                        blocked = true;   // this source's next rank is unknown
                    }
                }
                if (blocked || best < 0) break;
                auto& S = mg->src[best];
                const Item it = S.buf[b][S.pos[b]++];
                if (Q.has_last && !precedes(Q.last, it) &&
                    !(it.id == Q.last.id && it.score == Q.last.score)) {
                    Q.failed = true;   // a source broke the (score, id) order
                    break;
                }
                if (mg->shared.count(it.id)) {
                    auto f = Q.seen.find(it.id);
                    if (f != Q.seen.end()) {
                        if (f->second.score == it.score && f->second.version == it.version) continue;
                        Q.failed = true;   // two copies disagree (score or version)
                        break;
                    }
                    Q.seen.emplace(it.id, it);
                }
                Q.last = it;
                Q.has_last = true;
                out[b].push_back(it);
                Q.emitted += 1;
            }
            if (Q.failed) continue;
            if (static_cast<int32_t>(out[b].size()) < m) {
                bool open_left = false;
                for (size_t s = 0; s < ns; ++s) {
                    const auto& S = mg->src[s];
                    if (S.pos[b] < S.buf[b].size() || S.status[b] == EAHR_LIST_OPEN) open_left = true;
                }
                if (open_left) progress_needed = true;
            }
        }
        if (!progress_needed) break;
    }
    for (int32_t b = 0; b < B; ++b) {
        if (active && !active[b]) continue;
        auto& Q = mg->q[b];
        if (Q.failed) {
            out[b].clear();
            status[b] = EAHR_LIST_FAILED;
            continue;
        }
        bool left = false;
        for (size_t s = 0; s < ns; ++s) {
            const auto& S = mg->src[s];
            if (S.pos[b] < S.buf[b].size() || S.status[b] == EAHR_LIST_OPEN) left = true;
        }
        status[b] = left ? EAHR_LIST_OPEN : EAHR_LIST_EXHAUSTED;
    }
    return EAHR_OK;
}

void init_sources(pvs_merge* mg) {
    for (auto& S : mg->src) {
        S.buf.assign(mg->B, {});
        S.pos.assign(mg->B, 0);
        S.status.assign(mg->B, EAHR_LIST_OPEN);
    }
    mg->q.assign(mg->B, pvs_merge::Query{});
}

}  // namespace

extern "C" int pvs_merge_open(const pvs_index* const* segs, const int64_t* epochs,
                              const int64_t* const* gids, const int64_t* const* versions,
                              int32_t n_segs, const float* q, int32_t B, int32_t ptr_kind,
                              pvs_merge** out) {
    if (!out) EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_open: out is NULL");
    *out = nullptr;
    if (!segs || !gids || n_segs <= 0 || B <= 0 || !q)
        EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_open: bad arguments");
    std::unique_ptr<pvs_merge> mg(new (std::nothrow) pvs_merge());
    if (!mg) EAHR_FAIL(EAHR_E_OOM, "pvs_merge_open: host allocation");
    mg->B = B;
    mg->src.resize(n_segs);
    for (int32_t s = 0; s < n_segs; ++s) {
        if (!segs[s] || !gids[s]) EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_open: segment %d is NULL", s);
        int64_t rows = 0, vis = 0;
        int32_t d = 0;
        EAHR_TRY(pvs_info(segs[s], 0, &rows, &d, &vis));
        const int64_t e = epochs ? epochs[s] : 0;
        int64_t erows = 0;
        EAHR_TRY(pvs_info(segs[s], e, &erows, &d, &vis));
        auto& S = mg->src[s];
        S.gid.assign(gids[s], gids[s] + erows);
        for (int64_t r = 0; r < erows; ++r) {
            if (S.gid[r] < 0 || S.gid[r] >= (1LL << 31) - 1)
                EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_open: global id outside [0, 2^31 - 1)");
            if (r > 0 && S.gid[r] <= S.gid[r - 1])
                EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_open: segment %d ids not strictly ascending", s);
        }
        if (versions && versions[s]) S.version.assign(versions[s], versions[s] + erows);
    }
    init_sources(mg.get());
    for (int32_t s = 0; s < n_segs; ++s)
        EAHR_TRY(pvs_open_gen(segs[s], epochs ? epochs[s] : 0, q, B, ptr_kind, EAHR_GEN_INTERVALS,
                              &mg->src[s].st));
    // the visible rows of every Segment's snapshot
    for (int32_t s = 0; s < n_segs; ++s) {
        const auto& S = mg->src[s];
        const auto& sn = segs[s]->snaps[epochs ? epochs[s] : 0];
        std::vector<uint64_t> vis(static_cast<size_t>(std::max<int64_t>(1, (sn.rows + 63) / 64)));
        HIP_TRY(hipMemcpy(vis.data(), sn.vis, vis.size() * sizeof(uint64_t), hipMemcpyDeviceToHost));
        for (int64_t r = 0; r < sn.rows; ++r)
            if ((vis[r >> 6] >> (r & 63)) & 1ull)
                mg->copies.push_back(Copy{S.gid[r], S.st, r, S.version.empty() ? 0 : S.version[r]});
    }
    EAHR_TRY(find_conflicts(mg.get()));
    *out = mg.release();
    return EAHR_OK;
}

extern "C" int pvs_merge_shards(pvs_merge** shards, int32_t n_shards, pvs_merge** out) {
    if (!out) EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_shards: out is NULL");
    *out = nullptr;
    if (!shards || n_shards <= 0) EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_shards: bad arguments");
    const int32_t B = shards[0] ? shards[0]->B : 0;
    for (int32_t s = 0; s < n_shards; ++s) {
        if (!shards[s] || shards[s]->B != B)
            EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_shards: shard %d missing or of another batch size", s);
        for (int32_t t = 0; t < s; ++t)
            if (shards[t] == shards[s]) EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_shards: shard %d repeated", s);
        for (int32_t b = 0; b < B; ++b)
            if (shards[s]->q[b].emitted > 0)
                EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_shards: shard %d was already read", s);
    }
    std::unique_ptr<pvs_merge> mg(new (std::nothrow) pvs_merge());
    if (!mg) EAHR_FAIL(EAHR_E_OOM, "pvs_merge_shards: host allocation");
    mg->B = B;
    mg->src.resize(n_shards);
    for (int32_t s = 0; s < n_shards; ++s) mg->src[s].child = shards[s];
    init_sources(mg.get());
    // copies across Shards (each Shard has already compared its own)
    for (int32_t s = 0; s < n_shards; ++s) {
        const auto& c = shards[s]->copies;
        mg->copies.insert(mg->copies.end(), c.begin(), c.end());
    }
    EAHR_TRY(find_conflicts(mg.get()));
    for (int32_t s = 0; s < n_shards; ++s) std::vector<Copy>().swap(shards[s]->copies);
    mg->owns_children = true;   // the shards now belong to the request-level merge
    *out = mg.release();
    return EAHR_OK;
}

extern "C" int pvs_merge_next(pvs_merge* mg, int32_t m, const uint8_t* active, int64_t* ids,
                              float* scores, int32_t* count, int32_t* status) {
    if (!mg || m < 0 || (m > 0 && (!ids || !scores)) || !count || !status)
        EAHR_FAIL(EAHR_E_INVALID, "pvs_merge_next: bad arguments");
    const int32_t B = mg->B;
    std::vector<std::vector<Item>> items(B);
    std::vector<int32_t> stt(B, EAHR_LIST_OPEN);
    EAHR_TRY(merge_next_items(mg, m, active, items, stt));
    for (int32_t b = 0; b < B; ++b) {
        if (active && !active[b]) continue;
        const auto& it = items[b];
        for (size_t j = 0; j < it.size(); ++j) {
            ids[static_cast<int64_t>(b) * m + static_cast<int64_t>(j)] = it[j].id;
            scores[static_cast<int64_t>(b) * m + static_cast<int64_t>(j)] = it[j].score;
        }
        count[b] = static_cast<int32_t>(it.size());
        status[b] = stt[b];
    }
    return EAHR_OK;
}

extern "C" void pvs_merge_close(pvs_merge* mg) { delete mg; }

int32_t eahr_merge_batch(const pvs_merge* mg) { return mg ? mg->B : 0; }

bool eahr_merge_unread(const pvs_merge* mg) {
    if (!mg) return false;
    for (const auto& q : mg->q)
        if (q.emitted > 0) return false;
    return true;
}
