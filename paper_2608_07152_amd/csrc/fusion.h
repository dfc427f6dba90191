// Certification core of exact adaptive weighted-RRF fusion (Sec. 2.1, 2.2).
//
// g_i(r) = 1 / (r / w_i + k - 1) = w_i / (r + w_i (k - 1)) with integer k and
// w_i, so every bound is a sum of at most two unit terms w / D and compares
// exactly as a fraction (numerators < 2^43, denominators < 2^64, products
// < 2^107 in unsigned 128-bit integers).
//
// After every depth round the remaining observed items fall into three
// groups: seen by both lists (L = U = F), seen by the dense list only
// (L = g_d(r_d), U = L + u_s), seen by the sparse list only.  Inside a
// single-list group L and U strictly decrease with the rank, so the group's
// best L and best U belong to its first unfixed member; the both-seen group
// is a binary heap on (F desc, id asc), whose best two items are the root and
// the better child.  x_dag and its strongest competitor y are therefore among
// at most six items, and each position is decided as in Sec. 2.2:
// (L(x_dag), x_dag) must precede (U(y), y) for every other remaining y, and
// L(x_dag) > B strictly.
//
// A fixing takes the best of the items it compares, so with |A| positions
// fixed only the best K - |A| + 1 both-seen items can still be fixed or be
// the strongest rival of a fixed one (an item behind them stays third or
// later until the K-th position is fixed).  The heap keeps those; the rest
// are dropped when found, against a cutoff item with at least that many kept
// items at or before it.
//
// Bookkeeping without per-item hashing: each list keeps its prefix sorted by
// id, so the ranks of a round are radix-sorted and merge-joined against the
// other list to find items seen by both; a bitmap of live positions per list
// skips items that became both-seen or fixed a word at a time.  Ids must lie
// in [0, 2^31) and be distinct inside a list (a repeat sets dup).
//
// Once one list is closed (read to its end) nothing joins against the other
// list's id order any more: appends to the open list then test membership in
// the closed list with a bitmap over ids (and look up the rank in its id
// order only for the items it holds), and repeats with a second bitmap.
//
// Once the lists together hold at least 1/16 of the id range [0, universe)
// (when the caller knows it) while both are open, both lists switch to direct
// rank arrays indexed by id: an append then costs O(ranks appended) whatever
// the depth, where a merge into the id order costs O(depth).  This keeps
// schedules that append few ranks at a time to deep lists (checks every 16
// ranks, the frozen scheduler) linear in the depth reached.  A list appended
// after the other closed stays with the bitmaps, which are also linear and
// touch a bit per id instead of two rank arrays of 4 bytes per id.
//
// A long append (either kind) is split over `threads` host threads: the sort
// by id digit by digit, the joins and merges over ranges of ids (equal ids
// fall into one range), bits cleared atomically; the both-seen items are
// collected per range, and the heap order does not depend on their insertion
// order because (F, id) is a total order.
#pragma once
#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <memory>
#include <utility>
#include <vector>

#include "host_parallel.h"

namespace eahr {

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

// Ascending sort of (id << 32 | rank) keys by id (ids < 2^31): least-
// significant-digit radix sort on the id bytes (256 scatter targets stay in
// cache; 12-bit digits, one pass fewer for ids below 2^24, measured slower),
// skipping bytes equal in every id; short runs use a comparison sort.
inline void sort_by_id(std::vector<uint64_t>& a, std::vector<uint64_t>& tmp) {
    const size_t n = a.size();
    if (n < 1024) {
        std::sort(a.begin(), a.end());
        return;
    }
    tmp.resize(n);
    uint32_t cnt[4][256] = {};
    for (size_t i = 0; i < n; ++i) {
        const uint32_t id = static_cast<uint32_t>(a[i] >> 32);
        ++cnt[0][id & 0xff];
        ++cnt[1][(id >> 8) & 0xff];
        ++cnt[2][(id >> 16) & 0xff];
        ++cnt[3][id >> 24];
    }
    for (int d = 0; d < 4; ++d) {
        const int shift = 32 + 8 * d;
        uint32_t* c = cnt[d];
        if (c[(a[0] >> shift) & 0xff] == n) continue;   // one digit value
        uint32_t sum = 0;
        for (int v = 0; v < 256; ++v) {
            const uint32_t t = c[v];
            c[v] = sum;
            sum += t;
        }
        for (size_t i = 0; i < n; ++i) tmp[c[(a[i] >> shift) & 0xff]++] = a[i];
        a.swap(tmp);
    }
}

// sort_by_id over `parts` host threads: per digit, each part counts its
// slice, then scatters it (stable) at offsets ordered by (digit, part).
inline void sort_by_id_parallel(std::vector<uint64_t>& a, std::vector<uint64_t>& tmp, int parts) {
    const size_t n = a.size();
    tmp.resize(n);
    std::vector<uint32_t> cnt(static_cast<size_t>(parts) * 256);
    for (int d = 0; d < 4; ++d) {
        const int shift = 32 + 8 * d;
        std::fill(cnt.begin(), cnt.end(), 0u);
        parallel_for(parts, parts, [&](int64_t t) {
            uint32_t* c = cnt.data() + t * 256;
            for (size_t i = n * t / parts, e = n * (t + 1) / parts; i < e; ++i) ++c[(a[i] >> shift) & 0xff];
        });
        uint32_t sum = 0;
        bool one = false;
        for (int v = 0; v < 256; ++v) {
            uint32_t tot = 0;
            for (int t = 0; t < parts; ++t) {
                const uint32_t c = cnt[t * 256 + v];
                cnt[t * 256 + v] = sum + tot;
                tot += c;
            }
            one |= tot == n;
            sum += tot;
        }
        if (one) continue;   // one digit value
        parallel_for(parts, parts, [&](int64_t t) {
            uint32_t* c = cnt.data() + t * 256;
            for (size_t i = n * t / parts, e = n * (t + 1) / parts; i < e; ++i) tmp[c[(a[i] >> shift) & 0xff]++] = a[i];
        });
        a.swap(tmp);
    }
}

// A both-seen item: its ranks define F exactly; f is F in float64 (relative
// error below 2^-50), used to order items whose values are far apart.
struct Scored {
    double f;
    int32_t r0, r1;
    int64_t id;
};

inline Frac exact_F(const Params& P, const Scored& s) {
    return add(g(P, 0, s.r0), g(P, 1, s.r1));
}

// heap order: a below b when b precedes a (exact; float64 decides only when
// the two values differ by more than 1e-12 relative)
struct HeapLess {
    const Params* P;
    bool operator()(const Scored& a, const Scored& b) const {
        const double d = b.f - a.f, m = (a.f > b.f ? a.f : b.f) * 1e-12;
        if (d > m) return true;
        if (d < -m) return false;
        const int c = cmp(exact_F(*P, b), exact_F(*P, a));
        return c > 0 || (c == 0 && b.id < a.id);
    }
};

inline double g_double(const Params& P, int i, int64_t r) {
    if (P.w[i] == 0) return 0.0;
    return static_cast<double>(P.w[i]) / static_cast<double>(r + P.w[i] * (P.k - 1));
}

struct Fusion {
    struct List {
        std::vector<int64_t, NoInit<int64_t>> ids;   // exact prefix read so far
        std::vector<uint64_t> by_id;   // (id << 32 | rank), ascending id
        std::vector<uint64_t> alive;   // bit p: position p is an unfixed single-list item
        bool open = true;
        int64_t cursor = 0;

        // first live position at or after p (size() if none)
        int64_t find(int64_t p) const {
            const int64_t n = size();
            if (p >= n) return n;
            size_t w = static_cast<size_t>(p >> 6);
            uint64_t bits = alive[w] & (~0ull << (p & 63));
            while (!bits) {
                if (++w >= alive.size()) return n;
                bits = alive[w];
            }
            const int64_t q = static_cast<int64_t>(w * 64 + __builtin_ctzll(bits));
            return q < n ? q : n;
        }
        void kill(int64_t p) { alive[p >> 6] &= ~(1ull << (p & 63)); }
        void grow(int64_t n_new) {   // new positions start live
            const int64_t p0 = size(), p1 = p0 + n_new;
            alive.resize(static_cast<size_t>((p1 + 63) >> 6), 0);
            int64_t p = p0;
            for (; p < p1 && (p & 63); ++p) alive[p >> 6] |= 1ull << (p & 63);
            for (; p + 64 <= p1; p += 64) alive[p >> 6] = ~0ull;
            for (; p < p1; ++p) alive[p >> 6] |= 1ull << (p & 63);
        }
        int64_t size() const { return static_cast<int64_t>(ids.size()); }
    };

    // appends of at least this many ranks are split over up to `threads`
    // host threads
    static constexpr int64_t kParallelAppend = int64_t(1) << 16;

    const Params* P = nullptr;
    int threads = 1;
    List L[2];
    std::vector<Scored> both;   // binary heap of the best unfixed both-seen items
    std::vector<Scored> fresh;  // both-seen items of a one-part append
    std::vector<int64_t> A;     // fixed prefix
    bool resolved = false;
    bool dup = false;           // an id repeated inside one list
    std::vector<uint64_t> batch, tmp, merged;
    // closed-list mode: seen[i] has bit x set when list i holds id x; for
    // the closed list c = cum_list, cum[w] counts its ids below word w, so an
    // id's position in c's id order is cum[w] plus the set bits below it in
    // word w (a rank costs two reads instead of a binary search)
    bool bitmaps = false;
    std::vector<uint64_t> seen[2];
    std::vector<uint32_t> cum;
    int cum_list = -1;
    // direct mode: pos[2 x + i] is the 1-based rank of id x in list i (0:
    // not in it; both ranks of an id share a cache line); entered once the
    // lists hold universe / kDirectShare ranks
    static constexpr int64_t kDirectShare = 16;
    int64_t universe = 0;       // ids lie in [0, universe); 0: not known
    bool direct = false;
    std::vector<int32_t> pos;

    static bool test_bit(const std::vector<uint64_t>& b, int64_t x) {
        const size_t w = static_cast<size_t>(x >> 6);
        return w < b.size() && ((b[w] >> (x & 63)) & 1ull);
    }
    // sets bit x, returns whether it was already set
    static bool set_bit(std::vector<uint64_t>& b, int64_t x) {
        const size_t w = static_cast<size_t>(x >> 6);
        if (w >= b.size()) b.resize(std::max(w + 1, b.size() * 2), 0);
        const uint64_t m = 1ull << (x & 63);
        const bool had = (b[w] & m) != 0;
        b[w] |= m;
        return had;
    }
    void enter_bitmap_mode() {
        for (int i = 0; i < 2; ++i)
            for (int64_t x : L[i].ids) set_bit(seen[i], x);
        bitmaps = true;
    }
    // rank (1-based) of id x in list i, from its id order; x must be in it
    int64_t rank_of(int i, int64_t x) const {
        const auto& v = L[i].by_id;
        if (cum_list == i) {
            const size_t w = static_cast<size_t>(x >> 6);
            const uint64_t below = seen[i][w] & ((1ull << (x & 63)) - 1);
            return static_cast<int64_t>(v[cum[w] + static_cast<uint32_t>(__builtin_popcountll(below))] & 0xffffffffu);
        }
        const uint64_t key = static_cast<uint64_t>(x) << 32;
        const auto it = std::lower_bound(v.begin(), v.end(), key);
        return static_cast<int64_t>(*it & 0xffffffffu);
    }
    // prefix counts of closed list c's id bitmap (its id order is complete:
    // every rank it holds was merged in while the other list was open)
    void count_closed(int c) {
        const auto& b = seen[c];
        cum.resize(b.size() + 1);
        cum[0] = 0;
        for (size_t w = 0; w < b.size(); ++w) cum[w + 1] = cum[w] + static_cast<uint32_t>(__builtin_popcountll(b[w]));
        cum_list = c;
    }

    bool fixed(int64_t x) const { return std::find(A.begin(), A.end(), x) != A.end(); }

    // (F, id) order: a before b
    bool better(const Scored& a, const Scored& b) const { return HeapLess{P}(b, a); }
    // how many of the best both-seen items can still matter (at least 1)
    size_t keep() const {
        const int64_t m = P->K - static_cast<int64_t>(A.size()) + 1;
        return static_cast<size_t>(m < 1 ? 1 : m);
    }
    // An item that every kept item precedes or equals, with at least keep()
    // items at or before it; items behind it are never kept.
    struct Cut {
        Scored s{};
        bool on = false;
    };
    Cut cut;
    // Collector of the both-seen items of one part of an append: drops items
    // behind its cutoff and, once it holds many, keeps only its best m (its
    // m-th best becoming its cutoff), so a part stores O(m) items.
    struct Sink {
        std::vector<Scored>* out;
        Cut cut;
        size_t m;
    };
    Sink sink(std::vector<Scored>& out) const { return Sink{&out, cut, keep()}; }
    void prune(std::vector<Scored>& v, size_t m, Cut& c) const {
        std::nth_element(v.begin(), v.begin() + static_cast<std::ptrdiff_t>(m - 1), v.end(),
                         [this](const Scored& a, const Scored& b) { return better(a, b); });
        v.resize(m);
        c.s = v[m - 1];
        c.on = true;
    }
    static size_t prune_at(size_t m) { return m > (SIZE_MAX - 64) / 2 ? SIZE_MAX : 2 * m + 64; }
    void offer(Sink& k, const Scored& x) const {
        if (k.cut.on && !better(x, k.cut.s)) return;
        k.out->push_back(x);
        if (k.out->size() >= prune_at(k.m)) prune(*k.out, k.m, k.cut);
    }

    // Back to an empty fusion with both lists open, keeping the memory.
    void reset() {
        for (auto& l : L) {
            l.ids.clear();
            l.by_id.clear();
            l.alive.clear();
            l.open = true;
            l.cursor = 0;
        }
        both.clear();
        cut = Cut{};
        A.clear();
        resolved = false;
        dup = false;
        bitmaps = false;
        for (auto& b : seen) std::fill(b.begin(), b.end(), 0ull);
        cum_list = -1;
        direct = false;
        universe = 0;
        std::vector<int32_t>().swap(pos);   // only deep queries need it
    }

    void enter_direct_mode() {
        for (int i = 0; i < 2; ++i)
            for (int64_t x : L[i].ids) universe = std::max(universe, x + 1);
        pos.assign(2 * static_cast<size_t>(universe), 0);
        for (int i = 0; i < 2; ++i) {
            for (int64_t p = 0; p < L[i].size(); ++p) {
                int32_t& r = pos[2 * static_cast<size_t>(L[i].ids[p]) + i];
                if (r) dup = true;
                else r = static_cast<int32_t>(p + 1);
            }
        }
        direct = true;
    }

    // Ranks p0 + j + 1 (j in [j0, j1)) of list i in direct mode: repeats set
    // the flag, both-seen items go to out.  Atomic updates when parts of one
    // append run concurrently (the other list is not written meanwhile).
    template <bool Atomic>
    void direct_part(int i, const int64_t* ids, int64_t p0, int64_t j0, int64_t j1,
                     Sink& out, bool& rep) {
        List& me = L[i];
        List& other = L[1 - i];
        auto clear_bit = [](std::vector<uint64_t>& b, int64_t p) {
            const uint64_t m = ~(1ull << (p & 63));
            if (Atomic) __atomic_fetch_and(&b[static_cast<size_t>(p >> 6)], m, __ATOMIC_RELAXED);
            else b[static_cast<size_t>(p >> 6)] &= m;
        };
        int32_t* const ranks = pos.data();
        // the rank pairs are read at random ids: fetch a few ids ahead
        constexpr int64_t kAhead = 16;
        for (int64_t j = j0; j < j1; ++j) {
            if (j + kAhead < j1) __builtin_prefetch(ranks + 2 * ids[j + kAhead], 1, 0);
            const int64_t x = ids[j];
            const int64_t rank = p0 + j + 1;
            int32_t* const mine = ranks + 2 * x + i;
            int32_t prev;
            if (Atomic) {
                prev = __atomic_exchange_n(mine, static_cast<int32_t>(rank), __ATOMIC_RELAXED);
            } else {
                prev = *mine;
                if (!prev) *mine = static_cast<int32_t>(rank);
            }
            if (prev) {
                rep = true;
                clear_bit(me.alive, rank - 1);
                continue;
            }
            const int64_t ro = ranks[2 * x + 1 - i];
            if (!ro) continue;
            clear_bit(me.alive, rank - 1);
            clear_bit(other.alive, ro - 1);
            if (!fixed(x)) {
                const int64_t r0 = (i == 0) ? rank : ro, r1 = (i == 0) ? ro : rank;
                offer(out, Scored{g_double(*P, 0, r0) + g_double(*P, 1, r1),
                                 static_cast<int32_t>(r0), static_cast<int32_t>(r1), x});
            }
        }
    }

    void append_direct(int i, const int64_t* ids, int64_t n) {
        List& me = L[i];
        const int64_t p0 = me.size();
        me.grow(n);
        me.ids.insert(me.ids.end(), ids, ids + n);
        int64_t xmax = -1;
        for (int64_t j = 0; j < n; ++j) xmax = std::max(xmax, ids[j]);
        if (xmax >= universe) {   // an id beyond the announced range
            universe = xmax + 1;
            pos.resize(2 * static_cast<size_t>(universe), 0);
        }
        const size_t heap0 = both.size();
        const int parts = (threads > 1 && n >= kParallelAppend)
                        ? static_cast<int>(std::min<int64_t>(threads, n / (kParallelAppend / 4)))
                        : 1;
        if (parts <= 1) {
            bool rep = false;
            fresh.clear();
            Sink k = sink(fresh);
            direct_part<false>(i, ids, p0, 0, n, k, rep);
            dup |= rep;
            both.insert(both.end(), fresh.begin(), fresh.end());
        } else {
            std::vector<std::vector<Scored>> found(static_cast<size_t>(parts));
            std::vector<uint8_t> rep(static_cast<size_t>(parts), 0);
            parallel_for(parts, parts, [&](int64_t t) {
                bool r = false;
                Sink k = sink(found[t]);
                direct_part<true>(i, ids, p0, n * t / parts, n * (t + 1) / parts, k, r);
                rep[t] = r;
            });
            for (int t = 0; t < parts; ++t) {
                dup |= rep[t] != 0;
                both.insert(both.end(), found[t].begin(), found[t].end());
            }
        }
        restore_heap(heap0);
    }

    // Heap order after items were pushed behind position heap0: one push per
    // new item, or a linear rebuild when many were added.
    void restore_heap(size_t heap0) {
        const size_t m = keep();
        if (both.size() >= prune_at(m)) {
            prune(both, m, cut);
            std::make_heap(both.begin(), both.end(), HeapLess{P});
            return;
        }
        const size_t added = both.size() - heap0;
        if (added > heap0 / 8) {
            std::make_heap(both.begin(), both.end(), HeapLess{P});
        } else {
            for (size_t k = heap0 + 1; k <= both.size(); ++k)
                std::push_heap(both.begin(), both.begin() + k, HeapLess{P});
        }
    }

    // Append n ranks to list i (ids must be new to the list, else dup is set
    // and the bookkeeping is no longer meaningful).
    void append(int i, const int64_t* ids, int64_t n) {
        if (n <= 0) return;
        // (with the other list closed the bitmaps already cost O(n) per append)
        if (!direct && L[1 - i].open && universe > 0 &&
            (L[0].size() + L[1].size() + n) * kDirectShare >= universe)
            enter_direct_mode();
        if (direct) {
            append_direct(i, ids, n);
            return;
        }
        if (!L[1 - i].open) {
            append_closed_other(i, ids, n);
            return;
        }
        List& me = L[i];
        List& other = L[1 - i];
        const int64_t p0 = me.size();
        me.grow(n);
        me.ids.insert(me.ids.end(), ids, ids + n);
        batch.resize(static_cast<size_t>(n));
        for (int64_t j = 0; j < n; ++j)
            batch[j] = (static_cast<uint64_t>(ids[j]) << 32) | static_cast<uint64_t>(p0 + j + 1);
        const int parts = (threads > 1 && n >= kParallelAppend)
                        ? static_cast<int>(std::min<int64_t>(threads, n / (kParallelAppend / 4)))
                        : 1;
        if (parts > 1) sort_by_id_parallel(batch, tmp, parts);
        else sort_by_id(batch, tmp);
        // Parts of the id range: part t holds the ids from splitter t on (the
        // id of batch[n t / parts]) in the batch, the other list's id order
        // and this list's id order alike, so equal ids meet inside one part.
        const auto& ob = other.by_id;
        std::vector<size_t> sa(parts + 1), sb(parts + 1), sm(parts + 1);
        sa[0] = sb[0] = sm[0] = 0;
        sa[parts] = batch.size();
        sb[parts] = ob.size();
        sm[parts] = me.by_id.size();
        for (int t = 1; t < parts; ++t) {
            const uint64_t key = batch[static_cast<size_t>(n) * t / parts] & ~0xffffffffull;
            sa[t] = std::lower_bound(batch.begin(), batch.end(), key) - batch.begin();
            sb[t] = std::lower_bound(ob.begin(), ob.end(), key) - ob.begin();
            sm[t] = std::lower_bound(me.by_id.begin(), me.by_id.end(), key) - me.by_id.begin();
        }
        // merge-join with the other list: items now seen by both
        const size_t heap0 = both.size();
        std::vector<std::vector<Scored>> found(parts > 1 ? parts : 0);
        auto join = [&](size_t a, size_t ae, size_t b, size_t be, std::vector<Scored>& items, bool atomic) {
            Sink out = sink(items);
            // ids interleave at random: the advance is branch-free, only a
            // match (rarer) branches
            while (a < ae && b < be) {
                const uint64_t xa = batch[a] >> 32, xb = ob[b] >> 32;
                if (xa != xb) {
                    a += xa < xb;
                    b += xb < xa;
                } else {
                    const int64_t ri = static_cast<int64_t>(batch[a] & 0xffffffffu);
                    const int64_t rj = static_cast<int64_t>(ob[b] & 0xffffffffu);
                    if (atomic) {
                        __atomic_fetch_and(&me.alive[(ri - 1) >> 6], ~(1ull << ((ri - 1) & 63)), __ATOMIC_RELAXED);
                        __atomic_fetch_and(&other.alive[(rj - 1) >> 6], ~(1ull << ((rj - 1) & 63)), __ATOMIC_RELAXED);
                    } else {
                        me.kill(ri - 1);
                        other.kill(rj - 1);
                    }
                    const int64_t x = static_cast<int64_t>(xa);
                    if (!fixed(x)) {
                        const int64_t r0 = (i == 0) ? ri : rj, r1 = (i == 0) ? rj : ri;
                        offer(out, Scored{g_double(*P, 0, r0) + g_double(*P, 1, r1),
                                         static_cast<int32_t>(r0), static_cast<int32_t>(r1), x});
                    }
                    ++a;
                    ++b;
                }
            }
        };
        // merge into the id order; a repeated id meets its twin here (or,
        // inside the batch, its neighbour)
        merged.resize(me.by_id.size() + batch.size());
        auto merge = [&](size_t x0, size_t x1, size_t y0, size_t y1) -> bool {
            bool eq = false;
            for (size_t k = y0 + 1; k < y1; ++k) eq |= (batch[k] >> 32) == (batch[k - 1] >> 32);
            const uint64_t* x = me.by_id.data() + x0;
            const uint64_t* xe = me.by_id.data() + x1;
            const uint64_t* y = batch.data() + y0;
            const uint64_t* ye = batch.data() + y1;
            uint64_t* out = merged.data() + x0 + y0;
            while (x < xe && y < ye) {   // branch-free: the order of x and y is random
                const uint64_t vx = *x, vy = *y;
                eq |= (vx >> 32) == (vy >> 32);
                const bool ty = vy < vx;
                *out++ = ty ? vy : vx;
                y += ty;
                x += !ty;
            }
            out = std::copy(x, xe, out);
            std::copy(y, ye, out);
            return eq;
        };
        if (parts == 1) {
            fresh.clear();
            join(0, batch.size(), 0, ob.size(), fresh, false);
            both.insert(both.end(), fresh.begin(), fresh.end());
            dup |= merge(0, me.by_id.size(), 0, batch.size());
        } else {
            std::vector<uint8_t> eq(parts, 0);
            parallel_for(parts, parts, [&](int64_t t) {
                join(sa[t], sa[t + 1], sb[t], sb[t + 1], found[t], true);
                eq[t] = merge(sm[t], sm[t + 1], sa[t], sa[t + 1]);
            });
            for (int t = 0; t < parts; ++t) {
                dup |= eq[t] != 0;
                both.insert(both.end(), found[t].begin(), found[t].end());
            }
        }
        me.by_id.swap(merged);
        restore_heap(heap0);
    }

    // Ranks p0 + j + 1 (j in [j0, j1)) of list i while the other list is
    // closed: repeats set the flag, both-seen items go to out.  Atomic bit
    // updates when parts of one append run concurrently.
    template <bool Atomic>
    void closed_part(int i, const int64_t* ids, int64_t p0, int64_t j0, int64_t j1,
                     Sink& out, bool& rep) {
        List& me = L[i];
        List& other = L[1 - i];
        auto clear_bit = [](std::vector<uint64_t>& b, int64_t p) {
            const uint64_t m = ~(1ull << (p & 63));
            if (Atomic) __atomic_fetch_and(&b[static_cast<size_t>(p >> 6)], m, __ATOMIC_RELAXED);
            else b[static_cast<size_t>(p >> 6)] &= m;
        };
        uint64_t* mine = seen[i].data();
        for (int64_t j = j0; j < j1; ++j) {
            const int64_t x = ids[j];
            const int64_t rank = p0 + j + 1;
            const uint64_t m = 1ull << (x & 63);
            const bool had = Atomic ? (__atomic_fetch_or(&mine[x >> 6], m, __ATOMIC_RELAXED) & m) != 0
                                    : (mine[x >> 6] & m) != 0;
            if (!Atomic) mine[x >> 6] |= m;
            if (had) {
                rep = true;
                clear_bit(me.alive, rank - 1);
                continue;
            }
            if (!test_bit(seen[1 - i], x)) continue;
            const int64_t ro = rank_of(1 - i, x);
            clear_bit(me.alive, rank - 1);
            clear_bit(other.alive, ro - 1);
            if (!fixed(x)) {
                const int64_t r0 = (i == 0) ? rank : ro, r1 = (i == 0) ? ro : rank;
                offer(out, Scored{g_double(*P, 0, r0) + g_double(*P, 1, r1),
                                 static_cast<int32_t>(r0), static_cast<int32_t>(r1), x});
            }
        }
    }

    // Append to list i while the other list is closed (see the file header).
    void append_closed_other(int i, const int64_t* ids, int64_t n) {
        if (!bitmaps) enter_bitmap_mode();
        if (cum_list != 1 - i) count_closed(1 - i);
        List& me = L[i];
        const int64_t p0 = me.size();
        me.grow(n);
        const size_t heap0 = both.size();
        const int parts = (threads > 1 && n >= kParallelAppend)
                        ? static_cast<int>(std::min<int64_t>(threads, n / (kParallelAppend / 4)))
                        : 1;
        // the ids join the list and give the largest id (in parts when long)
        me.ids.resize(static_cast<size_t>(p0 + n));
        std::vector<int64_t> part_max(static_cast<size_t>(parts), 0);
        parallel_for(parts, parts, [&](int64_t t) {
            int64_t m = 0;
            int64_t* dst = me.ids.data() + p0;
            for (int64_t j = n * t / parts, e = n * (t + 1) / parts; j < e; ++j) {
                dst[j] = ids[j];
                m = std::max(m, ids[j]);
            }
            part_max[t] = m;
        });
        const int64_t xmax = *std::max_element(part_max.begin(), part_max.end());
        const size_t words = static_cast<size_t>(xmax >> 6) + 1;
        if (seen[i].size() < words) seen[i].resize(std::max(words, seen[i].size() * 2), 0);
        if (parts <= 1) {
            bool rep = false;
            fresh.clear();
            Sink k = sink(fresh);
            closed_part<false>(i, ids, p0, 0, n, k, rep);
            dup |= rep;
            both.insert(both.end(), fresh.begin(), fresh.end());
        } else {
            std::vector<std::vector<Scored>> found(static_cast<size_t>(parts));
            std::vector<uint8_t> rep(static_cast<size_t>(parts), 0);
            parallel_for(parts, parts, [&](int64_t t) {
                bool r = false;
                Sink k = sink(found[t]);
                closed_part<true>(i, ids, p0, n * t / parts, n * (t + 1) / parts, k, r);
                rep[t] = r;
            });
            for (int t = 0; t < parts; ++t) {
                dup |= rep[t] != 0;
                both.insert(both.end(), found[t].begin(), found[t].end());
            }
        }
        restore_heap(heap0);
    }

    int64_t single_from(int i, int64_t p) {
        const int64_t q = L[i].find(p);
        return q < L[i].size() ? q : -1;
    }

    Frac u(int i) const {
        return L[i].open ? g(*P, i, L[i].size() + 1) : Frac{0, 1};
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
                const Frac F0 = exact_F(*P, both[0]);
                c[nc++] = Cand{both[0].id, F0, F0, 0, -1};
            }
            for (int i = 0; i < 2; ++i) {
                const int64_t p = single_from(i, L[i].cursor);
                if (p >= 0) {
                    L[i].cursor = p;
                    const Frac Li = g(*P, i, p + 1);
                    c[nc++] = Cand{L[i].ids[p], Li, add(Li, ui[1 - i]), 1 + i, p};
                } else {
                    L[i].cursor = L[i].size();
                }
            }
            if (nc == 0) break;
            int xd = 0;
            for (int j = 1; j < nc; ++j)
                if (precedes(c[j].L, c[j].id, c[xd].L, c[xd].id)) xd = j;
            const Cand X = c[xd];
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
                    if (n > 2 && HeapLess{P}(both[1], both[2])) second = 2;
                    if (second >= 0)
                        ok = precedes(X.L, X.id, exact_F(*P, both[second]), both[second].id);
                } else {
                    const int i = X.kind - 1;
                    const int64_t p = single_from(i, X.pos + 1);
                    if (p >= 0) {
                        const Frac Li = g(*P, i, p + 1);
                        ok = precedes(X.L, X.id, add(Li, ui[1 - i]), L[i].ids[p]);
                    }
                }
            }
            if (!ok) break;
            A.push_back(X.id);
            if (X.kind == 0) {
                std::pop_heap(both.begin(), both.end(), HeapLess{P});
                both.pop_back();
            } else {
                L[X.kind - 1].kill(X.pos);
            }
        }
        if (static_cast<int64_t>(A.size()) >= P->K) {
            resolved = true;
        } else if (B.num == 0 && both.empty() && single_from(0, L[0].cursor) < 0 &&
                   single_from(1, L[1].cursor) < 0) {
            resolved = true;   // nothing unseen or remaining can score: q_K = |A|
        }
    }
};

}  // namespace eahr
