// The paper's frozen fusion scheduler (Sec. 3.5), an alternative to depth
// doubling.  It changes how many ranks are read and when certification runs,
// never the result (Sec. 2.4).
//
// Rules (the paper's values for Top-K with K = 20, generalised through K):
//  * a scheduling step reads at most 16 ranks from one list;
//  * the list read is the one whose next unread rank has the larger maximum
//    weighted-RRF contribution g_i(d_i + 1) (equal: the dense list), except
//    that a list skipped for 16 consecutive steps is read next (fairness);
//  * certification is checked after every step while the cumulative access
//    d_0 + d_1 is at most 4K ranks (80 for K = 20), then after a further
//    a / 8 ranks of access, clamped to [64, 1024], where a is the access at
//    the previous check;
//  * reading the last rank of a list triggers a check at once.
// Only the depths matter to these rules, so the scheduler is simulated from
// one check to the next over ranks already read, and the fusion receives one
// append per list per check.
#pragma once
#include <algorithm>
#include <cstdint>

#include "fusion.h"

namespace eahr {

struct FrozenSchedule {
    static constexpr int64_t kStep = 16;     // ranks per step
    static constexpr int kFair = 16;         // consecutive skips that force a read
    static constexpr int64_t kMinGap = 64, kMaxGap = 1024;
    // ranks a list may need between two checks: the largest gap plus a step
    static constexpr int64_t kHorizon = kMaxGap + kStep;

    int64_t d[2] = {0, 0};   // ranks scheduled so far per list
    int skipped[2] = {0, 0};

    // g_0(d_0 + 1) > g_1(d_1 + 1)?  (exact, integer weights and k)
    static int cmp_next(const Params& P, const int64_t dd[2]) {
        return cmp(g(P, 0, dd[0] + 1), g(P, 1, dd[1] + 1));
    }

    // Advance to the next check.  avail[i]: ranks of list i read so far;
    // done[i]: list i has no rank beyond avail[i]; use[i]: list i takes part
    // (positive weight).  The caller guarantees avail[i] >= d[i] + kHorizon
    // unless done[i].  Returns false when no list has an unscheduled rank.
    bool advance(const Params& P, const int64_t avail[2], const bool done[2], const bool use[2]) {
        const int64_t a0 = d[0] + d[1];
        const int64_t every_step = 4 * P.K;
        const int64_t target = a0 + std::min(kMaxGap, std::max(kMinGap, a0 / 8));
        bool stepped = false;
        for (;;) {
            bool can[2];
            for (int i = 0; i < 2; ++i) can[i] = use[i] && d[i] < avail[i];
            if (!can[0] && !can[1]) return stepped;
            int pick;
            if (can[0] && can[1]) {
                pick = (cmp_next(P, d) >= 0) ? 0 : 1;
                if (skipped[1 - pick] >= kFair) pick = 1 - pick;
            } else {
                pick = can[0] ? 0 : 1;
            }
            const int64_t take = std::min(kStep, avail[pick] - d[pick]);
            d[pick] += take;
            skipped[pick] = 0;
            if (can[1 - pick]) skipped[1 - pick] += 1;
            stepped = true;
            if (done[pick] && d[pick] == avail[pick]) return true;   // list read to its end
            const int64_t a = d[0] + d[1];
            if (a0 < every_step || a <= every_step) return true;       // a check after every step
            if (a >= target) return true;
        }
    }
};

}  // namespace eahr
