// Drives the host fusion (fusion.h) the way eahr_topk does under depth
// doubling, with the id range unknown: appends go through the id-order
// merges while both lists are open and through the bitmaps once one list is
// closed, split over host threads when long.  Reads two int64 rankings from
// files, prints the fixed Top-K ids (or "dup" when a list repeats an id)
// and, on stderr, the depth read in each list.
//
//   fusion_modes <dense.bin> <sparse.bin> K k w_dense w_sparse threads
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "fusion.h"

static std::vector<int64_t> read_list(const char* path) {
    std::vector<int64_t> v;
    FILE* f = std::fopen(path, "rb");
    if (!f) return v;
    int64_t x;
    while (std::fread(&x, sizeof(x), 1, f) == 1) v.push_back(x);
    std::fclose(f);
    return v;
}

int main(int argc, char** argv) {
    if (argc != 8) return 2;
    const std::vector<int64_t> lists[2] = {read_list(argv[1]), read_list(argv[2])};
    const eahr::Params P{std::atoll(argv[3]), std::atoll(argv[4]), {std::atoll(argv[5]), std::atoll(argv[6])}};
    eahr::Fusion f;
    f.P = &P;
    f.threads = std::atoi(argv[7]);
    for (int i = 0; i < 2; ++i) f.L[i].open = P.w[i] > 0 && !lists[i].empty();
    for (int64_t depth = 20; !f.resolved; depth *= 2) {
        for (int i = 0; i < 2; ++i) {
            if (!f.L[i].open) continue;
            const int64_t have = f.L[i].size();
            const int64_t len = static_cast<int64_t>(lists[i].size());
            const int64_t upto = depth < len ? depth : len;
            if (upto > have) f.append(i, lists[i].data() + have, upto - have);
            if (f.L[i].size() == len) f.L[i].open = false;
        }
        if (f.dup) {
            std::printf("dup\n");
            return 0;
        }
        f.certify();
        if (!f.resolved && !f.L[0].open && !f.L[1].open) return 3;   // complete lists always resolve
    }
    for (int64_t x : f.A) std::printf("%lld\n", static_cast<long long>(x));
    std::fprintf(stderr, "depth %lld %lld\n", static_cast<long long>(f.L[0].size()),
                 static_cast<long long>(f.L[1].size()));
    return 0;
}
