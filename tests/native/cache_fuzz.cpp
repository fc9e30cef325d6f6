// Randomised driver of the host-resident block cache (ls::BlockCache) for sanitizer builds:
// random request sequences over several layers, with and without a protected layer, checking
// after each request that hits + misses = n, that every requested block is resident in the
// slot its table names, that no slot is held by two blocks, and that a failed request changes
// nothing.  Exit status 0 when every check holds.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <vector>

#include "../../paper_2609_03079_amd/csrc/block_cache.h"

int main() {
    std::mt19937 rng(12345);
    for (int round = 0; round < 200; ++round) {
        const int L = 1 + (int)(rng() % 5), n_blk = 1 + (int)(rng() % 40);
        const int64_t slots = 1 + (int64_t)(rng() % 60);
        ls::BlockCache c(slots, L, n_blk);
        for (int it = 0; it < 100; ++it) {
            const int layer = (int)(rng() % L);
            const int n = (int)(rng() % (std::min<int64_t>(slots, n_blk) + 1));
            std::vector<int32_t> req;
            std::set<int> seen;
            while ((int)req.size() < n) {
                const int b = (int)(rng() % n_blk);
                if (seen.insert(b).second) req.push_back(b);
            }
            const int protect = (rng() % 3 == 0) ? (int)(rng() % L) : -1;
            std::vector<std::vector<int32_t>> before((size_t)L, std::vector<int32_t>((size_t)n_blk));
            for (int l = 0; l < L; ++l) c.slot_table(l, before[(size_t)l].data());
            std::vector<ls::BlockCache::Fill> fills;
            const auto r = c.request(layer, req.data(), n, &fills, protect);
            std::vector<std::vector<int32_t>> tab((size_t)L, std::vector<int32_t>((size_t)n_blk));
            for (int l = 0; l < L; ++l) c.slot_table(l, tab[(size_t)l].data());
            if (!r.ok) {
                if (tab != before) { std::puts("failed request changed the tables"); return 1; }
                continue;
            }
            if (r.hits + r.misses != n) { std::puts("hits + misses != n"); return 1; }
            if ((int)fills.size() != r.misses) { std::puts("fills != misses"); return 1; }
            for (int32_t b : req)
                if (tab[(size_t)layer][(size_t)b] < 0) { std::puts("requested block not resident"); return 1; }
            std::set<int32_t> used;
            for (int l = 0; l < L; ++l)
                for (int b = 0; b < n_blk; ++b) {
                    const int32_t sl = tab[(size_t)l][(size_t)b];
                    if (sl < 0) continue;
                    if (sl >= slots || !used.insert(sl).second) { std::puts("slot out of range or shared"); return 1; }
                }
            if (protect >= 0 && protect != layer)
                for (int b = 0; b < n_blk; ++b)
                    if (before[(size_t)protect][(size_t)b] >= 0 && tab[(size_t)protect][(size_t)b] < 0) {
                        std::puts("protected layer lost a block");
                        return 1;
                    }
            if (rng() % 17 == 0) c.invalidate_layer((int)(rng() % L));
        }
    }
    std::puts("cache_fuzz ok");
    return 0;
}
