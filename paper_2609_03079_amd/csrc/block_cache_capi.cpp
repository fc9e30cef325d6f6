// block_cache_capi.cpp - C entry points over ls::BlockCache for host-only unit tests
// (built with g++, no HIP).
#include <cstdint>
#include <vector>

#include "block_cache.h"

extern "C" {

void* bc_create(int64_t slots, int n_layers, int n_blk) {
    return new ls::BlockCache(slots, n_layers, n_blk);
}

void bc_destroy(void* h) { delete static_cast<ls::BlockCache*>(h); }

// Returns 1 on success; counts = {hits, misses, evictions};
// fills = n_fills x {pos, block, slot, evicted layer or -1}; protect_layer as in BlockCache::request.
int bc_request(void* h, int layer, const int32_t* blocks, int n, int64_t* counts, int32_t* fills,
               int32_t* n_fills, int protect_layer) {
    std::vector<ls::BlockCache::Fill> f;
    ls::BlockCache::Result r = static_cast<ls::BlockCache*>(h)->request(layer, blocks, n, &f, protect_layer);
    counts[0] = r.hits;
    counts[1] = r.misses;
    counts[2] = r.evictions;
    *n_fills = (int32_t)f.size();
    for (size_t i = 0; i < f.size(); ++i) {
        fills[4 * i + 0] = f[i].pos;
        fills[4 * i + 1] = f[i].block;
        fills[4 * i + 2] = f[i].slot;
        fills[4 * i + 3] = f[i].evicted_layer;
    }
    return r.ok ? 1 : 0;
}

void bc_slot_table(void* h, int layer, int32_t* out) {
    static_cast<ls::BlockCache*>(h)->slot_table(layer, out);
}

void bc_invalidate_layer(void* h, int layer) {
    static_cast<ls::BlockCache*>(h)->invalidate_layer(layer);
}
}
