// block_cache.h - host bookkeeping of the HBM block cache (no HIP, CPU-testable).
//
// The cache holds `slots` equal-sized slots; each holds one (layer, block).  A
// request lists blocks of one layer in priority order.  Blocks already cached
// are hits; every miss takes the least recently used slot that holds no block
// of the current request (all hits are marked used before any miss is placed,
// so the request never evicts itself).  Misses are reported in priority order,
// which is the order the copies are issued in (Sec. 3.2.2: arriving blocks are
// appended to the buffer in arrival order; the output does not depend on where
// a block lands).
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

namespace ls {

class BlockCache {
public:
    struct Fill {
        int pos;            // position of the block in the request
        int block;          // block id
        int slot;           // destination slot
        int evicted_layer;  // layer of the block the slot held before, or -1
    };
    struct Result {
        bool ok = false;
        int64_t hits = 0, misses = 0, evictions = 0;
    };

    BlockCache(int64_t slots, int n_layers, int n_blk)
        : slots_(slots), n_layers_(n_layers), n_blk_(n_blk),
          table_((size_t)n_layers * n_blk, -1), owner_((size_t)slots, -1),
          prev_((size_t)slots), next_((size_t)slots), mark_((size_t)slots, 0) {
        // LRU list: head = most recent; initially slot order
        for (int64_t i = 0; i < slots; ++i) {
            prev_[i] = i - 1;
            next_[i] = i + 1 < slots ? i + 1 : -1;
        }
        head_ = slots > 0 ? 0 : -1;
        tail_ = slots > 0 ? slots - 1 : -1;
    }

    int64_t slots() const { return slots_; }

    // Place blocks[0..n) of `layer`; fills receives the misses in priority order.  Blocks of
    // `protect_layer` (>= 0: a layer whose compute may still be queued) are not evicted either;
    // the request fails when the remaining slots cannot hold its misses.
    Result request(int layer, const int32_t* blocks, int n, std::vector<Fill>* fills, int protect_layer = -1) {
        Result r;
        if (fills) fills->clear();
        if (layer < 0 || layer >= n_layers_ || n < 0 || n > slots_) return r;
        ++epoch_;
        for (int i = 0; i < n; ++i)
            if (blocks[i] < 0 || blocks[i] >= n_blk_) return r;
        if (protect_layer >= 0 && protect_layer < n_layers_ && protect_layer != layer) {
            for (int b = 0; b < n_blk_; ++b) {
                const int64_t s = table_[key(protect_layer, b)];
                if (s >= 0) mark_[s] = epoch_;
            }
        }
        // pass 1: hits become most recent and are marked as part of this request
        std::vector<char> hit(n, 0);
        for (int i = 0; i < n; ++i) {
            const int64_t s = table_[key(layer, blocks[i])];
            if (s >= 0) {
                touch(s);
                mark_[s] = epoch_;
                hit[i] = 1;
                ++r.hits;
            }
        }
        // capacity check before any slot changes hands: the distinct misses must fit in the
        // slots this request may take (not its hits, not the protected layer's)
        {
            int64_t marked = 0, need = 0;
            for (int64_t s = 0; s < slots_; ++s) marked += mark_[s] == epoch_;
            std::vector<char> seen((size_t)n_blk_, 0);
            for (int i = 0; i < n; ++i)
                if (!hit[i] && !seen[(size_t)blocks[i]]) {
                    seen[(size_t)blocks[i]] = 1;
                    ++need;
                }
            if (need > slots_ - marked) return Result{};
        }
        // pass 2: misses take the least recent slot not marked by this request; a repeat of a
        // block placed earlier in this pass counts as a hit, so hits + misses == n.
        for (int i = 0; i < n; ++i) {
            if (hit[i]) continue;
            if (table_[key(layer, blocks[i])] >= 0) {
                ++r.hits;
                continue;
            }
            int64_t s = tail_;
            while (s >= 0 && mark_[s] == epoch_) s = prev_[s];  // least recent unprotected slot
            if (s < 0) return Result{};
            int evicted = -1;
            if (owner_[s] >= 0) {
                evicted = (int)(owner_[s] / n_blk_);
                table_[owner_[s]] = -1;
                ++r.evictions;
            }
            owner_[s] = (int64_t)key(layer, blocks[i]);
            table_[owner_[s]] = s;
            mark_[s] = epoch_;
            touch(s);
            ++r.misses;
            if (fills) fills->push_back(Fill{i, blocks[i], (int)s, evicted});
        }
        r.ok = true;
        return r;
    }

    // Drop every cached block of a layer (its weights changed).
    void invalidate_layer(int layer) {
        if (layer < 0 || layer >= n_layers_) return;
        for (int b = 0; b < n_blk_; ++b) {
            int64_t& s = table_[key(layer, b)];
            if (s >= 0) owner_[s] = -1;
            s = -1;
        }
    }

    // Slot of every block of a layer (-1: not cached).
    void slot_table(int layer, int32_t* out) const {
        for (int b = 0; b < n_blk_; ++b) out[b] = (int32_t)table_[key(layer, b)];
    }

    int64_t slot_of(int layer, int block) const { return table_[key(layer, block)]; }

private:
    size_t key(int layer, int block) const { return (size_t)layer * n_blk_ + block; }
    void touch(int64_t s) {
        if (s == head_) return;
        // unlink
        const int64_t p = prev_[s], nx = next_[s];
        if (p >= 0) next_[p] = nx;
        if (nx >= 0) prev_[nx] = p;
        if (s == tail_) tail_ = p;
        // push front
        prev_[s] = -1;
        next_[s] = head_;
        if (head_ >= 0) prev_[head_] = s;
        head_ = s;
        if (tail_ < 0) tail_ = s;
    }

    int64_t slots_;
    int n_layers_, n_blk_;
    std::vector<int64_t> table_;  // (layer, block) -> slot
    std::vector<int64_t> owner_;  // slot -> key or -1
    std::vector<int64_t> prev_, next_;
    std::vector<int64_t> mark_;
    int64_t head_ = -1, tail_ = -1;
    int64_t epoch_ = 0;
};

}  // namespace ls
