// ls_api.hip - host engine behind the C ABI of include/ls_ffn.h.
//
// Owns the per-layer weight arenas in the library's block layout, the
// workspaces of the decode step and the stream bookkeeping; validates every
// argument before anything is enqueued.
#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <thread>

#include "block_cache.h"
#include "ls_decode.h"
#include "ls_internal.h"

using ls::Shape;

struct ls_ffn {
    ls_ffn_desc desc{};
    Shape shape{};
    int device = 0;
    hipStream_t stream = nullptr;
    hipStream_t copy_stream = nullptr;
    // host-resident mode: a second copy stream takes every other block copy of a stage (one
    // stream keeps the host link about 92% busy with block-sized copies, two about 100%); it
    // forks from copy_stream at each request and joins back before each stage is signalled
    hipStream_t copy_stream2 = nullptr;
    hipEvent_t copy_fork = nullptr, copy_join = nullptr;
    size_t block_bytes = 0;
    size_t layer_bytes = 0;  // blocks + bias + predictor (resident arena of one layer)

    // per layer
    std::vector<uint8_t*> arena;  // device: [blocks][bias][predictor]  (resident mode)
    std::vector<ls::LayerDev> dev;
    std::vector<uint8_t> is_set;
    std::vector<ls::HashDev> hash;  // per layer: stacked hashing predictor (null until set)

    // workspaces (device)
    float* z = nullptr;       // [maxB, r]
    float* scores = nullptr;  // [maxB, n_blk]
    int32_t* idx = nullptr;   // [maxB, n_blk]
    int32_t* count = nullptr; // [maxB]
    float* a = nullptr;       // [maxB, F]
    float* xbuf = nullptr;    // [maxB, d]  ping-pong partner of the decode step
    float* dn_part = nullptr; // [kDownPartsMax, maxB, d]  parts of the split down projection
    int64_t last_act_n = 0;
    int32_t last_act_B = 0;
    const float* last_act_src = nullptr;  // activations buffer of the last sparse step

    // staging for set_layer (pinned host)
    uint8_t* staging = nullptr;
    size_t staging_bytes = 0;

    // host-resident weights (LS_WEIGHTS_HOST)
    std::vector<uint8_t*> host_blocks;  // per layer, pinned [n_blk][block_bytes] (one allocation per layer)
    uint8_t* cache = nullptr;        // device, [slots][block_bytes]
    int32_t* slot_tables = nullptr;  // device, [L][n_blk]
    int32_t* slot_tables_host = nullptr;  // pinned mirror
    ls::BlockCache* bcache = nullptr;
    // per layer: the copy stages of its latest request ([begin,end) of the list and the event
    // after the stage's copies), whether it was ever requested, and an event after its latest
    // compute (a copy into a slot waits only for the compute of the layer that held the slot)
    std::vector<std::vector<hipEvent_t>> stage_events;
    std::vector<std::vector<std::pair<int, int>>> stage_ranges;
    std::vector<uint8_t> streamed;
    std::vector<hipEvent_t> layer_done;
    std::vector<uint8_t> layer_done_recorded;
    int32_t* idx_pinned = nullptr;  // pinned [3][n_blk]: lists read back by the streamed decode step
    int32_t* spec_idx = nullptr;    // device [2][n_blk] + counts [2]: its speculative selections
    hipEvent_t spec_read[2] = {nullptr, nullptr};  // after the read-back of each speculative list

    std::vector<hipEvent_t> table_uploaded;  // per layer: last slot-table upload

    // kernel timing
    uint32_t timing = 0;      // bit i: bracket launches of kernel id i with events
    struct Pending {
        int kernel;
        hipEvent_t start, stop;
    };
    std::vector<Pending> pending;
    std::vector<hipEvent_t> event_pool;
    double kernel_ms[LS_K_COUNT] = {};
    int64_t kernel_launches[LS_K_COUNT] = {};

    // fused decode kernel
    uint64_t* mailbox = nullptr;  // tagged exchange words (device, zero-initialised)
    size_t mailbox_words = 0;
    ls::LayerPtrs* layer_tab = nullptr;  // device [L]
    std::vector<ls::LayerPtrs> layer_tab_host;
    int* dev_err = nullptr;       // device error flag
    uint32_t epoch = 0;
    int n_wg = 0;                 // compute units
    int decode_path = 0;          // LS_CFG_DECODE_PATH
    bool last_fused = false;      // the last ls_decode_step ran the fused kernel
    int trace_wg = -1;            // LS_CFG_TRACE_WG
    uint64_t* trace = nullptr;    // device [L][kTracePoints]
    int spec_blocks = 0;          // LS_CFG_SPEC_BLOCKS
    int cooperative = 1;          // LS_CFG_COOPERATIVE

    // streamed-step coordination (LS_CFG_STREAM_SYNC)
    int stream_sync = 0;
    uint32_t* arrive = nullptr;      // fine-grained device [L][kMaxStages]: copy-stage arrival words
    size_t arrive_bytes = 0;
    uint32_t* stage_done = nullptr;  // pinned coherent host [L][kMaxStages] done words, then the status word
    uint32_t* stage_cnt = nullptr;   // device [2][kMaxStages]: the stage consumer's counters
    uint32_t stage_tag = 0;          // last tag handed out
    int64_t stage_wait_us = 2000000; // LS_CFG_STAGE_WAIT_US
    std::vector<uint32_t> layer_tag; // per layer: tag of its latest flagged request
    std::vector<int> layer_stages;   // per layer: stages of that request

    ls_status sticky = LS_OK;
    std::string err;
};

namespace {

std::string g_create_error;

// Arrival words live in fine-grained device memory, which the library does not free while the
// process runs: a released buffer goes back to this pool for the next context that needs one
// of the same size.
std::mutex g_arrive_mu;
std::vector<std::pair<size_t, uint32_t*>> g_arrive_pool;

uint32_t* arrive_take(size_t bytes) {
    {
        std::lock_guard<std::mutex> lk(g_arrive_mu);
        for (size_t i = 0; i < g_arrive_pool.size(); ++i)
            if (g_arrive_pool[i].first == bytes) {
                uint32_t* p = g_arrive_pool[i].second;
                g_arrive_pool.erase(g_arrive_pool.begin() + (long)i);
                return p;
            }
    }
    void* p = nullptr;
    if (hipExtMallocWithFlags(&p, bytes, hipDeviceMallocFinegrained) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    return static_cast<uint32_t*>(p);
}

void arrive_give(uint32_t* p, size_t bytes) {
    std::lock_guard<std::mutex> lk(g_arrive_mu);
    g_arrive_pool.emplace_back(bytes, p);
}

ls_status fail(ls_ffn* c, ls_status st, const std::string& msg) {
    if (c) {
        c->err = msg;
        if (st == LS_E_DEVICE) c->sticky = LS_E_DEVICE;
    } else {
        g_create_error = msg;
    }
    return st;
}

ls_status hip_fail(ls_ffn* c, hipError_t e, const char* what) {
    std::string m = std::string(what) + ": " + hipGetErrorString(e);
    if (c) return fail(c, LS_E_DEVICE, m);
    g_create_error = m;
    return LS_E_DEVICE;
}

#define LS_HIP(ctx, call)                                   \
    do {                                                    \
        hipError_t e_ = (call);                             \
        if (e_ != hipSuccess) return hip_fail(ctx, e_, #call); \
    } while (0)

ls_status check_ctx(ls_ffn* c) {
    if (!c) return LS_E_INVAL;
    if (c->sticky != LS_OK) {
        c->err = "context is in a failed state after an earlier device error";
        return c->sticky;
    }
    return LS_OK;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

hipError_t take_event(ls_ffn* c, hipEvent_t* e) {
    if (!c->event_pool.empty()) {
        *e = c->event_pool.back();
        c->event_pool.pop_back();
        return hipSuccess;
    }
    return hipEventCreate(e);
}

// Launch `fn` (returning hipError_t); when timing is on, bracket it with an event pair.
template <typename Fn>
hipError_t timed(ls_ffn* c, int kernel, Fn&& fn) {
    if (!((c->timing >> kernel) & 1u)) return fn();
    hipEvent_t a, b;
    hipError_t e = take_event(c, &a);
    if (e != hipSuccess) return e;
    e = take_event(c, &b);
    if (e != hipSuccess) return e;
    if ((e = hipEventRecord(a, c->stream)) != hipSuccess) return e;
    if ((e = fn()) != hipSuccess) return e;
    if ((e = hipEventRecord(b, c->stream)) != hipSuccess) return e;
    c->pending.push_back({kernel, a, b});
    return hipSuccess;
}

hipError_t fold_timing(ls_ffn* c) {
    for (auto& p : c->pending) {
        hipError_t e = hipEventSynchronize(p.stop);
        if (e != hipSuccess) return e;
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, p.start, p.stop);
        if (e != hipSuccess) return e;
        c->kernel_ms[p.kernel] += ms;
        c->kernel_launches[p.kernel] += 1;
        c->event_pool.push_back(p.start);
        c->event_pool.push_back(p.stop);
    }
    c->pending.clear();
    return hipSuccess;
}

// Offsets inside one layer arena.  The predictor region holds either the folded fp32
// product [n_blk, d] (pf) or the two factors in the grouped row order (p1, then p2).
struct LayerLayout {
    size_t blocks, bias, p1, p2, pf, total;
};

LayerLayout layout_of(const Shape& s, size_t block_bytes) {
    const size_t es = ls::elem_size(s.dtype);
    LayerLayout L{};
    L.blocks = 0;
    L.bias = align_up((size_t)s.n_blk * block_bytes, 256);
    L.p1 = L.p2 = L.pf = align_up(L.bias + (size_t)s.F * es, 256);
    if (s.fold) {
        L.total = align_up(L.pf + (size_t)s.n_blk * s.d * sizeof(float), 256);
    } else {
        L.p2 = align_up(L.p1 + (size_t)s.G * s.p1_rpw * s.d * es, 256);
        L.total = align_up(L.p2 + (size_t)s.G * s.p2_rpw * s.r * es, 256);
    }
    return L;
}

// Convert one layer's FFN weights from nn.Linear layouts into the block layout:
// block b = [gate rows b*blk.. (blk x d) | up rows (blk x d) | down piece], where the
// down piece is [d/16][blk/V][16][V]: element (neuron q, column m) of the block sits at
// ((m/16) * (blk/V) + q/V) * 16*V + (m%16) * V + q%V.
void convert_blocks(const Shape& s, const uint8_t* gate, const uint8_t* up, const uint8_t* down,
                    uint8_t* dst, size_t block_bytes) {
    const size_t es = ls::elem_size(s.dtype);
    const int V = ls::vec_elems(s.dtype);
    const size_t rows_bytes = (size_t)s.blk * s.d * es;
    unsigned nth = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
    auto work = [&](unsigned t) {
        for (int b = (int)t; b < s.n_blk; b += (int)nth) {
            uint8_t* blk = dst + (size_t)b * block_bytes;
            std::memcpy(blk, gate + (size_t)b * rows_bytes, rows_bytes);
            std::memcpy(blk + rows_bytes, up + (size_t)b * rows_bytes, rows_bytes);
            uint8_t* dn = blk + 2 * rows_bytes;
            for (int m = 0; m < s.d; ++m) {
                const uint8_t* src_row = down + ((size_t)m * s.F + (size_t)b * s.blk) * es;
                const size_t tile_base = (size_t)(m / ls::kColTile) * (s.blk / V);
                const size_t col = m % ls::kColTile;
                for (int q = 0; q < s.blk; ++q) {
                    const size_t pos = ((tile_base + q / V) * ls::kColTile + col) * V + q % V;
                    std::memcpy(dn + pos * es, src_row + (size_t)q * es, es);
                }
            }
        }
    };
    std::vector<std::thread> th;
    for (unsigned t = 1; t < nth; ++t) th.emplace_back(work, t);
    work(0);
    for (auto& x : th) x.join();
}

ls_status validate_desc(const ls_ffn_desc* d) {
    if (!d) return fail(nullptr, LS_E_INVAL, "desc is NULL");
    if (d->n_layers < 1) return fail(nullptr, LS_E_INVAL, "n_layers must be >= 1");
    if (d->d_model < 64 || d->d_model % 64) return fail(nullptr, LS_E_INVAL, "d_model must be a positive multiple of 64");
    if (d->block < 8 || d->block % 8) return fail(nullptr, LS_E_INVAL, "block must be a positive multiple of 8");
    if (d->d_ff < d->block || d->d_ff % d->block) return fail(nullptr, LS_E_INVAL, "d_ff must be a positive multiple of block");
    if (d->d_ff / d->block > ls::kMaxBlocks) return fail(nullptr, LS_E_INVAL, "d_ff / block exceeds 2048 blocks");
    if (d->rank < 64 || d->rank % 64) return fail(nullptr, LS_E_INVAL, "rank must be a positive multiple of 64");
    if (d->max_batch < 1 || d->max_batch > ls::kMaxBatch) return fail(nullptr, LS_E_INVAL, "max_batch must be in 1..8");
    if (d->dtype != LS_F32 && d->dtype != LS_F16 && d->dtype != LS_BF16) return fail(nullptr, LS_E_INVAL, "bad dtype");
    if (d->act != LS_ACT_REGLU && d->act != LS_ACT_SWIGLU_THRESH) return fail(nullptr, LS_E_INVAL, "bad act");
    if (d->residency != LS_WEIGHTS_HBM && d->residency != LS_WEIGHTS_HOST) return fail(nullptr, LS_E_INVAL, "bad residency");
    if (d->prenorm_rms != 0 && d->prenorm_rms != 1) return fail(nullptr, LS_E_INVAL, "prenorm_rms must be 0 or 1");
    if (d->debug_flags != 0) return fail(nullptr, LS_E_INVAL, "debug_flags must be 0");
    return LS_OK;
}

void free_all(ls_ffn* c) {
    for (auto p : c->arena) if (p) (void)hipFree(p);
    c->arena.clear();
    for (auto& h : c->hash) if (h.w1) (void)hipFree(h.w1);  // one allocation per layer
    c->hash.clear();
    for (void* p : {(void*)c->z, (void*)c->scores, (void*)c->idx, (void*)c->count,
                    (void*)c->a, (void*)c->xbuf, (void*)c->dn_part, (void*)c->cache, (void*)c->slot_tables,
                    (void*)c->mailbox, (void*)c->layer_tab, (void*)c->dev_err, (void*)c->spec_idx,
                    (void*)c->trace, (void*)c->stage_cnt})
        if (p) (void)hipFree(p);
    if (c->staging) (void)hipHostFree(c->staging);
    for (auto p : c->host_blocks) if (p) (void)hipHostFree(p);
    c->host_blocks.clear();
    if (c->slot_tables_host) (void)hipHostFree(c->slot_tables_host);
    for (auto& v : c->stage_events)
        for (auto e : v) (void)hipEventDestroy(e);
    for (auto e : c->layer_done) if (e) (void)hipEventDestroy(e);
    for (auto e : c->spec_read) if (e) (void)hipEventDestroy(e);
    if (c->idx_pinned) (void)hipHostFree(c->idx_pinned);
    if (c->stage_done) (void)hipHostFree(c->stage_done);
    if (c->arrive) arrive_give(c->arrive, c->arrive_bytes);
    if (c->copy_stream2) (void)hipStreamSynchronize(c->copy_stream2);
    if (c->copy_stream) (void)hipStreamDestroy(c->copy_stream);
    if (c->copy_stream2) (void)hipStreamDestroy(c->copy_stream2);
    if (c->copy_fork) (void)hipEventDestroy(c->copy_fork);
    if (c->copy_join) (void)hipEventDestroy(c->copy_join);
    for (auto e : c->table_uploaded) if (e) (void)hipEventDestroy(e);
    for (auto& p : c->pending) {
        (void)hipEventDestroy(p.start);
        (void)hipEventDestroy(p.stop);
    }
    for (auto e : c->event_pool) (void)hipEventDestroy(e);
    delete c->bcache;
}

template <typename T>
hipError_t dmalloc(T** p, size_t n) {
    return hipMalloc(reinterpret_cast<void**>(p), std::max<size_t>(n, 1) * sizeof(T));
}

// The fused kernel's bare 32-bit exchange words start empty (0xffffffff): the layer inputs
// and, in every layer's activation row, the list's two halves (its first F 64-bit words).
hipError_t empty_bare_words(ls_ffn* c) {
    const ls::Shape& s = c->shape;
    const int L = c->desc.n_layers;
    hipError_t e = hipMemset(c->mailbox, 0xff, ls::fused_input_words(s, L) * sizeof(uint64_t));
    if (e != hipSuccess) return e;
    return hipMemset2D(c->mailbox + ls::fused_acts_offset(s, L), 2 * (size_t)s.F * sizeof(uint64_t), 0xff,
                       (size_t)s.F * sizeof(uint64_t), (size_t)L);
}

}  // namespace

extern "C" {

static bool resolve_scratch(int device);

ls_status ls_ffn_create(const ls_ffn_desc* desc, ls_ffn** out) {
    if (!out) return fail(nullptr, LS_E_INVAL, "out is NULL");
    *out = nullptr;
    ls_status st = validate_desc(desc);
    if (st != LS_OK) return st;
    ls_ffn* c = new (std::nothrow) ls_ffn();
    if (!c) return fail(nullptr, LS_E_NOMEM, "host allocation failed");
    c->desc = *desc;
    Shape& s = c->shape;
    s.d = desc->d_model;
    s.F = desc->d_ff;
    s.blk = desc->block;
    s.r = desc->rank;
    s.n_blk = desc->d_ff / desc->block;
    s.dtype = desc->dtype;
    s.act = desc->act;
    s.prenorm = desc->prenorm_rms;
    s.block_elems = (size_t)3 * s.blk * s.d;
    c->block_bytes = s.block_elems * ls::elem_size(s.dtype);
    c->stream = static_cast<hipStream_t>(desc->stream);
    {
        hipDeviceProp_t prop;
        if (hipGetDevice(&c->device) != hipSuccess || hipGetDeviceProperties(&prop, c->device) != hipSuccess) {
            delete c;
            return fail(nullptr, LS_E_DEVICE, "no HIP device");
        }
        c->n_wg = prop.multiProcessorCount;
        if (!resolve_scratch(c->device)) {
            delete c;
            return fail(nullptr, LS_E_DEVICE, "could not resolve the static scratch array on this device");
        }
        s.G = c->n_wg;
        s.p1_rpw = (s.r + s.G - 1) / s.G;
        s.p2_rpw = (s.n_blk + s.G - 1) / s.G;
    }
    s.fold = ls::predictor_folds(s.d, s.r, s.n_blk, s.dtype);
    const int L = desc->n_layers, B = desc->max_batch;
    auto bail = [&](ls_status code, const std::string& m) {
        free_all(c);
        delete c;
        return fail(nullptr, code, m);
    };
    const LayerLayout lay = layout_of(s, c->block_bytes);
    c->dev.resize(L);
    c->is_set.assign(L, 0);
    c->arena.assign(L, nullptr);
    if (desc->residency == LS_WEIGHTS_HBM) {
        c->layer_bytes = lay.total;
        for (int l = 0; l < L; ++l) {
            if (hipMalloc(reinterpret_cast<void**>(&c->arena[l]), lay.total) != hipSuccess) {
                (void)hipGetLastError();
                return bail(LS_E_NOMEM, "device allocation of the weight arena failed");
            }
            c->dev[l].blocks = c->arena[l] + lay.blocks;
            c->dev[l].bias = c->arena[l] + lay.bias;
            c->dev[l].p1 = c->arena[l] + lay.p1;
            c->dev[l].p2 = c->arena[l] + lay.p2;
            c->dev[l].pf = reinterpret_cast<const float*>(c->arena[l] + lay.pf);
        }
    } else {
        // predictors and bias stay resident in HBM; the blocks live in pinned host memory and
        // are streamed into a bounded HBM cache.
        const size_t small = lay.total - lay.bias;
        c->layer_bytes = small;
        const int64_t slots = (int64_t)(desc->hbm_cache_bytes / c->block_bytes);
        if (slots < 1) return bail(LS_E_INVAL, "hbm_cache_bytes holds no block");
        for (int l = 0; l < L; ++l) {
            if (hipMalloc(reinterpret_cast<void**>(&c->arena[l]), small) != hipSuccess) {
                (void)hipGetLastError();
                return bail(LS_E_NOMEM, "device allocation of the predictor arena failed");
            }
            c->dev[l].bias = c->arena[l];
            c->dev[l].p1 = c->arena[l] + (lay.p1 - lay.bias);
            c->dev[l].p2 = c->arena[l] + (lay.p2 - lay.bias);
            c->dev[l].pf = reinterpret_cast<const float*>(c->arena[l] + (lay.pf - lay.bias));
        }
        // one pinned allocation per layer: a single one of the whole stack (e.g. 107.5 GiB for
        // the 70B shape) is refused by the runtime where per-layer ones are not
        const size_t layer_host_bytes = (size_t)s.n_blk * c->block_bytes;
        c->host_blocks.assign(L, nullptr);
        for (int l = 0; l < L; ++l) {
            if (hipHostMalloc(reinterpret_cast<void**>(&c->host_blocks[l]), layer_host_bytes, hipHostMallocDefault) !=
                hipSuccess) {
                (void)hipGetLastError();
                c->host_blocks[l] = nullptr;
                return bail(LS_E_NOMEM, "pinned host allocation of the weight arena failed at layer " + std::to_string(l) +
                                            " (" + std::to_string(layer_host_bytes >> 20) + " MiB per layer)");
            }
        }
        if (hipMalloc(reinterpret_cast<void**>(&c->cache), (size_t)slots * c->block_bytes) != hipSuccess) {
            (void)hipGetLastError();
            return bail(LS_E_NOMEM, "device allocation of the block cache failed");
        }
        if (dmalloc(&c->slot_tables, (size_t)L * s.n_blk) != hipSuccess ||
            hipHostMalloc(reinterpret_cast<void**>(&c->slot_tables_host), (size_t)L * s.n_blk * sizeof(int32_t),
                          hipHostMallocDefault) != hipSuccess) {
            (void)hipGetLastError();
            return bail(LS_E_NOMEM, "slot table allocation failed");
        }
        for (size_t i = 0; i < (size_t)L * s.n_blk; ++i) c->slot_tables_host[i] = -1;
        if (hipMemcpy(c->slot_tables, c->slot_tables_host, (size_t)L * s.n_blk * sizeof(int32_t),
                      hipMemcpyHostToDevice) != hipSuccess)
            return bail(LS_E_DEVICE, "slot table upload failed");
        c->bcache = new (std::nothrow) ls::BlockCache(slots, L, s.n_blk);
        if (!c->bcache) return bail(LS_E_NOMEM, "host allocation failed");
        if (hipStreamCreateWithFlags(&c->copy_stream, hipStreamNonBlocking) != hipSuccess ||
            hipStreamCreateWithFlags(&c->copy_stream2, hipStreamNonBlocking) != hipSuccess ||
            hipEventCreateWithFlags(&c->copy_fork, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&c->copy_join, hipEventDisableTiming) != hipSuccess)
            return bail(LS_E_DEVICE, "stream creation failed");
        c->table_uploaded.assign(L, nullptr);
        c->layer_done.assign(L, nullptr);
        c->layer_done_recorded.assign(L, 0);
        c->streamed.assign(L, 0);
        c->stage_events.assign(L, {});
        c->stage_ranges.assign(L, {});
        for (int l = 0; l < L; ++l)
            if (hipEventCreateWithFlags(&c->table_uploaded[l], hipEventDisableTiming) != hipSuccess ||
                hipEventCreateWithFlags(&c->layer_done[l], hipEventDisableTiming) != hipSuccess)
                return bail(LS_E_DEVICE, "event creation failed");
        if (hipHostMalloc((void**)&c->idx_pinned, 3 * (size_t)s.n_blk * sizeof(int32_t)) != hipSuccess ||
            dmalloc(&c->spec_idx, 2 * (size_t)s.n_blk + 2) != hipSuccess) {
            (void)hipGetLastError();
            return bail(LS_E_NOMEM, "streamed-step buffers allocation failed");
        }
        for (auto& e : c->spec_read)
            if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess)
                return bail(LS_E_DEVICE, "event creation failed");
    }
    if (dmalloc(&c->z, (size_t)B * (s.fold ? 1 : s.r)) != hipSuccess ||
        dmalloc(&c->scores, (size_t)B * s.n_blk) != hipSuccess ||
        dmalloc(&c->idx, (size_t)B * s.n_blk) != hipSuccess || dmalloc(&c->count, (size_t)B) != hipSuccess ||
        dmalloc(&c->a, (size_t)B * s.F) != hipSuccess || dmalloc(&c->xbuf, (size_t)B * s.d) != hipSuccess ||
        dmalloc(&c->dn_part, (size_t)ls::kDownPartsMax * B * s.d) != hipSuccess) {
        (void)hipGetLastError();
        return bail(LS_E_NOMEM, "workspace allocation failed");
    }
    {
        c->mailbox_words = ls::fused_mailbox_words(s, L, c->n_wg);
        c->layer_tab_host.assign(L, ls::LayerPtrs{});
        if (dmalloc(&c->mailbox, c->mailbox_words) != hipSuccess || dmalloc(&c->layer_tab, (size_t)L) != hipSuccess ||
            dmalloc(&c->dev_err, 1) != hipSuccess) {
            (void)hipGetLastError();
            return bail(LS_E_NOMEM, "fused-kernel workspace allocation failed");
        }
        if (hipMemset(c->mailbox, 0, c->mailbox_words * sizeof(uint64_t)) != hipSuccess ||
            empty_bare_words(c) != hipSuccess ||
            hipMemset(c->dev_err, 0, sizeof(int)) != hipSuccess ||
            hipMemset(c->layer_tab, 0, (size_t)L * sizeof(ls::LayerPtrs)) != hipSuccess)
            return bail(LS_E_DEVICE, "workspace initialisation failed");
    }
    *out = c;
    return LS_OK;
}

ls_status ls_ffn_destroy(ls_ffn* c) {
    if (!c) return LS_E_INVAL;
    (void)hipStreamSynchronize(c->stream);
    if (c->copy_stream) (void)hipStreamSynchronize(c->copy_stream);
    free_all(c);
    delete c;
    return LS_OK;
}

const char* ls_last_error(const ls_ffn* c) { return c ? c->err.c_str() : g_create_error.c_str(); }

static ls_status upload_table(ls_ffn* c, int32_t layer);

ls_status ls_ffn_set_layer(ls_ffn* c, int32_t layer, const ls_layer_weights* w) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    if (layer < 0 || layer >= c->desc.n_layers) return fail(c, LS_E_INVAL, "layer out of range");
    if (!w || !w->w_gate || !w->w_up || !w->w_down || !w->p1 || !w->p2)
        return fail(c, LS_E_INVAL, "null weight pointer");
    const size_t es = ls::elem_size(s.dtype);
    const LayerLayout lay = layout_of(s, c->block_bytes);
    // staged bytes: blocks (resident mode), bias and the factored predictor; the folded
    // predictor is formed on the device instead
    const size_t staged_end = s.fold ? lay.pf : lay.total;
    const size_t need = c->desc.residency == LS_WEIGHTS_HBM ? staged_end : staged_end - lay.bias;
    if (!c->staging || c->staging_bytes < need) {
        if (c->staging) (void)hipHostFree(c->staging);
        c->staging = nullptr;
        if (hipHostMalloc(reinterpret_cast<void**>(&c->staging), need, hipHostMallocDefault) != hipSuccess) {
            (void)hipGetLastError();
            c->staging_bytes = 0;
            return fail(c, LS_E_NOMEM, "pinned staging allocation failed");
        }
        c->staging_bytes = need;
    }
    LS_HIP(c, hipStreamSynchronize(c->stream));  // staging may still feed an earlier copy
    // host-resident blocks of this layer may still feed queued cache fills
    if (c->copy_stream) LS_HIP(c, hipStreamSynchronize(c->copy_stream));
    uint8_t* blocks_dst;
    size_t off_small;
    if (c->desc.residency == LS_WEIGHTS_HBM) {
        blocks_dst = c->staging;
        off_small = lay.bias;
    } else {
        blocks_dst = c->host_blocks[layer];
        off_small = 0;
    }
    convert_blocks(s, static_cast<const uint8_t*>(w->w_gate), static_cast<const uint8_t*>(w->w_up),
                   static_cast<const uint8_t*>(w->w_down), blocks_dst, c->block_bytes);
    uint8_t* sm = c->staging + off_small;
    std::memset(sm, 0, lay.p1 - lay.bias);
    if (w->b_gate) std::memcpy(sm, w->b_gate, (size_t)s.F * es);
    if (!s.fold) {
        // predictor rows in the grouped order (padding rows stay zero)
        std::memset(sm + (lay.p1 - lay.bias), 0, lay.total - lay.p1);
        for (int i = 0; i < s.r; ++i)
            std::memcpy(sm + (lay.p1 - lay.bias) + ((size_t)(i % s.G) * s.p1_rpw + i / s.G) * s.d * es,
                        static_cast<const uint8_t*>(w->p1) + (size_t)i * s.d * es, (size_t)s.d * es);
        for (int i = 0; i < s.n_blk; ++i)
            std::memcpy(sm + (lay.p2 - lay.bias) + ((size_t)(i % s.G) * s.p2_rpw + i / s.G) * s.r * es,
                        static_cast<const uint8_t*>(w->p2) + (size_t)i * s.r * es, (size_t)s.r * es);
    }
    LS_HIP(c, hipMemcpyAsync(c->arena[layer], c->staging, need, hipMemcpyHostToDevice, c->stream));
    LS_HIP(c, hipStreamSynchronize(c->stream));
    if (s.fold) {
        // P2 P1 on the device (fp64 accumulation), written into the predictor region
        const size_t p1_bytes = (size_t)s.r * s.d * es, p2_bytes = (size_t)s.n_blk * s.r * es;
        uint8_t* tmp = nullptr;
        if (hipMalloc(reinterpret_cast<void**>(&tmp), p1_bytes + p2_bytes) != hipSuccess) {
            (void)hipGetLastError();
            return fail(c, LS_E_NOMEM, "device allocation for the predictor fold failed");
        }
        hipError_t e = hipMemcpy(tmp, w->p1, p1_bytes, hipMemcpyHostToDevice);
        if (e == hipSuccess) e = hipMemcpy(tmp + p1_bytes, w->p2, p2_bytes, hipMemcpyHostToDevice);
        if (e == hipSuccess)
            e = ls::launch_fold_predictor(s.dtype, tmp, tmp + p1_bytes, s.r, s.d, s.n_blk,
                                          const_cast<float*>(c->dev[layer].pf), c->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
        const hipError_t ef = hipFree(tmp);
        LS_HIP(c, e);
        LS_HIP(c, ef);
    }
    c->dev[layer].bias =
        w->b_gate ? c->arena[layer] + (c->desc.residency == LS_WEIGHTS_HBM ? lay.bias : 0) : nullptr;
    c->dev[layer].threshold = w->threshold;
    if (c->desc.residency == LS_WEIGHTS_HOST) {
        // the cached copies hold the old weights: drop them, give the device an empty table
        // and require a new ls_stream_weights before the next step of this layer
        c->bcache->invalidate_layer(layer);
        ls_status st2 = upload_table(c, layer);
        if (st2 != LS_OK) return st2;
        LS_HIP(c, hipStreamSynchronize(c->copy_stream));
        c->streamed[layer] = 0;
        c->stage_ranges[layer].clear();
    }
    {
        ls::LayerPtrs lp{};
        lp.blocks = c->dev[layer].blocks;
        lp.bias = c->dev[layer].bias;
        lp.pf = c->dev[layer].pf;
        lp.threshold = w->threshold;
        c->layer_tab_host[layer] = lp;
        LS_HIP(c, hipMemcpy(c->layer_tab + layer, &lp, sizeof lp, hipMemcpyHostToDevice));
    }
    c->is_set[layer] = 1;
    return LS_OK;
}

// scores = P2 (P1 h) for the layer input x (h = its RMS prenorm, applied inside the first
// GEMV): one GEMV over the folded rows, or the two factors in turn.
static ls_status predictor_gemv(ls_ffn* c, const ls::LayerDev& L, const float* x, int B, float* scores) {
    const Shape& s = c->shape;
    const bool rms = s.prenorm != 0;
    if (s.fold) {
        LS_HIP(c, timed(c, LS_K_PRED_P1, [&] { return ls::launch_gemv_rows(LS_F32, L.pf, s.n_blk, s.d, 1, s.n_blk, x, B, rms, scores, c->stream); }));
        return LS_OK;
    }
    LS_HIP(c, timed(c, LS_K_PRED_P1, [&] { return ls::launch_gemv_rows(s.dtype, L.p1, s.r, s.d, s.G, s.p1_rpw, x, B, rms, c->z, c->stream); }));
    LS_HIP(c, timed(c, LS_K_PRED_P2, [&] { return ls::launch_gemv_rows(s.dtype, L.p2, s.n_blk, s.r, s.G, s.p2_rpw, c->z, B, false, scores, c->stream); }));
    return LS_OK;
}

ls_status ls_predict(ls_ffn* c, int32_t layer, const float* x, int32_t B, float* scores) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    if (layer < 0 || layer >= c->desc.n_layers) return fail(c, LS_E_INVAL, "layer out of range");
    if (!x || !scores) return fail(c, LS_E_INVAL, "null pointer");
    if (B < 1 || B > c->desc.max_batch) return fail(c, LS_E_INVAL, "B out of range");
    if (!c->is_set[layer]) return fail(c, LS_E_STATE, "layer weights not set");
    return predictor_gemv(c, c->dev[layer], x, B, scores);
}

ls_status ls_select_blocks(ls_ffn* c, const float* scores, int32_t B, ls_sel_mode mode, int32_t k,
                           float tau, int32_t union_batch, int32_t cap, int32_t* idx, int32_t* count) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const int n = c->shape.n_blk;
    if (!scores || !idx || !count) return fail(c, LS_E_INVAL, "null pointer");
    if (B < 1 || B > c->desc.max_batch) return fail(c, LS_E_INVAL, "B out of range");
    if (mode != LS_SEL_TOPK && mode != LS_SEL_THRESHOLD) return fail(c, LS_E_INVAL, "bad selection mode");
    const bool uni = union_batch && B > 1;
    if (mode == LS_SEL_TOPK) {
        if (k < 1 || k > n) return fail(c, LS_E_INVAL, "k must be in 1..n_blk");
        const int need = uni ? std::min(n, B * k) : k;
        if (cap < need) return fail(c, LS_E_INVAL, "cap too small for the selection");
    } else if (cap < n) {
        return fail(c, LS_E_INVAL, "threshold selection needs cap >= n_blk");
    }
    LS_HIP(c, timed(c, LS_K_SELECT, [&] {
        return ls::launch_select(scores, B, n, (int)mode, k, tau, union_batch ? 1 : 0, cap, idx, count, c->stream);
    }));
    return LS_OK;
}

// Waits of the compute stream for the copy stages of a streamed layer that overlap [begin,end).
static ls_status wait_stages(ls_ffn* c, int32_t layer, int32_t begin, int32_t end) {
    if (c->desc.residency != LS_WEIGHTS_HOST) return LS_OK;
    const auto& ranges = c->stage_ranges[layer];
    for (size_t s = 0; s < ranges.size(); ++s)
        if (ranges[s].first < end && begin < ranges[s].second)
            LS_HIP(c, hipStreamWaitEvent(c->stream, c->stage_events[layer][s], 0));
    return LS_OK;
}

// The sparse step over [begin, end) of the list with the given scratch: a_buf [B, F]
// activations, part [kDownPartsMax, B, d] parts of the split down projection.
// may_time: bracket the launches with timing events when kernel timing is on (taking an
// event can create one); false launches them bare.
static ls_status sparse_step(ls_ffn* c, int32_t layer, const float* x_in, int32_t B, const int32_t* idx,
                             const int32_t* count, int32_t begin, int32_t end, float* x_acc, float* a_buf,
                             float* part, bool may_time) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    if (layer < 0 || layer >= c->desc.n_layers) return fail(c, LS_E_INVAL, "layer out of range");
    if (!x_in || !idx || !count || !x_acc) return fail(c, LS_E_INVAL, "null pointer");
    if (x_in == x_acc) return fail(c, LS_E_INVAL, "x_in and x_acc must not alias");
    if (B < 1 || B > c->desc.max_batch) return fail(c, LS_E_INVAL, "B out of range");
    if (begin < 0 || end < begin) return fail(c, LS_E_INVAL, "need 0 <= begin <= end");
    if (!c->is_set[layer]) return fail(c, LS_E_STATE, "layer weights not set");
    end = std::min(end, s.n_blk);
    begin = std::min(begin, end);
    ls::LayerDev L = c->dev[layer];
    const int32_t* slot_table = nullptr;
    if (c->desc.residency == LS_WEIGHTS_HOST) {
        if (!c->streamed[layer])
            return fail(c, LS_E_STATE, "blocks of this layer were not streamed (ls_stream_weights)");
        L.blocks = c->cache;
        slot_table = c->slot_tables + (size_t)layer * s.n_blk;
        // the layer's table may have been rewritten since its own stages (another layer's
        // request evicted some of its blocks)
        LS_HIP(c, hipStreamWaitEvent(c->stream, c->table_uploaded[layer], 0));
        st = wait_stages(c, layer, begin, end);
        if (st != LS_OK) return st;
    }
    auto gateup = [&] { return ls::launch_gateup(s, L, slot_table, x_in, B, idx, count, begin, end, a_buf, c->stream); };
    auto down = [&] { return ls::launch_down(s, L, slot_table, a_buf, B, idx, count, begin, end, x_in, x_acc, part, c->stream); };
    LS_HIP(c, may_time ? timed(c, LS_K_GATEUP, gateup) : gateup());
    LS_HIP(c, may_time ? timed(c, LS_K_DOWN, down) : down());
    if (c->desc.residency == LS_WEIGHTS_HOST) {
        LS_HIP(c, hipEventRecord(c->layer_done[layer], c->stream));
        c->layer_done_recorded[layer] = 1;
    }
    c->last_act_n = (int64_t)end * s.blk;
    c->last_act_B = B;
    c->last_act_src = a_buf;
    return LS_OK;
}

ls_status ls_sparse_ffn_step(ls_ffn* c, int32_t layer, const float* x_in, int32_t B,
                             const int32_t* idx, const int32_t* count, int32_t begin, int32_t end,
                             float* x_acc) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    return sparse_step(c, layer, x_in, B, idx, count, begin, end, x_acc, c->a, c->dn_part, true);
}

// ---- the sparse step without allocation -------------------------------------------------
// A fixed device array holds the scratch of ls_sparse_ffn_step_static (activations [B, F],
// then the split down projection's parts [kDownPartsMax, B, d]).  Each GPU the library runs on
// holds its own copy until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address is resolved once per device, with that
// device current, by ls_ffn_create, and only that address is handed to kernels.
constexpr size_t kScratchFloats = (size_t)LS_STATIC_SCRATCH_BYTES / sizeof(float);
static __device__ __align__(256) float scratch[kScratchFloats];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static float* g_scratch_ptr[kMaxDevices];

// Resolve the scratch array's address on `device` (the current device) once.
static bool resolve_scratch(int device) {
    if (device < 0 || device >= kMaxDevices) return false;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[device]) return true;
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
        (void)hipGetLastError();
        return false;
    }
    g_scratch_ptr[device] = static_cast<float*>(ptr);
    return true;
}

static float* scratch_ptr(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
}

ls_status ls_sparse_ffn_step_static(ls_ffn* c, int32_t layer, const float* x_in, int32_t B,
                                    const int32_t* idx, const int32_t* count, int32_t begin,
                                    int32_t end, float* x_acc) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    if (B < 1 || B > c->desc.max_batch) return fail(c, LS_E_INVAL, "B out of range");
    const size_t need = (size_t)B * s.F + (size_t)ls::kDownPartsMax * B * s.d;
    if (need > kScratchFloats)
        return fail(c, LS_E_CAPACITY, "B * (d_ff + 8 * d_model) floats exceed the static scratch (LS_STATIC_SCRATCH_BYTES)");
    float* base = scratch_ptr(c->device);
    if (!base) return fail(c, LS_E_STATE, "static scratch of this device was not resolved");
    return sparse_step(c, layer, x_in, B, idx, count, begin, end, x_acc, base, base + (size_t)B * s.F, false);
}

ls_status ls_debug_last_activations(ls_ffn* c, float* dst, int64_t cap, int64_t* n_out) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    if (!dst || !n_out) return fail(c, LS_E_INVAL, "null pointer");
    const int64_t n = c->last_act_n;
    *n_out = n;
    if (cap < (int64_t)c->last_act_B * n) return fail(c, LS_E_INVAL, "cap too small");
    const float* src = c->last_act_src ? c->last_act_src : c->a;
    for (int b = 0; b < c->last_act_B; ++b)
        LS_HIP(c, hipMemcpyAsync(dst + (size_t)b * n, src + (size_t)b * c->shape.F, (size_t)n * sizeof(float),
                                 hipMemcpyDeviceToDevice, c->stream));
    return LS_OK;
}

// Host-resident mode: rewrite the device slot table of `layer` from the block cache, on the
// copy stream (so copies queued after it see it first) and record table_uploaded[layer], which
// every later sparse step of the layer waits for.  The pinned mirror may still feed the
// previous upload, hence the wait on the same event first.
static ls_status upload_table(ls_ffn* c, int32_t layer) {
    const Shape& s = c->shape;
    int32_t* tab = c->slot_tables_host + (size_t)layer * s.n_blk;
    LS_HIP(c, hipEventSynchronize(c->table_uploaded[layer]));
    c->bcache->slot_table(layer, tab);
    LS_HIP(c, hipMemcpyAsync(c->slot_tables + (size_t)layer * s.n_blk, tab, (size_t)s.n_blk * sizeof(int32_t),
                             hipMemcpyHostToDevice, c->copy_stream));
    LS_HIP(c, hipEventRecord(c->table_uploaded[layer], c->copy_stream));
    return LS_OK;
}

// Host-resident request (validated by the caller): place idx_host[0..n) of `layer` in the block
// cache and queue the misses' copies in n_stages stages.  The copy stream first waits for the
// latest compute of every layer that held a reassigned slot and of `layer` itself (whose slot
// table it rewrites); compute of other layers keeps running under the copies.  The stages of
// the latest request of a layer are what its sparse steps wait for (earlier requests' copies
// precede them on the copy stream).  copied (may be null) receives the blocks copied.
// With a nonzero arrive_tag (for the stage-consuming kernel) the tag is written into the
// layer's arrival word of stage 0 and of every later stage that copies blocks, once its
// copies are done; wait_on[s] receives the word stage s must wait for (the last one written
// at or before it), and the request records one event after all its stages instead of one
// per stage.
static ls_status stream_request(ls_ffn* c, int32_t layer, const int32_t* idx_host, int32_t n, int32_t n_stages,
                                ls_stream_stats* stats, std::vector<int32_t>* copied, int protect_layer = -1,
                                uint32_t arrive_tag = 0, uint8_t* wait_on = nullptr) {
    const Shape& s = c->shape;
    if (n > c->bcache->slots()) return fail(c, LS_E_CAPACITY, "request exceeds the HBM cache slots");
    std::vector<ls::BlockCache::Fill> fills;
    ls::BlockCache::Result res = c->bcache->request(layer, idx_host, n, &fills, protect_layer);
    if (!res.ok) return fail(c, LS_E_CAPACITY, "cache could not place the request");
    {
        std::vector<uint8_t> wait((size_t)c->desc.n_layers, 0);
        wait[(size_t)layer] = 1;
        for (const auto& f : fills)
            if (f.evicted_layer >= 0) wait[(size_t)f.evicted_layer] = 1;
        for (int l = 0; l < c->desc.n_layers; ++l)
            if (wait[(size_t)l] && c->layer_done_recorded[(size_t)l])
                LS_HIP(c, hipStreamWaitEvent(c->copy_stream, c->layer_done[(size_t)l], 0));
        // Tables first, all before any copy: every other layer that lost a slot gets a table
        // without that block (a block not in the cache contributes nothing), and this layer's
        // table only changes entries of blocks filled below.  No compute queued so far reads
        // the slots being reassigned (the copy stream waited for it), and later steps of those
        // layers wait for their new table.
        for (int l = 0; l < c->desc.n_layers; ++l)
            if (wait[(size_t)l] && l != layer) {
                ls_status st = upload_table(c, l);
                if (st != LS_OK) return st;
            }
    }
    {
        ls_status st = upload_table(c, layer);
        if (st != LS_OK) return st;
    }
    auto& events = c->stage_events[layer];
    auto& ranges = c->stage_ranges[layer];
    while ((int)events.size() < n_stages) {
        hipEvent_t e;
        LS_HIP(c, hipEventCreateWithFlags(&e, hipEventDisableTiming));
        events.push_back(e);
    }
    ranges.clear();
    size_t fi = 0;
    const uint8_t* layer_host = c->host_blocks[layer];
    int written = 0;
    // the second copy stream starts after everything queued on the first (the waits and table
    // uploads above included)
    if (!fills.empty()) {
        LS_HIP(c, hipEventRecord(c->copy_fork, c->copy_stream));
        LS_HIP(c, hipStreamWaitEvent(c->copy_stream2, c->copy_fork, 0));
    }
    for (int sidx = 0; sidx < n_stages; ++sidx) {
        const int lo = (int)((int64_t)sidx * n / n_stages), hi = (int)((int64_t)(sidx + 1) * n / n_stages);
        const size_t fi0 = fi;
        for (; fi < fills.size() && fills[fi].pos < hi; ++fi) {
            const auto& f = fills[fi];
            LS_HIP(c, hipMemcpyAsync(c->cache + (size_t)f.slot * c->block_bytes,
                                     layer_host + (size_t)f.block * c->block_bytes, c->block_bytes,
                                     hipMemcpyHostToDevice, (fi - fi0) % 2 ? c->copy_stream2 : c->copy_stream));
            if (copied) copied->push_back(f.block);
        }
        if (fi - fi0 > 1) {  // the stage's copies on the second stream are done before it is signalled
            LS_HIP(c, hipEventRecord(c->copy_join, c->copy_stream2));
            LS_HIP(c, hipStreamWaitEvent(c->copy_stream, c->copy_join, 0));
        }
        if (!arrive_tag) {
            LS_HIP(c, hipEventRecord(events[sidx], c->copy_stream));
            ranges.emplace_back(lo, hi);
            continue;
        }
        if (sidx == 0 || fi > fi0) {
            LS_HIP(c, hipStreamWriteValue32(c->copy_stream, c->arrive + (size_t)layer * ls::kMaxStages + sidx,
                                            arrive_tag, 0));
            written = sidx;
        }
        wait_on[sidx] = (uint8_t)written;
    }
    if (arrive_tag) {  // per-call steps on this layer wait for the whole request
        LS_HIP(c, hipEventRecord(events[0], c->copy_stream));
        ranges.emplace_back(0, n);
    }
    c->streamed[layer] = 1;
    if (stats) {
        stats->hits = res.hits;
        stats->misses = res.misses;
        stats->bytes = (int64_t)res.misses * (int64_t)c->block_bytes;
        stats->evictions = res.evictions;
    }
    return LS_OK;
}

ls_status ls_stream_weights(ls_ffn* c, int32_t layer, const int32_t* idx_host, int32_t n,
                            int32_t n_stages, ls_stream_stats* stats) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    if (layer < 0 || layer >= c->desc.n_layers) return fail(c, LS_E_INVAL, "layer out of range");
    if (n < 0 || (n > 0 && !idx_host)) return fail(c, LS_E_INVAL, "bad idx_host / n");
    if (n_stages < 1) return fail(c, LS_E_INVAL, "n_stages must be >= 1");
    for (int i = 0; i < n; ++i)
        if (idx_host[i] < 0 || idx_host[i] >= s.n_blk) return fail(c, LS_E_INVAL, "block id out of range");
    if (!c->is_set[layer]) return fail(c, LS_E_STATE, "layer weights not set");
    if (c->desc.residency == LS_WEIGHTS_HBM) {
        if (stats) *stats = ls_stream_stats{n, 0, 0, 0};
        return LS_OK;
    }
    return stream_request(c, layer, idx_host, n, n_stages, stats, nullptr);
}

// Device list -> host: copies n ids after the work queued on the compute stream and waits.
static ls_status read_list(ls_ffn* c, const int32_t* dev, int32_t n, int32_t* host) {
    LS_HIP(c, hipMemcpyAsync(host, dev, (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost, c->stream));
    LS_HIP(c, hipStreamSynchronize(c->stream));
    return LS_OK;
}

ls_status ls_set_hash_predictor(ls_ffn* c, int32_t layer, const ls_hash_weights* w) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    if (layer < 0 || layer >= c->desc.n_layers) return fail(c, LS_E_INVAL, "layer out of range");
    if (!w || !w->w1 || !w->w_bin || !w->tables || !w->head) return fail(c, LS_E_INVAL, "null pointer");
    if (c->hash.empty()) c->hash.assign((size_t)c->desc.n_layers, ls::HashDev{});
    ls::HashDev& h = c->hash[(size_t)layer];
    const size_t n_w1 = (size_t)s.d * 8 * sizeof(float), n_wb = 4 * 8 * 8 * sizeof(uint32_t),
                 n_tb = 4 * 256 * 8 * sizeof(uint32_t), n_hd = 256 * (size_t)s.n_blk;
    if (!h.w1) {
        uint8_t* p = nullptr;
        if (hipMalloc((void**)&p, n_w1 + n_wb + n_tb + n_hd) != hipSuccess) {
            (void)hipGetLastError();
            return fail(c, LS_E_NOMEM, "hashing predictor allocation failed");
        }
        h.w1 = reinterpret_cast<float*>(p);
        h.w_bin = reinterpret_cast<uint32_t*>(p + n_w1);
        h.tables = reinterpret_cast<uint32_t*>(p + n_w1 + n_wb);
        h.head = p + n_w1 + n_wb + n_tb;
    }
    LS_HIP(c, hipMemcpy(h.w1, w->w1, n_w1, hipMemcpyHostToDevice));
    LS_HIP(c, hipMemcpy(h.w_bin, w->w_bin, n_wb, hipMemcpyHostToDevice));
    LS_HIP(c, hipMemcpy(h.tables, w->tables, n_tb, hipMemcpyHostToDevice));
    LS_HIP(c, hipMemcpy(h.head, w->head, n_hd, hipMemcpyHostToDevice));
    return LS_OK;
}

ls_status ls_hash_predict(ls_ffn* c, int32_t layer, const float* x, int32_t B, float* scores) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    if (layer < 0 || layer >= c->desc.n_layers) return fail(c, LS_E_INVAL, "layer out of range");
    if (!x || !scores) return fail(c, LS_E_INVAL, "null pointer");
    if (B < 1 || B > c->desc.max_batch) return fail(c, LS_E_INVAL, "B out of range");
    if (c->hash.empty() || !c->hash[(size_t)layer].w1) return fail(c, LS_E_STATE, "no hashing predictor for this layer");
    const ls::HashDev& h = c->hash[(size_t)layer];
    LS_HIP(c, timed(c, LS_K_HASH, [&] { return ls::launch_hash_predict(s.d, s.n_blk, x, B, h, scores, c->stream); }));
    return LS_OK;
}

// One launch of the stage-consuming kernel for `layer` (its list is in c->idx, its copies and
// arrival words queued with `tag`).  Every earlier consumer launch on the stream has finished
// by now (the host read back a list enqueued after it), so its status word is final.
static ls_status launch_stage_consumer(ls_ffn* c, int32_t layer, const float* x_in, float* x_out, int32_t n,
                                       int32_t n_stages, uint32_t tag, const uint8_t* wait_on) {
    const Shape& s = c->shape;
    const size_t L = (size_t)c->desc.n_layers;
    volatile uint32_t* status = c->stage_done + L * ls::kMaxStages;
    if (*status) return fail(c, LS_E_DEVICE, "a bounded wait in the stage-consuming kernel timed out");
    ls::StageArgs a{};
    a.blocks = c->cache;
    a.block_bytes = c->block_bytes;
    a.slot_table = c->slot_tables + (size_t)layer * s.n_blk;
    a.bias = c->dev[layer].bias;
    a.thresh = c->dev[layer].threshold;
    a.x_in = x_in;
    a.x_acc = x_out;
    a.a_buf = c->a;
    a.idx = c->idx;
    a.n = n;
    a.K = n_stages;
    a.d = s.d;
    a.blk = s.blk;
    a.n_blk = s.n_blk;
    a.F = s.F;
    a.arrive = c->arrive + (size_t)layer * ls::kMaxStages;
    a.done = c->stage_done + (size_t)layer * ls::kMaxStages;
    a.cnt = c->stage_cnt;
    a.status = c->stage_done + L * ls::kMaxStages;
    a.tag = tag;
    for (int i = 0; i < n_stages; ++i) a.wait_on[i] = wait_on[i];
    a.limit = (uint64_t)c->stage_wait_us * 100u;  // wall-clock ticks at 100 MHz
    LS_HIP(c, timed(c, LS_K_STAGE, [&] { return ls::launch_stage_consumer(s, a, c->n_wg, c->cooperative != 0, c->stream); }));
    LS_HIP(c, hipEventRecord(c->layer_done[(size_t)layer], c->stream));
    c->layer_done_recorded[(size_t)layer] = 1;
    c->last_act_n = (int64_t)n * s.blk;
    c->last_act_B = 1;
    c->last_act_src = c->a;
    return LS_OK;
}

ls_status ls_decode_step_streamed(ls_ffn* c, float* x, int32_t k, int32_t n_stages, int32_t mode,
                                  int32_t k_spec, ls_stream_report* report) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    const int L = c->desc.n_layers, nb = s.n_blk;
    if (!x) return fail(c, LS_E_INVAL, "null pointer");
    if (c->desc.residency != LS_WEIGHTS_HOST) return fail(c, LS_E_UNSUPPORTED, "needs host-resident weights");
    if (k < 1 || k > nb) return fail(c, LS_E_INVAL, "k must be in 1..n_blk");
    if (n_stages < 1) return fail(c, LS_E_INVAL, "n_stages must be >= 1");
    if (mode < LS_PREFETCH_NONE || mode > LS_PREFETCH_REFINE) return fail(c, LS_E_INVAL, "unknown prefetch mode");
    if (mode != LS_PREFETCH_NONE && (k_spec < 1 || k_spec > nb)) return fail(c, LS_E_INVAL, "k_spec must be in 1..n_blk");
    const bool flags = c->stream_sync == 1;
    if (flags && mode == LS_PREFETCH_REFINE)
        return fail(c, LS_E_UNSUPPORTED, "refined prefetch needs per-stage launches (LS_CFG_STREAM_SYNC 0 or 2)");
    if (flags && n_stages > ls::kMaxStages) return fail(c, LS_E_INVAL, "n_stages exceeds 64 with device flags");
    for (int l = 0; l < L; ++l)
        if (!c->is_set[l]) return fail(c, LS_E_STATE, "layer weights not set");
    ls_stream_report rep{};
    const int64_t bb = (int64_t)c->block_bytes;
    int32_t* fin_h = c->idx_pinned;                      // the current layer's final list
    int32_t* spec_h[2] = {c->idx_pinned + nb, c->idx_pinned + 2 * (size_t)nb};
    int32_t* spec_d[2] = {c->spec_idx, c->spec_idx + nb};
    int32_t* spec_cnt = c->spec_idx + 2 * (size_t)nb;
    float* cur = x;
    float* nxt = c->xbuf;
    std::vector<int32_t> fin((size_t)k), spec_copied;
    // final list of layer 0
    if ((st = ls_predict(c, 0, cur, 1, c->scores)) != LS_OK) return st;
    if ((st = ls_select_blocks(c, c->scores, 1, LS_SEL_TOPK, k, 0.f, 0, k, c->idx, c->count)) != LS_OK) return st;
    if ((st = read_list(c, c->idx, k, fin_h)) != LS_OK) return st;
    for (int l = 0; l < L; ++l) {
        const bool next = l + 1 < L;
        std::copy(fin_h, fin_h + k, fin.begin());
        ls_stream_stats ss{};
        uint8_t wait_on[ls::kMaxStages] = {};
        uint32_t tag = 0;
        if (flags) {
            tag = ++c->stage_tag;
            if (tag == 0) tag = ++c->stage_tag;
            c->layer_tag[(size_t)l] = tag;
            c->layer_stages[(size_t)l] = n_stages;
        }
        if ((st = stream_request(c, l, fin.data(), k, n_stages, &ss, nullptr, -1, tag, wait_on)) != LS_OK) return st;
        rep.final_bytes += (int64_t)k * bb;
        rep.late_bytes += ss.bytes;
        spec_copied.clear();
        // one speculative list of layer l+1 from the device list in spec_d[b]: read back and
        // request the blocks not yet resident, protecting layer l's blocks (its stages may
        // still be queued)
        auto prefetch = [&](int b) -> ls_status {
            LS_HIP(c, hipEventSynchronize(c->spec_read[b]));
            ls_stream_stats sp{};
            ls_status r = stream_request(c, l + 1, spec_h[b], k_spec, 1, &sp, &spec_copied, l);
            if (r == LS_OK) rep.spec_bytes += sp.bytes;
            return r;
        };
        auto speculate = [&](const float* feat, int b) -> ls_status {
            ls_status r = ls_predict(c, l + 1, feat, 1, c->scores);
            if (r == LS_OK) r = ls_select_blocks(c, c->scores, 1, LS_SEL_TOPK, k_spec, 0.f, 0, k_spec, spec_d[b], spec_cnt + b);
            if (r == LS_OK && (hipMemcpyAsync(spec_h[b], spec_d[b], (size_t)k_spec * sizeof(int32_t),
                                              hipMemcpyDeviceToHost, c->stream) != hipSuccess ||
                               hipEventRecord(c->spec_read[b], c->stream) != hipSuccess))
                r = fail(c, LS_E_DEVICE, "list read-back failed");
            return r;
        };
        if (next && mode == LS_PREFETCH_ONESHOT) {
            if ((st = speculate(cur, 0)) != LS_OK || (st = prefetch(0)) != LS_OK) return st;
        }
        int pending = -1;  // a refined list read back but not yet requested
        if (flags && (st = launch_stage_consumer(c, l, cur, nxt, k, n_stages, tag, wait_on)) != LS_OK) return st;
        for (int j = 0; j < (flags ? 0 : n_stages); ++j) {
            const int lo = (int)((int64_t)j * k / n_stages), hi = (int)((int64_t)(j + 1) * k / n_stages);
            if (hi > lo || j == 0)
                if ((st = ls_sparse_ffn_step(c, l, cur, 1, c->idx, c->count, lo, hi, nxt)) != LS_OK) return st;
            if (c->stream_sync == 2) LS_HIP(c, hipStreamSynchronize(c->stream));  // host waits for every stage
            if (next && mode == LS_PREFETCH_REFINE) {
                // x~^(j+1) is in nxt: score layer l+1 on it; the list of the previous stage is
                // requested meanwhile (the host waits for it while this stage runs)
                if ((st = speculate(nxt, j & 1)) != LS_OK) return st;
                if (pending >= 0 && (st = prefetch(pending)) != LS_OK) return st;
                pending = j & 1;
            }
        }
        if (pending >= 0 && (st = prefetch(pending)) != LS_OK) return st;
        if (next) {
            // layer l+1's final list from its complete input
            if ((st = ls_predict(c, l + 1, nxt, 1, c->scores)) != LS_OK) return st;
            if ((st = ls_select_blocks(c, c->scores, 1, LS_SEL_TOPK, k, 0.f, 0, k, c->idx, c->count)) != LS_OK) return st;
            if ((st = read_list(c, c->idx, k, fin_h)) != LS_OK) return st;
            for (int32_t b : spec_copied)
                if (std::find(fin_h, fin_h + k, b) == fin_h + k) rep.wasted_bytes += bb;
        }
        std::swap(cur, nxt);
    }
    if (cur != x) LS_HIP(c, hipMemcpyAsync(x, cur, (size_t)s.d * sizeof(float), hipMemcpyDeviceToDevice, c->stream));
    rep.copied_bytes = rep.late_bytes + rep.spec_bytes;
    if (report) *report = rep;
    return LS_OK;
}

ls_status ls_decode_step(ls_ffn* c, float* x, int32_t B, int32_t k) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    if (!x) return fail(c, LS_E_INVAL, "null pointer");
    if (B < 1 || B > c->desc.max_batch) return fail(c, LS_E_INVAL, "B out of range");
    if (k < 1 || k > s.n_blk) return fail(c, LS_E_INVAL, "k must be in 1..n_blk");
    for (int l = 0; l < c->desc.n_layers; ++l)
        if (!c->is_set[l]) return fail(c, LS_E_STATE, "layer weights not set");
    if (c->desc.residency != LS_WEIGHTS_HBM)
        return fail(c, LS_E_UNSUPPORTED, "ls_decode_step needs HBM-resident weights; use the per-layer calls");
    if (c->decode_path != 1) {
        int kp = c->spec_blocks > 0 ? c->spec_blocks : k + (k + 3) / 4;
        kp = std::min(kp, ls::fused_max_spec(s, c->n_wg));
        kp = std::max(kp, k);
        const ls::FusedSupport sup = ls::fused_supported(s, B, k, kp, c->n_wg, c->desc.n_layers);
        if (sup.ok) {
            if (c->epoch == 0xffffffffu) {  // epoch tags wrap: clear the mailboxes first
                LS_HIP(c, hipStreamSynchronize(c->stream));
                LS_HIP(c, hipMemset(c->mailbox, 0, c->mailbox_words * sizeof(uint64_t)));
                LS_HIP(c, empty_bare_words(c));
                c->epoch = 0;
            }
            ls::FusedArgs a{};
            a.layers = c->layer_tab;
            a.L = c->desc.n_layers;
            a.d = s.d;
            a.nb = s.n_blk;
            a.blk = s.blk;
            a.F = s.F;
            a.k = k;
            a.kp = kp;
            a.prenorm = s.prenorm;
            a.block_bytes = c->block_bytes;
            a.x = x;
            const size_t L = (size_t)c->desc.n_layers;
            a.xmb = c->mailbox;
            a.smb = a.xmb + L * s.d;
            a.amb = a.smb + L * ls::fused_score_words(s);
            a.tag = ++c->epoch;
            a.err = c->dev_err;
            a.trace = c->trace_wg >= 0 ? c->trace : nullptr;
            a.trace_wg = c->trace_wg;
            LS_HIP(c, timed(c, LS_K_DECODE, [&] { return ls::launch_decode_fused(s, a, c->n_wg, c->cooperative != 0, c->stream); }));
            c->last_fused = true;
            c->last_act_n = 0;
            c->last_act_B = 0;
            return LS_OK;
        }
        if (c->decode_path == 2) return fail(c, LS_E_UNSUPPORTED, std::string("fused decode: ") + sup.why);
    }
    c->last_fused = false;
    const int cap = B > 1 ? std::min(s.n_blk, B * k) : k;
    float* cur = x;
    float* nxt = c->xbuf;
    for (int l = 0; l < c->desc.n_layers; ++l) {
        const ls::LayerDev& L = c->dev[l];
        st = predictor_gemv(c, L, cur, B, c->scores);
        if (st != LS_OK) return st;
        if (ls::gateup_select_ok(s, B, k)) {
            // batch 1: the selection runs inside the gate/up launch (one launch fewer per layer)
            LS_HIP(c, timed(c, LS_K_GATEUP, [&] {
                return ls::launch_gateup_select(s, L, cur, c->scores, k, c->idx, c->count, c->a, c->stream);
            }));
        } else {
            LS_HIP(c, timed(c, LS_K_SELECT, [&] {
                return ls::launch_select(c->scores, B, s.n_blk, LS_SEL_TOPK, k, 0.f, 1, cap, c->idx, c->count,
                                         c->stream);
            }));
            LS_HIP(c, timed(c, LS_K_GATEUP, [&] {
                return ls::launch_gateup(s, L, nullptr, cur, B, c->idx, c->count, 0, cap, c->a, c->stream);
            }));
        }
        LS_HIP(c, timed(c, LS_K_DOWN, [&] { return ls::launch_down(s, L, nullptr, c->a, B, c->idx, c->count, 0, cap, cur, nxt, c->dn_part, c->stream); }));
        std::swap(cur, nxt);
    }
    if (cur != x)
        LS_HIP(c, hipMemcpyAsync(x, cur, (size_t)B * s.d * sizeof(float), hipMemcpyDeviceToDevice, c->stream));
    c->last_act_n = (int64_t)cap * s.blk;
    c->last_act_B = B;
    return LS_OK;
}

ls_status ls_configure(ls_ffn* c, int32_t key, int64_t value) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    if (key == LS_CFG_DECODE_PATH) {
        if (value < 0 || value > 2) return fail(c, LS_E_INVAL, "decode path must be 0, 1 or 2");
        c->decode_path = (int)value;
        return LS_OK;
    }
    if (key == LS_CFG_TRACE_WG) {
        if (value < -1 || value >= c->n_wg) return fail(c, LS_E_INVAL, "trace workgroup out of range");
        if (value >= 0 && !c->trace) {
            const size_t n = (size_t)c->desc.n_layers * ls::kTracePoints;
            LS_HIP(c, hipMalloc(reinterpret_cast<void**>(&c->trace), n * sizeof(uint64_t)));
            LS_HIP(c, hipMemset(c->trace, 0, n * sizeof(uint64_t)));
        }
        c->trace_wg = (int)value;
        return LS_OK;
    }
    if (key == LS_CFG_BATCH_MFMA) {
        if (value != 0 && value != 1) return fail(c, LS_E_INVAL, "batch MFMA must be 0 or 1");
        c->shape.batch_mfma = (int)value;
        return LS_OK;
    }
    if (key == LS_CFG_STREAM_SYNC) {
        if (value < 0 || value > 2) return fail(c, LS_E_INVAL, "stream sync must be 0, 1 or 2");
        if (value == 1 && !c->arrive) {
            const size_t L = (size_t)c->desc.n_layers, words = L * ls::kMaxStages;
            c->arrive_bytes = words * sizeof(uint32_t);
            c->arrive = arrive_take(c->arrive_bytes);
            if (!c->arrive) return fail(c, LS_E_NOMEM, "fine-grained arrival words could not be allocated");
            LS_HIP(c, hipMemset(c->arrive, 0, c->arrive_bytes));
            if (hipHostMalloc(reinterpret_cast<void**>(&c->stage_done), (words + 1) * sizeof(uint32_t),
                              hipHostMallocCoherent) != hipSuccess) {
                (void)hipGetLastError();
                c->stage_done = nullptr;
                return fail(c, LS_E_NOMEM, "pinned done words could not be allocated");
            }
            std::memset(c->stage_done, 0, (words + 1) * sizeof(uint32_t));
            if (dmalloc(&c->stage_cnt, 2 * (size_t)ls::kMaxStages) != hipSuccess) {
                (void)hipGetLastError();
                return fail(c, LS_E_NOMEM, "stage counters could not be allocated");
            }
            LS_HIP(c, hipMemset(c->stage_cnt, 0, 2 * (size_t)ls::kMaxStages * sizeof(uint32_t)));
            c->layer_tag.assign(L, 0u);
            c->layer_stages.assign(L, 0);
        }
        c->stream_sync = (int)value;
        return LS_OK;
    }
    if (key == LS_CFG_STAGE_WAIT_US) {
        if (value < 1 || value > 60000000) return fail(c, LS_E_INVAL, "stage wait limit must be 1 us .. 60 s");
        c->stage_wait_us = value;
        return LS_OK;
    }
    if (key == LS_CFG_ZERO_SKIP) {
        if (value != 0 && value != 1) return fail(c, LS_E_INVAL, "zero skip must be 0 or 1");
        c->shape.zero_skip = (int)value;
        return LS_OK;
    }
    if (key == LS_CFG_COOPERATIVE) {
        if (value != 0 && value != 1) return fail(c, LS_E_INVAL, "cooperative must be 0 or 1");
        c->cooperative = (int)value;
        return LS_OK;
    }
    if (key == LS_CFG_SPEC_BLOCKS) {
        if (value < 0 || value > c->shape.n_blk) return fail(c, LS_E_INVAL, "speculative width out of range");
        c->spec_blocks = (int)value;
        return LS_OK;
    }
    return fail(c, LS_E_INVAL, "unknown configuration key");
}

ls_status ls_debug_decode_trace(ls_ffn* c, int32_t layer, float* x_in, float* scores) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    const Shape& s = c->shape;
    if (layer < 0 || layer >= c->desc.n_layers) return fail(c, LS_E_INVAL, "layer out of range");
    if (!c->last_fused) return fail(c, LS_E_STATE, "the last ls_decode_step did not run the fused kernel");
    const size_t L = (size_t)c->desc.n_layers;
    const uint64_t* xmb = c->mailbox;
    const uint64_t* smb = xmb + L * s.d;
    if (x_in) {
        if (layer == 0) return fail(c, LS_E_INVAL, "layer 0 input is the caller's own x");
        // the last launch's half of the input rows: bare fp32 words
        const float* rows = reinterpret_cast<const float*>(c->mailbox) + (size_t)(c->epoch & 1u) * L * s.d;
        LS_HIP(c, hipMemcpyAsync(x_in, rows + (size_t)layer * s.d, (size_t)s.d * sizeof(float),
                                 hipMemcpyDeviceToDevice, c->stream));
    }
    if (scores)
        LS_HIP(c, ls::launch_untag(smb + (size_t)layer * ls::fused_score_words(s), s.n_blk, ls::kScoreStride, scores, c->stream));
    return LS_OK;
}

ls_status ls_debug_phase_trace(ls_ffn* c, int64_t* host_out, int64_t cap, int64_t* n) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    if (!host_out || !n) return fail(c, LS_E_INVAL, "null pointer");
    const int64_t total = (int64_t)c->desc.n_layers * ls::kTracePoints;
    *n = total;
    if (!c->trace) return fail(c, LS_E_STATE, "tracing was never enabled (LS_CFG_TRACE_WG)");
    if (cap < total) return fail(c, LS_E_INVAL, "cap too small");
    LS_HIP(c, hipStreamSynchronize(c->stream));
    LS_HIP(c, hipMemcpy(host_out, c->trace, (size_t)total * sizeof(int64_t), hipMemcpyDeviceToHost));
    return LS_OK;
}

ls_status ls_debug_stages_done(ls_ffn* c, int32_t layer, int32_t* n_done) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    if (!n_done) return fail(c, LS_E_INVAL, "null pointer");
    if (layer < 0 || layer >= c->desc.n_layers) return fail(c, LS_E_INVAL, "layer out of range");
    if (!c->stage_done || !c->layer_tag[(size_t)layer]) return fail(c, LS_E_STATE, "no flagged step has run this layer");
    LS_HIP(c, hipStreamSynchronize(c->stream));
    const volatile uint32_t* w = c->stage_done + (size_t)layer * ls::kMaxStages;
    int32_t n = 0;
    for (int sidx = 0; sidx < c->layer_stages[(size_t)layer]; ++sidx) n += w[sidx] == c->layer_tag[(size_t)layer];
    *n_done = n;
    return LS_OK;
}

ls_status ls_measure_read_bandwidth(ls_ffn* c, const void* buf, int64_t bytes, int32_t reps,
                                    double* best_gbs, double* median_gbs) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    if (!buf || !best_gbs || !median_gbs) return fail(c, LS_E_INVAL, "null pointer");
    if (bytes < (1 << 20) || bytes % 16) return fail(c, LS_E_INVAL, "bytes must be >= 1 MiB and a multiple of 16");
    if (reps < 1 || reps > 1000) return fail(c, LS_E_INVAL, "reps must be in 1..1000");
    int dev = 0, cus = 0;
    LS_HIP(c, hipGetDevice(&dev));
    LS_HIP(c, hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    const int grid = 8 * std::max(cus, 1);
    uint32_t* out = nullptr;
    if (hipMalloc(reinterpret_cast<void**>(&out), (size_t)grid * 4 * sizeof(uint32_t)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(c, LS_E_NOMEM, "device allocation for the read probe failed");
    }
    std::vector<hipEvent_t> ev((size_t)reps + 1, nullptr);
    hipError_t e = hipSuccess;
    for (auto& x : ev)
        if (e == hipSuccess) e = hipEventCreate(&x);
    // one untimed pass so the first timed one does not pay for first-touch work
    if (e == hipSuccess) e = ls::launch_read_probe(buf, (size_t)bytes, out, grid, c->stream);
    if (e == hipSuccess) e = hipEventRecord(ev[0], c->stream);
    for (int r = 0; r < reps && e == hipSuccess; ++r) {
        e = ls::launch_read_probe(buf, (size_t)bytes, out, grid, c->stream);
        if (e == hipSuccess) e = hipEventRecord(ev[(size_t)r + 1], c->stream);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    std::vector<double> gbs;
    for (int r = 0; r < reps && e == hipSuccess; ++r) {
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, ev[(size_t)r], ev[(size_t)r + 1]);
        if (e == hipSuccess) gbs.push_back((double)bytes / (ms * 1e-3) / 1e9);
    }
    for (auto x : ev)
        if (x) (void)hipEventDestroy(x);
    const hipError_t ef = hipFree(out);
    LS_HIP(c, e);
    LS_HIP(c, ef);
    std::sort(gbs.begin(), gbs.end());
    *best_gbs = gbs.back();
    *median_gbs = gbs[gbs.size() / 2];
    return LS_OK;
}

#ifndef LS_BUILD_DIGEST
#define LS_BUILD_DIGEST "unknown"
#endif
const char* ls_build_digest(void) { return LS_BUILD_DIGEST; }

ls_status ls_ffn_sync(ls_ffn* c) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    LS_HIP(c, hipStreamSynchronize(c->stream));
    int e = 0;
    LS_HIP(c, hipMemcpy(&e, c->dev_err, sizeof e, hipMemcpyDeviceToHost));
    if (e) return fail(c, LS_E_DEVICE, "a bounded wait in the fused decode kernel timed out");
    if (c->stage_done && c->stage_done[(size_t)c->desc.n_layers * ls::kMaxStages])
        return fail(c, LS_E_DEVICE, "a bounded wait in the stage-consuming kernel timed out");
    return LS_OK;
}

ls_status ls_set_kernel_timing(ls_ffn* c, int32_t enable) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    // 1 (the bit of the prenorm id, which launches nothing) and -1: every kernel
    c->timing = (enable == 1 || enable == -1) ? ~0u : (uint32_t)enable;
    return LS_OK;
}

ls_status ls_kernel_timing(ls_ffn* c, int32_t kernel, int32_t reset, double* total_ms,
                           int64_t* launches) {
    ls_status st = check_ctx(c);
    if (st != LS_OK) return st;
    if (kernel < 0 || kernel >= LS_K_COUNT) return fail(c, LS_E_INVAL, "kernel id out of range");
    LS_HIP(c, fold_timing(c));
    if (total_ms) *total_ms = c->kernel_ms[kernel];
    if (launches) *launches = c->kernel_launches[kernel];
    if (reset)
        for (int i = 0; i < LS_K_COUNT; ++i) {
            c->kernel_ms[i] = 0.0;
            c->kernel_launches[i] = 0;
        }
    return LS_OK;
}

}  // extern "C"
