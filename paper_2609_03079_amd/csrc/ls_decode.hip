// ls_decode.hip - one decode step of the whole FFN stack in one persistent launch.
//
// Speculate-and-refine on the GPU (Sec. 2.1, Eq. 2): while layer l runs, the
// input of layer l (available before layer l's own FFN output) also drives a
// speculative prediction of layer l+1's priority list; the weight blocks of
// that list are streamed from HBM into registers while layer l finishes, and
// layer l+1 computes only its exact top-k blocks (taken from the registers,
// or loaded on demand for the few the speculation missed).  The result is the
// exact composition predict -> select -> gate/up -> down of every layer; only
// the time at which bytes are read changes.
//
// One workgroup per compute unit (cooperative launch, all resident).  Wave 0
// of every workgroup is the control wave: it waits for values published by
// other workgroups and publishes this workgroup's results.  Waves 1..3 are
// worker waves: they hold prefetched weights in registers and compute.  The
// control wave never has weight loads in flight, so its waits are not held up
// by the in-order completion of the workers' streaming loads.
//
// Cross-workgroup exchange: every published value is one 64-bit word
// (launch epoch << 32 | fp32 bits) written and read with agent-scope relaxed
// atomics, which are coherent across the XCDs without cache maintenance; a
// reader spins on the word until its epoch matches.  Each layer has its own
// mailbox rows, so no value is overwritten within a launch.  Every wait is
// bounded: on timeout an error flag is set and the kernel runs to completion.
//
// Per layer l (all reductions in a fixed order):
//   X   h_l = prenorm(x_l)                     (x_l from the previous layer)
//   Z   z_l = P1_l h_l, z~_{l+1} = P1_{l+1} h_l (rows of this workgroup)
//   S   s_l = P2_l z_l, s~_{l+1} = P2_{l+1} z~   (block scores of this workgroup)
//   SEL E_l = topk(s_l, k); P_{l+1} = topk(s~_{l+1}, kp)  (every workgroup)
//   GU  a_j for the neurons of E_l held in this workgroup's slots
//   D   y over E_l for this workgroup's 16-column tile; x_{l+1} = x_l + y
#include "ls_decode.h"
#include "ls_device.h"

#include <algorithm>

namespace ls {
namespace {

constexpr int kThreads = 256;           // one wave per SIMD: each wave may use 512 registers
constexpr int kWaves = kThreads / 64;
constexpr int kWorkers = kWaves - 1;    // worker waves 1..3
constexpr int kWL = kWorkers * 64;      // worker lanes
constexpr int kSlots = 2;               // neuron slots per worker wave
constexpr int kMaxP1 = 11;              // P1 wave-chunks (64 x 16 B) per worker wave (per layer)
constexpr int kDnPos = 8;               // speculative list positions per worker wave
constexpr int kDnPer = 2;               // 16-byte down chunks per lane per position
constexpr int kMaxDn = kDnPos * kDnPer;
constexpr int kMaxD = 4096;
constexpr int kMaxR = 1024;
constexpr int kMaxNb = 256;
constexpr int kMaxKp = 64;
constexpr int kMaxA = 4096;             // k * block
constexpr int kMaxRowsPerWg = 8;        // predictor rows per workgroup
constexpr int kMaxScoresPerWg = 4;
constexpr int kMaxLayers = 128;
constexpr unsigned kSpinLimit = 1u << 18;  // ~0.3 s of polling per wait

// Phase stamp of the traced workgroup (tracing aid; off when P.trace is null).
#define LS_STAMP(P, g, l, pt, cond)                                                     \
    do {                                                                                \
        if ((P).trace && (g).w == (P).trace_wg && (cond))                                \
            (P).trace[(size_t)(l) * kTracePoints + (pt)] = wall_clock64();              \
    } while (0)

// LDS-only workgroup barrier: orders LDS accesses without waiting for the
// workers' outstanding global loads.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ uint64_t mb_load(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void mb_store(uint64_t* p, uint32_t tag, float v) {
    __hip_atomic_store(p, ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(v), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// Control wave: wait until the tagged words src[0..n) all carry `tag`.  Lane l holds word
// l + 64u in v[u] (u < W, W*64 >= n; indices past n read the last word and are ignored).
// All W loads of a round are in flight together; a round re-reads every word (branch-free,
// so the loop stays small and the values stay in registers).
template <int W>
__device__ __forceinline__ void wait_words(const uint64_t* src, int n, uint32_t tag, int lane,
                                           int* err, uint64_t (&v)[W]) {
    const int last = n - 1;
    for (unsigned spins = 0;; ++spins) {
#pragma unroll
        for (int u = 0; u < W; ++u) v[u] = mb_load(src + min(u * 64 + lane, last));
        bool done = true;
#pragma unroll
        for (int u = 0; u < W; ++u) done &= (uint32_t)(v[u] >> 32) == tag;
        if (__all(done)) break;
        if (spins > kSpinLimit) {
            if (lane == 0) atomicOr(err, 1);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

__device__ __forceinline__ float word_value(uint64_t w) { return __uint_as_float((uint32_t)w); }

// Keep a prefetched register in its storage type until this point: without it the compiler
// may widen 16-bit weights to fp32 right after their load and hold twice the registers.
__device__ __forceinline__ u32x4 pin(u32x4 v) {
    asm volatile("" : "+v"(v));
    return v;
}

template <ls_dtype T>
__device__ __forceinline__ float dot_chunk(const u32x4& raw_in, const float* x) {
    constexpr int V = Wt<T>::V;
    const u32x4 raw = pin(raw_in);
    float w[V];
    Wt<T>::widen(raw, w);
    const f32x4* x4 = reinterpret_cast<const f32x4*>(x);
    float acc = 0.f;
#pragma unroll
    for (int q = 0; q < V / 4; ++q) {
        const f32x4 xv = x4[q];
        acc = fmaf(w[4 * q + 0], xv.x, acc);
        acc = fmaf(w[4 * q + 1], xv.y, acc);
        acc = fmaf(w[4 * q + 2], xv.z, acc);
        acc = fmaf(w[4 * q + 3], xv.w, acc);
    }
    return acc;
}

struct Smem {
    u32x4 p1s[2][kMaxP1 * kWorkers * 64];  // this workgroup's P1 rows of two layers (by parity)
    LayerPtrs lt[kMaxLayers];  // the layer table (LDS reads keep weight loads off the wait path)
    u32x4 p2s[2][kWL];         // this workgroup's P2 rows of two layers (by parity)
    float hs[kMaxD];
    float xt[kColTile];
    float zres[2 * kMaxRowsPerWg];
    float zall[2 * 1024];
    float sp[2][kWL];
    float sres[2 * kMaxScoresPerWg];
    alignas(16) uint64_t key[2][kMaxNb + 2];  // composite keys, padded with 0 to even length
    int E[kMaxKp];
    int Plist[2][kMaxKp];
    int slot_entry[kMaxKp];
    int slot_miss[kMaxKp];
    int missE[kMaxKp];
    int posE[kMaxNb];   // block -> position in E, or -1
    int posP[kMaxNb];   // block -> position in the current speculative list, or -1
    float a_loc[kWorkers * kSlots];
    int a_pos[kWorkers * kSlots];
    float aall[kMaxA];
    float dpart[kWL];
};

// Static shape of one launch, shared by both roles.
struct Geo {
    int w, G, L, r, nb, blk, k, kp, F;
    int RPW, P1C, CPR2, SPW, P2C, NPC, RPWmax, SPWmax;
    bool has_tile;
    uint32_t tag;
};

// Row sums shared by all eight waves: rows [0, rows) of the exact set and, unless
// skip_spec, of the speculative set (stored set_stride apart); lane-strided partial
// sums then a butterfly, a fixed order.
__device__ __forceinline__ void reduce_rows(const float* part, int set_stride, int rows, int per_row,
                                            bool skip_spec, float* res, int wave, int lane) {
    for (int m2 = wave; m2 < 2 * rows; m2 += kWaves) {
        const int set = m2 / rows, m = m2 % rows;
        if (set == 1 && skip_spec) continue;
        const float* src = part + (size_t)set * set_stride + (size_t)m * per_row;
        float acc = 0.f;
        for (int c = lane; c < per_row; c += 64) acc += src[c];
        acc = wave_sum_dpp(acc);
        if (lane == 0) res[m2] = acc;
    }
}

// Predictor projection rows of this workgroup, shared by all waves: row m (of RPW) of the
// exact set (layer l) and, unless last, of the speculative set (layer l+1), from the P1 rows
// staged in LDS and h; wave v takes rows v, v+4, ...; results in zres[set * RPW + m].
template <ls_dtype T, int CPR>
__device__ __forceinline__ void z_rows(Smem& sm, const Geo g, int l, bool last, int wave, int lane) {
    constexpr int V = Wt<T>::V;
    for (int m2 = wave; m2 < 2 * g.RPW; m2 += kWaves) {
        const int set = m2 / g.RPW, m = m2 % g.RPW;
        if (set == 1 && last) continue;
        const u32x4* row = sm.p1s[(l + set) & 1] + m * CPR;
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < CPR / 64; ++i) {
            const int c = lane + 64 * i;
            acc += dot_chunk<T>(row[c], sm.hs + c * V);
        }
        acc = wave_sum_dpp(acc);
        if (lane == 0) sm.zres[m2] = acc;
    }
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

// Top-m set of one list, run by one wave without LDS traffic.  The priority order is the
// composite key (order_key << 32 | ~index): larger first.  A bitwise search from the top
// bit finds T, the m-th largest order key (the largest T with at least m keys >= T); the
// set is every key > T plus the elements equal to T with the smallest indices.  Members
// are written to out[] in index order (the set is what matters to the fused step; its
// summation order is fixed by the slot map).  Needs 1 <= m <= n.
__device__ __forceinline__ void top_set(const uint64_t* keys, int n, int m, int* out, int lane) {
    constexpr int Q = kMaxNb / 64;
    uint32_t ok[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int i = q * 64 + lane;
        ok[q] = i < n ? (uint32_t)(keys[i] >> 32) : 0u;  // padding compares below every c >= 1
    }
    uint32_t T = 0u;
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t c = T | (1u << bit);
        int cnt = 0;
#pragma unroll
        for (int q = 0; q < Q; ++q) cnt += __popcll(__ballot(ok[q] >= c));
        if (cnt >= m) T = c;
    }
    int gt = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) gt += __popcll(__ballot(ok[q] > T));
    const int rem = m - gt;  // elements equal to T that are taken (>= 1)
    const uint64_t below = (1ull << lane) - 1ull;
    int eq_before = 0, mem_before = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int i = q * 64 + lane;
        const bool valid = i < n;
        const bool eq = valid && ok[q] == T;
        const uint64_t eqb = __ballot(eq);
        const bool mem = valid && (ok[q] > T || (eq && eq_before + __popcll(eqb & below) < rem));
        const uint64_t memb = __ballot(mem);
        if (mem) out[mem_before + __popcll(memb & below)] = i;
        eq_before += __popcll(eqb);
        mem_before += __popcll(memb);
    }
}

// Exact top-k of layer l into E (wave 0) and, unless last, the speculative top-kp of layer
// l+1 into Pn (wave 1).
__device__ __forceinline__ void rank_all(Smem& sm, const Geo g, bool last, int* Pn, int wave,
                                         int lane) {
    if (wave == 0) top_set(sm.key[0], g.nb, g.k, sm.E, lane);
    else if (wave == 1 && !last) top_set(sm.key[1], g.nb, g.kp, Pn, lane);
}

// ---------------------------------------------------------------------------------------
// Control wave: waits, publications, the slot map.
template <ls_dtype T, int NC>
__device__ __forceinline__ void control_loop(const FusedArgs P, Smem& sm, const Geo g, int lane) {
    constexpr int V = Wt<T>::V;
    constexpr int D = NC * V * 64;
    for (int l = 0; l < g.L; ++l) {
        const bool last = l == g.L - 1;
        int* Pc = sm.Plist[l & 1];
        int* Pn = sm.Plist[(l + 1) & 1];
        LS_STAMP(P, g, l, 0, lane == 0);
        // X: the layer input (layer 0's was tagged into the mailbox before the launch), the
        // RMS scale from the values in registers, h into LDS, this tile's raw x into xt.
        {
            uint64_t v[D / 64];
            wait_words<D / 64>(P.xmb + (size_t)l * D, D, g.tag, lane, P.err, v);
            float ss = 0.f;
#pragma unroll
            for (int u = 0; u < D / 64; ++u) ss = fmaf(word_value(v[u]), word_value(v[u]), ss);
            ss = wave_sum_dpp(ss);
            const float sc = P.prenorm ? 1.f / sqrtf(ss / (float)D + 1e-6f) : 1.f;
#pragma unroll
            for (int u = 0; u < D / 64; ++u) {
                const int i = u * 64 + lane;
                const float x = word_value(v[u]);
                if (g.has_tile && (i >> 4) == g.w) sm.xt[i & (kColTile - 1)] = x;
                sm.hs[i] = x * sc;
            }
        }
        LS_STAMP(P, g, l, 1, lane == 0);
        lds_barrier();  // 1: h ready (and this layer's P1 rows staged)
        z_rows<T, D / V>(sm, g, l, last, 0, lane);
        lds_barrier();  // 2: z rows of this workgroup ready
        for (int m2 = lane; m2 < 2 * g.RPW; m2 += 64) {
            const int set = m2 / g.RPW, m = m2 % g.RPW;
            if (set == 1 && last) continue;
            mb_store(P.zmb + (size_t)l * 2 * g.r + set * g.r + (g.w + g.G * m), g.tag, sm.zres[m2]);
        }
        LS_STAMP(P, g, l, 2, lane == 0);
        // S: z of every workgroup (exact, then speculative)
        {
            const int n = last ? g.r : 2 * g.r;
            uint64_t v[2 * kMaxR / 64];
            wait_words<2 * kMaxR / 64>(P.zmb + (size_t)l * 2 * g.r, n, g.tag, lane, P.err, v);
#pragma unroll
            for (int u = 0; u < 2 * kMaxR / 64; ++u) {
                const int i = u * 64 + lane;
                if (i < n) sm.zall[i] = word_value(v[u]);
            }
        }
        LS_STAMP(P, g, l, 3, lane == 0);
        lds_barrier();  // 4: z of every workgroup ready
        lds_barrier();  // 5: S partials ready
        reduce_rows(&sm.sp[0][0], kWL, g.SPW, g.CPR2, last, sm.sres, 0, lane);
        lds_barrier();  // 6: scores reduced
        for (int m2 = lane; m2 < 2 * g.SPW; m2 += 64) {
            const int set = m2 / g.SPW, m = m2 % g.SPW;
            if (set == 1 && last) continue;
            mb_store(P.smb + (size_t)l * 2 * g.nb + set * g.nb + (g.w + g.G * m), g.tag, sm.sres[m2]);
        }
        LS_STAMP(P, g, l, 4, lane == 0);
        // SEL: scores of every block (exact, then speculative) as composite keys
        // order_key(s) << 32 | ~index: distinct, larger = earlier in the priority order
        {
            const int n = last ? g.nb : 2 * g.nb;
            uint64_t v[2 * kMaxNb / 64];
            wait_words<2 * kMaxNb / 64>(P.smb + (size_t)l * 2 * g.nb, n, g.tag, lane, P.err, v);
#pragma unroll
            for (int u = 0; u < 2 * kMaxNb / 64; ++u) {
                const int i = u * 64 + lane;
                if (i < n) {
                    const int list = i >= g.nb, b = i - list * g.nb;
                    sm.key[list][b] = ((uint64_t)order_key(word_value(v[u])) << 32) |
                                      (uint64_t)(0xffffffffu - (uint32_t)b);
                }
            }
            if (lane < 2) {  // pad to even length: below every real key
                sm.key[0][g.nb + lane] = 0ull;
                sm.key[1][g.nb + lane] = 0ull;
            }
        }
        LS_STAMP(P, g, l, 5, lane == 0);
        lds_barrier();  // 7: keys ready
        LS_STAMP(P, g, l, 12, lane == 0);
        rank_all(sm, g, last, Pn, 0, lane);
        LS_STAMP(P, g, l, 13, lane == 0);
        lds_barrier();  // 8: E and the speculative list ready
        LS_STAMP(P, g, l, 14, lane == 0);
        if (l == 0) {
            sm.slot_entry[lane] = lane < g.k ? lane : -1;
            sm.slot_miss[lane] = 1;
            Pc[lane] = lane < g.k ? sm.E[lane] : -1;
        } else {
            // block -> position tables of E and of the current speculative list
            for (int b = lane; b < g.nb; b += 64) {
                sm.posE[b] = -1;
                sm.posP[b] = -1;
            }
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
            if (lane < g.k) sm.posE[sm.E[lane]] = lane;
            if (lane < g.kp) sm.posP[Pc[lane]] = lane;
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
            const int ie = lane < g.kp ? sm.posE[Pc[lane]] : -1;
            const bool miss = lane < g.k && sm.posP[sm.E[lane]] < 0;
            const bool hole = lane < g.kp && ie < 0;
            const uint64_t mm = __ballot(miss), hm = __ballot(hole);
            const uint64_t below = (1ull << lane) - 1ull;
            if (miss) sm.missE[__popcll(mm & below)] = lane;
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
            int se = -1, ms = 0;
            if (lane < g.kp) {
                if (!hole) {
                    se = ie;
                } else {
                    const int hr = __popcll(hm & below);
                    if (hr < __popcll(mm)) {
                        se = sm.missE[hr];
                        ms = 1;
                    }
                }
            }
            sm.slot_entry[lane] = se;
            sm.slot_miss[lane] = ms;
        }
        LS_STAMP(P, g, l, 6, lane == 0);
        lds_barrier();  // 9: slot map ready
        lds_barrier();  // 10: activations of this workgroup ready
        LS_STAMP(P, g, l, 7, lane == 0);
        if (lane < kWorkers * kSlots && sm.a_pos[lane] >= 0)
            mb_store(P.amb + (size_t)l * g.F + sm.a_pos[lane], g.tag, sm.a_loc[lane]);
        // D: activations of every workgroup, in priority-list order
        {
            const int n = g.k * g.blk;
            for (int base = 0; base < n; base += 32 * 64) {
                uint64_t v[32];
                wait_words<32>(P.amb + (size_t)l * g.F + base, min(n - base, 32 * 64), g.tag, lane,
                               P.err, v);
#pragma unroll
                for (int u = 0; u < 32; ++u) {
                    const int i = base + u * 64 + lane;
                    if (i < n) sm.aall[i] = word_value(v[u]);
                }
            }
        }
        LS_STAMP(P, g, l, 8, lane == 0);
        lds_barrier();  // 11: activations of every workgroup ready
        lds_barrier();  // 12: down partials ready
        LS_STAMP(P, g, l, 9, lane == 0);
        if (g.has_tile && lane < kColTile) {
            float y = 0.f;
            for (int i = 0; i < kWL / kColTile; ++i) y += sm.dpart[lane + kColTile * i];
            const float xn = sm.xt[lane] + y;
            if (last) P.x[g.w * kColTile + lane] = xn;
            else mb_store(P.xmb + (size_t)(l + 1) * D + g.w * kColTile + lane, g.tag, xn);
        }
    }
}

// ---------------------------------------------------------------------------------------
// Worker waves: registers hold the predictor factors of the next two layers and the
// speculatively prefetched blocks of the next layer.
template <ls_dtype T, ls_act A, int NC>
__device__ __forceinline__ void worker_loop(const FusedArgs P, Smem& sm, const Geo g, int wave, int lane) {
    constexpr int V = Wt<T>::V;
    constexpr int KB = Wt<T>::kBytes;
    constexpr int D = NC * V * 64;
    constexpr int CPR = D / V;
    const int wl = (wave - 1) * 64 + lane;
    const size_t row_bytes = (size_t)D * KB;
    const size_t down_off = 2 * (size_t)g.blk * row_bytes + (size_t)g.w * g.blk * kColTile * KB;
    const size_t bb = P.block_bytes;
    const u32x4 zero4 = {0u, 0u, 0u, 0u};
    // pr: P1 rows in flight (one layer), moved to LDS one layer after they were requested
    u32x4 pr[kMaxP1], p2r = zero4, gg[kSlots][NC], uu[kSlots][NC], dn[kMaxDn];
#pragma unroll
    for (int j = 0; j < kMaxP1; ++j) pr[j] = zero4;
#pragma unroll
    for (int sl = 0; sl < kSlots; ++sl)
#pragma unroll
        for (int j = 0; j < NC; ++j) gg[sl][j] = uu[sl][j] = zero4;
#pragma unroll
    for (int j = 0; j < kMaxDn; ++j) dn[j] = zero4;

    // P1 and P2 rows are stored grouped by owning workgroup (row w + G*m at storage row
    // w*RPW + m), so this workgroup's rows are one contiguous range.
    const size_t p1_off = (size_t)g.w * g.RPWmax * row_bytes;
    const size_t p2_off = (size_t)g.w * g.SPWmax * g.r * KB;
    // P1: wave-chunk wc = (wave-1) + 7j covers 64 consecutive 16-byte chunks of row wc / (CPR/64)
    auto load_p1 = [&](int layer) {
        const uint8_t* base = sm.lt[layer].p1 + p1_off;
#pragma unroll
        for (int j = 0; j < kMaxP1; ++j) {
            const int wc = (wave - 1) + kWorkers * j;
            if (wc < g.P1C) pr[j] = gload_u(base, (uint32_t)(wc * 64 + lane) * 16u);
        }
    };
    auto stash_p1 = [&](int layer) {  // pr -> LDS buffer of `layer`
        u32x4* dst = sm.p1s[layer & 1];
#pragma unroll
        for (int j = 0; j < kMaxP1; ++j) {
            const int wc = (wave - 1) + kWorkers * j;
            if (wc < g.P1C) dst[wc * 64 + lane] = pr[j];
        }
    };
    auto load_p2 = [&](int layer) {
        if (wl < g.P2C) p2r = gload_u(sm.lt[layer].p2 + p2_off, (uint32_t)wl * 16u);
    };
    auto stash_p2 = [&](int layer) {
        if (wl < g.P2C) sm.p2s[layer & 1][wl] = p2r;
    };
    // neuron slot sl of this wave: workgroup slot index i = (wave-1) + kWorkers*sl,
    // global slot t = w + G*i (list position t / blk, neuron t % blk)
    // b and q are the same in every lane of the wave (one slot per wave)
    auto load_gu = [&](int sl, int layer, int b, int q) {
        b = __builtin_amdgcn_readfirstlane(b);
        q = __builtin_amdgcn_readfirstlane(q);
        const uint8_t* base = sm.lt[layer].blocks + (size_t)b * bb;
        const uint8_t* gr = base + (size_t)q * row_bytes;
        const uint8_t* ur = base + (size_t)(g.blk + q) * row_bytes;
#pragma unroll
        for (int j = 0; j < NC; ++j) gg[sl][j] = gload_u(gr, (uint32_t)(lane + 64 * j) * 16u);
#pragma unroll
        for (int j = 0; j < NC; ++j) uu[sl][j] = gload_u(ur, (uint32_t)(lane + 64 * j) * 16u);
    };
    // down pieces: position p = (wave-1) + 7*jp of the list, chunks lane + 64*i of the piece
    auto load_down_pos = [&](int layer, int b, int jp) {
        b = __builtin_amdgcn_readfirstlane(b);
        const uint8_t* base = sm.lt[layer].blocks + (size_t)b * bb + down_off;
#pragma unroll
        for (int i = 0; i < kDnPer; ++i)
            if (lane + 64 * i < g.NPC) dn[jp * kDnPer + i] = gload_u(base, (uint32_t)(lane + 64 * i) * 16u);
    };

    load_p1(0);
    load_p2(0);

    for (int l = 0; l < g.L; ++l) {
        const bool last = l == g.L - 1;
        const int* Pn = sm.Plist[(l + 1) & 1];
        // P1 and P2 rows of layer l+1 (requested one layer ago) go to LDS before Z needs them
        if (l == 0) {
            stash_p1(0);
            stash_p2(0);
            if (g.L > 1) {
                load_p1(1);
                load_p2(1);
                stash_p1(1);
                stash_p2(1);
            }
        } else if (!last) {
            stash_p1(l + 1);
            stash_p2(l + 1);
        }
        lds_barrier();  // 1: h ready
        z_rows<T, CPR>(sm, g, l, last, wave, lane);
        lds_barrier();  // 2
        if (l + 2 < g.L) load_p1(l + 2);
        lds_barrier();  // 4: z of every workgroup ready
        if (wl < g.P2C) {
            const int c = wl % g.CPR2;
            sm.sp[0][wl] = dot_chunk<T>(sm.p2s[l & 1][wl], sm.zall + c * V);
            if (!last) sm.sp[1][wl] = dot_chunk<T>(sm.p2s[(l + 1) & 1][wl], sm.zall + g.r + c * V);
        }
        lds_barrier();  // 5
        reduce_rows(&sm.sp[0][0], kWL, g.SPW, g.CPR2, last, sm.sres, wave, lane);
        lds_barrier();  // 6
        if (l + 2 < g.L) load_p2(l + 2);
        lds_barrier();  // 7: keys ready
        rank_all(sm, g, last, const_cast<int*>(Pn), wave, lane);
        LS_STAMP(P, g, l, 15, wave == 1 && lane == 0);
        lds_barrier();  // 8
        lds_barrier();  // 9: slot map ready
        // GU
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            const int i = (wave - 1) + kWorkers * sl, t = g.w + g.G * i;
            float a_val = 0.f;
            int a_at = -1;
            if (t < g.kp * g.blk) {
                const int p = t / g.blk, q = t % g.blk;
                const int e = sm.slot_entry[p];
                if (e >= 0) {
                    const int b = sm.E[e];
                    if (sm.slot_miss[p]) load_gu(sl, l, b, q);
                    float gs = 0.f, us = 0.f;
#pragma unroll
                    for (int j = 0; j < NC; ++j) {
                        const float* hx = sm.hs + (lane + 64 * j) * V;
                        gs += dot_chunk<T>(gg[sl][j], hx);
                        us += dot_chunk<T>(uu[sl][j], hx);
                        __builtin_amdgcn_sched_barrier(0);
                    }
                    const void* bias = sm.lt[l].bias;
                    gs = wave_sum(gs) + (bias ? Wt<T>::scalar(bias, (size_t)b * g.blk + q) : 0.f);
                    us = wave_sum(us);
                    if (A == LS_ACT_REGLU) {
                        a_val = fmaxf(gs, 0.f) * us;
                    } else {
                        const float sg = gs / (1.f + expf(-gs));
                        a_val = fabsf(sg) > sm.lt[l].threshold ? sg * us : 0.f;
                    }
                    a_at = e * g.blk + q;
                }
            }
            if (lane == 0) {
                sm.a_loc[i] = a_val;
                sm.a_pos[i] = a_at;
            }
        }
        LS_STAMP(P, g, l, 10, wave == 1 && lane == 0);
        lds_barrier();  // 10
        if (!last) {
#pragma unroll
            for (int sl = 0; sl < kSlots; ++sl) {
                const int t = g.w + g.G * ((wave - 1) + kWorkers * sl);
                if (t < g.kp * g.blk) load_gu(sl, l + 1, Pn[t / g.blk], t % g.blk);
            }
        }
        lds_barrier();  // 11: activations of every workgroup ready
        if (g.has_tile) {
            float acc = 0.f;
#pragma unroll
            for (int jp = 0; jp < kDnPos; ++jp) {
                const int p = (wave - 1) + kWorkers * jp;
                const int e = p < g.kp ? sm.slot_entry[p] : -1;
                if (e >= 0) {
                    if (sm.slot_miss[p]) load_down_pos(l, sm.E[e], jp);
#pragma unroll
                    for (int i = 0; i < kDnPer; ++i) {
                        const int cc = lane + 64 * i;
                        if (cc < g.NPC) {
                            float wv[V];
                            Wt<T>::widen(pin(dn[jp * kDnPer + i]), wv);
                            const float* ap = sm.aall + e * g.blk + (cc / kColTile) * V;
#pragma unroll
                            for (int v = 0; v < V; ++v) acc = fmaf(ap[v], wv[v], acc);
                        }
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            sm.dpart[wl] = acc;
        }
        LS_STAMP(P, g, l, 11, wave == 1 && lane == 0);
        lds_barrier();  // 12
        if (!last && g.has_tile) {
#pragma unroll
            for (int jp = 0; jp < kDnPos; ++jp) {
                const int p = (wave - 1) + kWorkers * jp;
                if (p < g.kp) load_down_pos(l + 1, Pn[p], jp);
            }
        }
    }
}

template <ls_dtype T, ls_act A, int NC>
__global__ __launch_bounds__(kThreads, 1) void decode_fused_kernel(FusedArgs P) {
    constexpr int V = Wt<T>::V;
    constexpr int KB = Wt<T>::kBytes;
    constexpr int D = NC * V * 64;
    __shared__ Smem sm;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    Geo g;
    g.w = blockIdx.x;
    g.G = gridDim.x;
    g.L = P.L;
    g.r = P.r;
    g.nb = P.nb;
    g.blk = P.blk;
    g.k = P.k;
    g.kp = P.kp;
    g.F = P.F;
    g.RPW = g.w < g.r ? (g.r - 1 - g.w) / g.G + 1 : 0;
    g.RPWmax = (g.r + g.G - 1) / g.G;
    g.SPWmax = (g.nb + g.G - 1) / g.G;
    g.P1C = g.RPW * (D / V) / 64;  // 64-lane wave-chunks of this workgroup's rows
    g.CPR2 = g.r / V;
    g.SPW = g.w < g.nb ? (g.nb - 1 - g.w) / g.G + 1 : 0;
    g.P2C = g.SPW * g.CPR2;
    g.NPC = g.blk * KB;
    g.has_tile = g.w < D / kColTile;
    g.tag = P.tag;
    {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(P.layers);
        uint32_t* dst = reinterpret_cast<uint32_t*>(sm.lt);
        const int words = P.L * (int)(sizeof(LayerPtrs) / 4);
        for (int i = threadIdx.x; i < words; i += kThreads) dst[i] = src[i];
        __syncthreads();
    }
    if (wave == 0) control_loop<T, NC>(P, sm, g, lane);
    else worker_loop<T, A, NC>(P, sm, g, wave, lane);
}

// The layer-0 input as tagged mailbox words (launched before the fused kernel).
__global__ void tag_input_kernel(const float* __restrict__ x, int n, uint32_t tag, uint64_t* __restrict__ dst) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(x[i]);
}

template <ls_dtype T, ls_act A>
hipError_t launch_t(const Shape& s, const FusedArgs& a, int n_wg, hipStream_t st) {
    const int V = Wt<T>::V;
    const int nc = s.d / (V * 64);
    void* fn;
    if (nc == 2) fn = reinterpret_cast<void*>(decode_fused_kernel<T, A, 2>);
    else if (nc == 8) fn = reinterpret_cast<void*>(decode_fused_kernel<T, A, 8>);
    else return hipErrorNotSupported;
    hipLaunchKernelGGL(tag_input_kernel, dim3((s.d + 255) / 256), dim3(256), 0, st, a.x, s.d, a.tag, a.xmb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    FusedArgs copy = a;
    void* args[] = {&copy};
    return hipLaunchCooperativeKernel(fn, dim3(n_wg), dim3(kThreads), args, 0, st);
}

__global__ void untag_kernel(const uint64_t* __restrict__ src, int n, float* __restrict__ dst) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = __uint_as_float((uint32_t)src[i]);
}

}  // namespace

hipError_t launch_untag(const uint64_t* src, int n, float* dst, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(untag_kernel, dim3((n + 255) / 256), dim3(256), 0, st, src, n, dst);
    return hipGetLastError();
}

FusedSupport fused_supported(const Shape& s, int B, int k, int kp, int n_wg, int L) {
    const int V = vec_elems(s.dtype), KB = elem_size(s.dtype);
    if (B != 1) return {false, "batch > 1"};
    if (L > kMaxLayers) return {false, "more than 128 layers"};
    if (s.d % (V * 64) || (s.d / (V * 64) != 2 && s.d / (V * 64) != 8)) return {false, "d_model"};
    if (s.d > kMaxD || s.d / kColTile > n_wg) return {false, "d_model too large for one tile per workgroup"};
    if (s.r > kMaxR || s.r % V) return {false, "rank"};
    const int rpw = (s.r + n_wg - 1) / n_wg;
    if (rpw > kMaxRowsPerWg || rpw * (s.d / V) / 64 > kMaxP1 * kWorkers) return {false, "rank rows per workgroup"};
    const int spw = (s.n_blk + n_wg - 1) / n_wg;
    if (spw > kMaxScoresPerWg || spw * (s.r / V) > kWL) return {false, "scores per workgroup"};
    if ((s.d / V) % 64) return {false, "d_model"};
    if (s.n_blk > kMaxNb) return {false, "n_blk"};
    if (k < 1 || kp < k || kp > kMaxKp || kp > s.n_blk) return {false, "k / speculative width"};
    (void)0;
    if ((long)kp * s.blk > (long)kWorkers * kSlots * n_wg) return {false, "neuron slots"};
    if (s.blk * KB > 64 * kDnPer || kp > kDnPos * kWorkers) return {false, "down chunks"};
    if ((long)k * s.blk > kMaxA) return {false, "k * block"};
    return {true, ""};
}

int fused_max_spec(const Shape& s, int n_wg) {
    const long by_slots = (long)kWorkers * kSlots * n_wg / s.blk;
    long m = std::min<long>(by_slots, (long)kDnPos * kWorkers);
    m = std::min<long>(m, kMaxKp);
    return (int)std::min<long>(m, s.n_blk);
}

size_t fused_mailbox_words(const Shape& s, int L) {
    return (size_t)L * ((size_t)s.d + 2 * (size_t)s.r + 2 * (size_t)s.n_blk + (size_t)s.F);
}

hipError_t launch_decode_fused(const Shape& s, const FusedArgs& a, int n_wg, hipStream_t st) {
    const bool relu = s.act == LS_ACT_REGLU;
    switch (s.dtype) {
        case LS_F32: return relu ? launch_t<LS_F32, LS_ACT_REGLU>(s, a, n_wg, st) : launch_t<LS_F32, LS_ACT_SWIGLU_THRESH>(s, a, n_wg, st);
        case LS_F16: return relu ? launch_t<LS_F16, LS_ACT_REGLU>(s, a, n_wg, st) : launch_t<LS_F16, LS_ACT_SWIGLU_THRESH>(s, a, n_wg, st);
        case LS_BF16: return relu ? launch_t<LS_BF16, LS_ACT_REGLU>(s, a, n_wg, st) : launch_t<LS_BF16, LS_ACT_SWIGLU_THRESH>(s, a, n_wg, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace ls
