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
// reader spins on the word until its epoch matches.  The layer inputs, the largest
// exchange (every workgroup reads all d values of every layer), travel as bare 32-bit
// words instead, so a poll moves half the bytes: each launch uses one of two halves of
// the input rows (by the parity of its epoch), where an empty word holds a pattern no
// published value has (NaNs are published in their canonical form), and every
// workgroup empties its tile of the other half as it publishes, for the next launch.
// Each layer has its own mailbox rows, so no value is overwritten within a launch.
// Every wait is bounded: on timeout an error flag is set and the kernel runs to
// completion.
//
// The predictor runs in its folded form Pf = P2 P1 (fp32 [n_blk, d], Sec. 3.3.3 with the
// projection and the head applied as one matrix), so a layer needs three exchanges.
//
// Per layer l (all reductions in a fixed order):
//   X   h_l = prenorm(x_l)                     (x_l from the previous layer)
//   S   s_l = Pf_l h_l, s~_{l+1} = Pf_{l+1} h_l (block scores of this workgroup's rows)
//   SEL E_l = topk(s_l, k); P_{l+1} = topk(s~_{l+1}, kp)  (every workgroup)
//   GU  activations of every neuron of the speculative list P_l held in this workgroup's
//       slots (rows prefetched during layer l-1), published at their list positions
//       while SEL runs; an E_l block missing from P_l borrows the slots of a list
//       position outside E_l and is loaded and computed on demand
//   D   this workgroup's 16-column tile of the down partial of every list position (and
//       of every miss), from pieces staged in LDS; y = sum of the partials of E_l in E_l
//       order; x_{l+1} = x_l + y
// The weights of P_{l+1} (gate/up rows into registers, down pieces later into LDS) are
// requested as soon as P_{l+1} is ranked.
#include "ls_decode.h"
#include "ls_device.h"

#include <algorithm>
#include <type_traits>

namespace ls {
namespace {

constexpr int kThreads = 256;           // one wave per SIMD: each wave may use 512 registers
constexpr int kWaves = kThreads / 64;
constexpr int kWorkers = kWaves - 1;    // worker waves 1..3
constexpr int kWL = kWorkers * 64;      // worker lanes
constexpr int kSlots = 3;               // neuron slots per worker wave
constexpr int kDnPos = 9;               // down positions per worker wave
constexpr int kDnPer = 2;               // 16-byte down chunks per lane per position
constexpr int kMaxDn = kDnPos * kDnPer;
constexpr int kMaxDnTot = kDnPos * kWorkers;  // down positions held per workgroup
constexpr int kMaxD = 4096;
constexpr int kMaxNb = 256;
constexpr int kMaxKp = 64;
constexpr int kMaxA = 4096;             // speculative width * block
constexpr int kEarlySlots = 1;           // next-layer slots whose loads precede this layer's down rounds
constexpr int kMaxSRows = 1;            // folded predictor rows (block scores) per workgroup
constexpr int kPfPer = (kMaxD / 4 + kWL - 1) / kWL;  // 16-byte chunks of one row per worker lane
constexpr int kMaxLayers = 128;
constexpr unsigned kSpinLimit = 1u << 18;  // ~0.3 s of polling per wait
constexpr uint32_t kXEmpty = 0xffffffffu;  // an input word not yet published

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

// Same, for words at arbitrary addresses: addr(u) is this lane's u-th word; only the first
// `used` (wave-uniform) of the W loads are issued.
template <int W, typename Addr>
__device__ __forceinline__ void wait_gather(Addr addr, int used, uint32_t tag, int lane, int* err,
                                            uint64_t (&v)[W]) {
    const uint64_t* a[W];
#pragma unroll
    for (int u = 0; u < W; ++u) a[u] = addr(u);
    for (unsigned spins = 0;; ++spins) {
#pragma unroll
        for (int u = 0; u < W; ++u)
            if (u < used) v[u] = mb_load(a[u]);
        bool done = true;
#pragma unroll
        for (int u = 0; u < W; ++u)
            if (u < used) done &= (uint32_t)(v[u] >> 32) == tag;
        if (__all(done)) break;
        if (spins > kSpinLimit) {
            if (lane == 0) atomicOr(err, 1);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// Same, for words base[off(u)] with a wave-uniform base and 32-bit offsets.
template <int W, typename Off>
__device__ __forceinline__ void wait_gather_off(const uint64_t* base, Off off, int used, uint32_t tag,
                                                int lane, int* err, uint64_t (&v)[W]) {
    uint32_t o[W];
#pragma unroll
    for (int u = 0; u < W; ++u) o[u] = off(u);
    for (unsigned spins = 0;; ++spins) {
#pragma unroll
        for (int u = 0; u < W; ++u)
            if (u < used) v[u] = mb_load(base + o[u]);
        bool done = true;
#pragma unroll
        for (int u = 0; u < W; ++u)
            if (u < used) done &= (uint32_t)(v[u] >> 32) == tag;
        if (__all(done)) break;
        if (spins > kSpinLimit) {
            if (lane == 0) atomicOr(err, 1);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

__device__ __forceinline__ float word_value(uint64_t w) { return __uint_as_float((uint32_t)w); }

// Layer-input rows of the launch with epoch `tag` (half tag & 1 of the input region, [L][d]
// 32-bit words), and the bits published for v (canonical NaN, never kXEmpty).
__device__ __forceinline__ uint32_t* x_rows(const FusedArgs& P, uint32_t tag) {
    return reinterpret_cast<uint32_t*>(P.xmb) + (size_t)(tag & 1u) * P.L * P.d;
}
__device__ __forceinline__ uint32_t x_bits(float v) { return v != v ? 0x7fc00000u : __float_as_uint(v); }

// List activations of layer l of the launch with epoch `tag`: half tag & 1 of the first F
// 64-bit words of the layer's activation row, as F bare 32-bit words (the misses follow,
// tagged, at word F of the row).
__device__ __forceinline__ uint32_t* acts_rows(const FusedArgs& P, int AW, int F, int l, uint32_t tag) {
    return reinterpret_cast<uint32_t*>(P.amb + (size_t)l * AW) + (size_t)(tag & 1u) * F;
}

// Wait until the bare words src[0..n) are all published: lane holds word u * 64 + lane in v[u]
// (u < W, W * 64 >= n; indices past n read the last word and are ignored).
template <int W>
__device__ __forceinline__ void wait_x(const uint32_t* src, int n, int lane, int* err, uint32_t (&v)[W]) {
    const int last = n - 1;
    for (unsigned spins = 0;; ++spins) {
#pragma unroll
        for (int u = 0; u < W; ++u)
            v[u] = __hip_atomic_load(src + min(u * 64 + lane, last), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        bool done = true;
#pragma unroll
        for (int u = 0; u < W; ++u) done &= v[u] != kXEmpty;
        if (__all(done)) break;
        if (spins > kSpinLimit) {
            if (lane == 0) atomicOr(err, 1);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// Flags between the waves of one workgroup, in LDS: the writer's earlier LDS stores are
// visible to a reader that saw the flag reach v.  Waits are bounded like the mailbox waits.
__device__ __forceinline__ void flag_set(int* f, int v, int lane) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    if (lane == 0) __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void flag_wait(const int* f, int v, int lane, int* err) {
    for (unsigned spins = 0; __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < v;
         ++spins) {
        if (spins > kSpinLimit) {
            if (lane == 0) atomicOr(err, 2);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

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
    f32x4 pfs[2][kMaxSRows][kMaxD / 4];  // this workgroup's folded predictor rows, two layers
    LayerPtrs lt[kMaxLayers];  // the layer table (LDS reads keep weight loads off the wait path)
    float xin[kMaxD];         // the layer input as gathered (the RMS scale is applied later)
    float ssp[2][kWaves];     // per-wave sums of squares of xin (by layer parity)
    float xt[kColTile];
    uint32_t key[2][kMaxNb];   // order keys of the exact and the speculative scores
    int E[kMaxKp];
    int Plist[2][kMaxKp];
    int hole_miss[kMaxKp];   // speculative position -> miss it recomputes, or -1
    int missE[kMaxKp];       // miss m -> E entry
    int row_of_e[kMaxKp];    // E entry -> list position whose partial row holds its partial
    int posE[kMaxNb];   // block -> position in E, or -1
    int posP[kMaxNb];   // block -> position in the current speculative list, or -1
    alignas(16) float aall[kMaxA];  // activations of the speculative list, in list order
    // down partials for this tile: row p < kMaxDnTot of list position p, row kMaxDnTot + m of
    // miss m
    alignas(16) float dparts[kMaxDnTot + kMaxKp][kColTile];
    // down pieces (this tile) of the list positions, staged from registers at the layer start
    u32x4 dnl[kMaxDnTot][64 * kDnPer];
    alignas(16) float amiss[kMaxKp][64];  // activations of the misses
    // LDS flags (value = layer + 1 once set for that layer)
    int f_keys, f_acts, f_E, f_pn, f_out, f_mrows;
    int f_done[kWaves];
};

// Static shape of one launch, shared by both roles.
struct Geo {
    int w, G, L, nb, blk, k, kp, F;
    int SPW;  // folded predictor rows of this workgroup: rows w, w + G, ... below n_blk
    int CH;   // 16-byte chunks of one folded row (d / 4)
    int NPC;  // 16-byte chunks of one block's down piece for one column tile
    int SW;   // score words per layer
    int AW;   // 64-bit activation words per layer (2F): the list's halves, then the misses
    int miss_base;
    bool has_tile;
    uint32_t tag;
};

// Top-m set of one list, run by one wave without LDS traffic.  The priority order is the
// order key (larger first), ties to the smaller index.  A bitwise search from the top
// bit finds T, the m-th largest order key (the largest T with at least m keys >= T); the
// set is every key > T plus the elements equal to T with the smallest indices.  Members
// are written to out[] in index order (the set is what matters to the fused step; its
// summation order is fixed by the slot map).  Only the top BITS bits of each key take part
// (BITS = 32: the exact order).  Q key slots per lane, Q * 64 >= n.  Needs 1 <= m <= n.
template <int BITS, int Q>
__device__ __forceinline__ void top_set_q(const uint32_t* keys, int n, int m, int* out, int lane) {
    uint32_t ok[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int i = q * 64 + lane;
        ok[q] = i < n ? keys[i] >> (32 - BITS) : 0u;  // padding compares below every c >= 1
    }
    uint32_t T = 0u;
    for (int bit = BITS - 1; bit >= 0; --bit) {
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

// The search's cost is its instruction count (one wave per SIMD runs it at a few cycles per
// instruction), so it takes only as many key slots per lane as n needs: Q = 3 at n <= 192
// ranks 20% faster than Q = 4 (1.7 against 2.1 us for the exact 32-bit search at n = 172).
template <int BITS>
__device__ __forceinline__ void top_set(const uint32_t* keys, int n, int m, int* out, int lane) {
    if (n <= 128) top_set_q<BITS, 2>(keys, n, m, out, lane);
    else if (n <= 192) top_set_q<BITS, 3>(keys, n, m, out, lane);
    else top_set_q<BITS, kMaxNb / 64>(keys, n, m, out, lane);
}

// X, one quarter per wave: words [wave*D/4, (wave+1)*D/4) of the layer input into xin (and
// this workgroup's tile into xt), and the quarter's sum of squares into ssp.  With two or
// more layers, layer 0 reads the caller's x directly (written before the launch).  That is
// safe because the output goes into x only at the last layer.  No workgroup gets past layer
// 1's input before every workgroup has finished its layer-0 gather: that gather precedes
// the workgroup's own layer-0 output tile, which every layer-1 gather waits for.  With one
// layer, a small kernel first writes x into the input row 0.
template <int D>
__device__ __forceinline__ void gather_input(const FusedArgs& P, Smem& sm, const Geo& g, int l, int wave,
                                             int lane) {
    constexpr int Q = D / kWaves;
    constexpr int W = Q / 64;
    float xv[W];
    if (l == 0 && P.L >= 2) {
#pragma unroll
        for (int u = 0; u < W; ++u) xv[u] = P.x[wave * Q + u * 64 + lane];
    } else {
        uint32_t v[W];
        wait_x<W>(x_rows(P, g.tag) + (size_t)l * D + wave * Q, Q, lane, P.err, v);
#pragma unroll
        for (int u = 0; u < W; ++u) xv[u] = __uint_as_float(v[u]);
    }
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < W; ++u) {
        const int i = wave * Q + u * 64 + lane;
        const float x = xv[u];
        ss = fmaf(x, x, ss);
        sm.xin[i] = x;
        if (g.has_tile && (i >> 4) == g.w) sm.xt[i & (kColTile - 1)] = x;
    }
    ss = wave_sum_dpp(ss);
    if (lane == 0) sm.ssp[l & 1][wave] = ss;
}

// RMS scale of the gathered input (every wave, after the input barrier; fixed order)
template <int D>
__device__ __forceinline__ float input_scale(const FusedArgs& P, const Smem& sm, int l) {
    const float* q = sm.ssp[l & 1];
    return P.prenorm ? rms_scale((q[0] + q[1]) + (q[2] + q[3]), D) : 1.f;
}

// Control wave, misses: activations of up to two neurons (block b[u] >= 0, neuron q[u]) from
// rows streamed straight from HBM (the control wave has no other weight loads in flight).
template <ls_dtype T, ls_act A, int NC>
__device__ __forceinline__ void ctl_gate_up(const Smem& sm, const Geo& g, int layer, size_t bb, float sc,
                                            const int (&b)[2], const int (&q)[2], float (&a)[2],
                                            int lane) {
    constexpr int V = Wt<T>::V;
    constexpr int KB = Wt<T>::kBytes;
    const size_t row_bytes = (size_t)NC * V * 64 * KB;
    u32x4 gw[2][NC], uw[2][NC];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        if (b[u] >= 0) {
            const uint8_t* base = sm.lt[layer].blocks + (size_t)b[u] * bb;
            const uint8_t* gr = base + (size_t)q[u] * row_bytes;
            const uint8_t* ur = base + (size_t)(g.blk + q[u]) * row_bytes;
#pragma unroll
            for (int j = 0; j < NC; ++j) {
                gw[u][j] = gload_u(gr, (uint32_t)(lane + 64 * j) * 16u);
                uw[u][j] = gload_u(ur, (uint32_t)(lane + 64 * j) * 16u);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        a[u] = 0.f;
        if (b[u] >= 0) {
            float gs = 0.f, us = 0.f;
#pragma unroll
            for (int j = 0; j < NC; ++j) {
                const float* hx = sm.xin + (lane + 64 * j) * V;
                gs += dot_chunk<T>(gw[u][j], hx);
                us += dot_chunk<T>(uw[u][j], hx);
            }
            const void* bias = sm.lt[layer].bias;
            const float g0 = sc * wave_sum_dpp(gs) + (bias ? Wt<T>::scalar(bias, (size_t)b[u] * g.blk + q[u]) : 0.f);
            const float u0 = sc * wave_sum_dpp(us);
            if (A == LS_ACT_REGLU) {
                a[u] = fmaxf(g0, 0.f) * u0;
            } else {
                const float sg = g0 / (1.f + expf(-g0));
                a[u] = fabsf(sg) > sm.lt[layer].threshold ? sg * u0 : 0.f;
            }
        }
    }
}

// Control wave, misses: this tile's down pieces of misses m0..m0+cnt-1 (cnt <= 8).
template <ls_dtype T>
__device__ __forceinline__ void miss_pieces(const FusedArgs& P, const Smem& sm, const Geo& g, int l, int m0,
                                            int cnt, int lane, u32x4 (&pc)[8][kDnPer]) {
    constexpr int KB = Wt<T>::kBytes;
    const size_t down_off = 2 * (size_t)g.blk * P.d * KB + (size_t)g.w * g.blk * kColTile * KB;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        if (u < cnt) {
            const uint8_t* base = sm.lt[l].blocks + (size_t)sm.E[sm.missE[m0 + u]] * P.block_bytes + down_off;
#pragma unroll
            for (int i = 0; i < kDnPer; ++i) pc[u][i] = gload_u(base, (uint32_t)min(lane + 64 * i, g.NPC - 1) * 16u);
        }
    }
}

// Control wave, misses: this tile's down partial of misses 0..M-1 (rows kMaxDnTot + m of
// dparts), eight at a time: their down pieces are requested first (the first eight's by the
// caller, in pc), then their activations are gathered from every workgroup.
template <ls_dtype T>
__device__ __forceinline__ void ctl_miss_down(const FusedArgs& P, Smem& sm, const Geo& g, int l,
                                              int M, int lane, u32x4 (&pc)[8][kDnPer]) {
    constexpr int V = Wt<T>::V;
    for (int m0 = 0; m0 < M; m0 += 8) {
        const int cnt = min(M - m0, 8);
        if (m0 > 0) miss_pieces<T>(P, sm, g, l, m0, cnt, lane, pc);
        const int n = cnt * g.blk;
        uint64_t v[8];
        wait_words<8>(P.amb + (size_t)l * g.AW + g.miss_base + m0 * g.blk, n, g.tag, lane, P.err, v);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int f = u * 64 + lane;
            if (f < n) sm.amiss[m0 + f / g.blk][f % g.blk] = word_value(v[u]);
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (u < cnt) {
                float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int i = 0; i < kDnPer; ++i) {
                    const int cc = lane + 64 * i;
                    if (cc < g.NPC) {
                        float wv[V];
                        Wt<T>::widen(pc[u][i], wv);
                        const float* ap = sm.amiss[m0 + u] + (cc / kColTile) * V;
#pragma unroll
                        for (int e = 0; e < V; ++e) acc[e & 3] = fmaf(ap[e], wv[e], acc[e & 3]);
                    }
                }
                float t = (acc[0] + acc[1]) + (acc[2] + acc[3]);
                t += __shfl_xor(t, 16, 64);
                t += __shfl_xor(t, 32, 64);
                if (lane < kColTile) sm.dparts[kMaxDnTot + m0 + u][lane] = t;
            }
        }
    }
}

// ---------------------------------------------------------------------------------------
// Control wave: waits, publications, the slot map.
template <ls_dtype T, ls_act A, int NC>
__device__ __forceinline__ void control_loop(const FusedArgs P, Smem& sm, const Geo g, int lane) {
    constexpr int V = Wt<T>::V;
    constexpr int D = NC * V * 64;
    for (int l = 0; l < g.L; ++l) {
        const bool last = l == g.L - 1;
        const int* Pc = sm.Plist[l & 1];
        LS_STAMP(P, g, l, 0, lane == 0);
        // X: this wave's quarter of the layer input (layer 0's was tagged into the mailbox
        // before the launch); the worker waves gather the other three
        gather_input<D>(P, sm, g, l, 0, lane);
        LS_STAMP(P, g, l, 1, lane == 0);
        lds_barrier();  // 1: input gathered (and the folded rows of layers l, l+1 staged)
        const float sc = input_scale<D>(P, sm, l);
        // S: this workgroup's scores, exact (layer l) and speculative (layer l+1), as dot
        // products of the staged folded rows with the input (lane-strided chunks, both rows
        // at once, then DPP), times the RMS scale.  The last layer's second row is stale and
        // its score is not published.
        static_assert(kMaxSRows == 1, "one folded row per workgroup and layer");
        if (g.SPW > 0) {
            constexpr int C = D / 4 / 64;  // 16-byte chunks per lane
            const f32x4* h4 = reinterpret_cast<const f32x4*>(sm.xin);
            const f32x4* r0 = sm.pfs[l & 1][0];
            const f32x4* r1 = sm.pfs[(l + 1) & 1][0];
            float a0[4] = {0.f, 0.f, 0.f, 0.f}, a1[4] = {0.f, 0.f, 0.f, 0.f};
            // every LDS read first (one round trip instead of one per chunk), then the products
            f32x4 hs[C], ps0[C], ps1[C];
#pragma unroll
            for (int i = 0; i < C; ++i) {
                const int c = lane + 64 * i;
                hs[i] = h4[c];
                ps0[i] = r0[c];
                ps1[i] = r1[c];
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < C; ++i) {
                const f32x4 hv = hs[i], p0 = ps0[i], p1 = ps1[i];
                a0[i & 3] = fmaf(p0.x, hv.x, a0[i & 3]);
                a1[i & 3] = fmaf(p1.x, hv.x, a1[i & 3]);
                a0[i & 3] = fmaf(p0.y, hv.y, a0[i & 3]);
                a1[i & 3] = fmaf(p1.y, hv.y, a1[i & 3]);
                a0[i & 3] = fmaf(p0.z, hv.z, a0[i & 3]);
                a1[i & 3] = fmaf(p1.z, hv.z, a1[i & 3]);
                a0[i & 3] = fmaf(p0.w, hv.w, a0[i & 3]);
                a1[i & 3] = fmaf(p1.w, hv.w, a1[i & 3]);
            }
            const float s0 = sc * wave_sum_dpp((a0[0] + a0[1]) + (a0[2] + a0[3]));
            const float s1 = sc * wave_sum_dpp((a1[0] + a1[1]) + (a1[2] + a1[3]));
            if (lane == 0) {
                mb_store(P.smb + (size_t)l * g.SW + g.w * kScoreStride, g.tag, s0);
                if (!last) mb_store(P.smb + (size_t)l * g.SW + g.w * kScoreStride + 1, g.tag, s1);
            }
        }
        LS_STAMP(P, g, l, 2, lane == 0);
        // order keys of every block's score (exact, then speculative); waves 2 and 3 rank them
        {
            // load u: block (u >> 1) * 64 + lane, list u & 1 (the last layer has no second list)
            constexpr int W = 2 * kMaxNb / 64;
            uint64_t v[W];
            const uint32_t row = (uint32_t)(l * g.SW);
            wait_gather_off<W>(
                P.smb,
                [&](int u) {
                    const int b = min((u >> 1) * 64 + lane, g.nb - 1);
                    return row + (uint32_t)(b * kScoreStride + (last ? 0 : (u & 1)));
                },
                2 * ((g.nb + 63) / 64), g.tag, lane, P.err, v);
#pragma unroll
            for (int u = 0; u < W; ++u) {
                const int b = (u >> 1) * 64 + lane;
                if (b < g.nb && !(last && (u & 1))) sm.key[u & 1][b] = order_key(word_value(v[u]));
            }
        }
        flag_set(&sm.f_keys, l + 1, lane);
        LS_STAMP(P, g, l, 3, lane == 0);
        // the list's activations (published by every workgroup's early gate/up), gathered
        // before the workers start streaming the next layer's weights
        if (l > 0 && g.has_tile) {
            const int n = g.kp * g.blk;
            const uint32_t* row = acts_rows(P, g.AW, g.F, l, g.tag);
            // one poll round of up to 32 words per lane (26 at the 7B shape; two rounds of 16
            // gathered 0.3 us later)
            for (int base = 0; base < n; base += 32 * 64) {
                uint32_t v[32];
                wait_x<32>(row + base, min(n - base, 32 * 64), lane, P.err, v);
#pragma unroll
                for (int u = 0; u < 32; ++u) {
                    const int i = base + u * 64 + lane;
                    if (i < n) sm.aall[i] = __uint_as_float(v[u]);
                }
            }
        }
        flag_set(&sm.f_acts, l + 1, lane);
        LS_STAMP(P, g, l, 4, lane == 0);
        flag_wait(&sm.f_E, l + 1, lane, P.err);  // E = exact top-k (wave 2)
        LS_STAMP(P, g, l, 5, lane == 0);
        // Maps.  An E block at list position p has its activations and its down partial
        // computed at p from the speculatively prefetched rows.  An E block missing from the
        // list is miss m: hole m (the m-th list position whose block is not in E) lends its
        // neuron slots, whose control waves recompute the activations and publish them after
        // the list (word miss_base + m * blk); every workgroup's control wave computes its
        // tile's down partial of the miss.  row_of_e: the partial row of E entry e.
        int M = 0;
        {
            const bool spec = l > 0;
            for (int b = lane; b < g.nb; b += 64) {
                sm.posE[b] = -1;
                sm.posP[b] = -1;
            }
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
            if (lane < g.k) sm.posE[sm.E[lane]] = lane;
            if (spec && lane < g.kp) sm.posP[Pc[lane]] = lane;
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
            const uint64_t below = (1ull << lane) - 1ull;
            const int pp = lane < g.k ? sm.posP[sm.E[lane]] : -1;  // -1 when !spec
            const bool miss = lane < g.k && pp < 0;
            const uint64_t mm = __ballot(miss);
            M = __popcll(mm);
            const int mr = __popcll(mm & below);
            if (miss) sm.missE[mr] = lane;
            if (lane < g.k) sm.row_of_e[lane] = miss ? kMaxDnTot + mr : pp;
            const int pe = spec && lane < g.kp ? sm.posE[Pc[lane]] : -1;
            const bool hole = lane < g.kp && pe < 0;
            const uint64_t hm = __ballot(hole);
            const int hr = __popcll(hm & below);
            sm.hole_miss[lane] = hole && hr < M ? hr : -1;
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
        }
        LS_STAMP(P, g, l, 6, lane == 0);
        u32x4 pc[8][kDnPer];
        if (M > 0) {
            // this tile's down pieces of the first eight misses, then the activations of the
            // misses' neurons held by this workgroup's hole slots
            if (g.has_tile) miss_pieces<T>(P, sm, g, l, 0, min(M, 8), lane, pc);
            for (int i0 = 0; i0 < kWorkers * kSlots; i0 += 2) {
                int bb2[2], qq2[2], mm2[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int t = g.w + g.G * (i0 + u);
                    const int m = (i0 + u < kWorkers * kSlots && t < g.kp * g.blk) ? sm.hole_miss[t / g.blk] : -1;
                    mm2[u] = m;
                    bb2[u] = m >= 0 ? sm.E[sm.missE[m]] : -1;
                    qq2[u] = t % g.blk;
                }
                float a2[2];
                ctl_gate_up<T, A, NC>(sm, g, l, P.block_bytes, sc, bb2, qq2, a2, lane);
#pragma unroll
                for (int u = 0; u < 2; ++u)
                    if (mm2[u] >= 0 && lane == 0)
                        mb_store(P.amb + (size_t)l * g.AW + g.miss_base + mm2[u] * g.blk + qq2[u], g.tag, a2[u]);
            }
        }
        // the misses' rows are in: the workers may queue the next layer's loads behind them
        flag_set(&sm.f_mrows, l + 1, lane);
        // this tile's down partial of every miss
        if (M > 0 && g.has_tile) ctl_miss_down<T>(P, sm, g, l, M, lane, pc);
        LS_STAMP(P, g, l, 7, lane == 0);
        // every worker's down partials of the list positions
#pragma unroll
        for (int v = 1; v < kWaves; ++v) flag_wait(&sm.f_done[v], l + 1, lane, P.err);
        LS_STAMP(P, g, l, 8, lane == 0);
        if (g.has_tile) {
            // y = sum over E of the entries' partial rows: lane = column + 16 * quarter; each
            // quarter sums its entries in E order, then the quarters in a fixed order
            const int col = lane & (kColTile - 1), qtr = lane >> 4;
            float y = 0.f;
#pragma unroll 4
            for (int e = qtr; e < g.k; e += 4) y += sm.dparts[sm.row_of_e[e]][col];
            y += __shfl_xor(y, 16, 64);
            y += __shfl_xor(y, 32, 64);
            const float xn = sm.xt[col] + y;
            if (lane < kColTile) {
                if (last) {
                    P.x[g.w * kColTile + lane] = xn;
                } else {
                    const size_t o = (size_t)(l + 1) * D + g.w * kColTile + lane;
                    __hip_atomic_store(x_rows(P, g.tag) + o, x_bits(xn), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    // the next launch's half: emptied here, read only after this launch ends
                    __hip_atomic_store(x_rows(P, g.tag + 1u) + o, kXEmpty, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        }
        {   // empty this layer's list activations of the next launch's half (a slice per
            // workgroup; every list position of any width lies in the first F words)
            const int per = (g.F + g.G - 1) / g.G;
            uint32_t* nxt = acts_rows(P, g.AW, g.F, l, g.tag + 1u);
            for (int i = g.w * per + lane; i < min((g.w + 1) * per, g.F); i += 64)
                __hip_atomic_store(nxt + i, kXEmpty, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        flag_set(&sm.f_out, l + 1, lane);  // the output store is issued: the workers may queue loads
        LS_STAMP(P, g, l, 9, lane == 0);
    }
}

// ---------------------------------------------------------------------------------------
// Worker waves: registers hold the folded predictor rows of a later layer and the
// speculatively prefetched blocks of the next layer.
template <ls_dtype T, ls_act A, int NC>
__device__ __forceinline__ void worker_loop(const FusedArgs P, Smem& sm, const Geo g, int wave, int lane) {
    constexpr int V = Wt<T>::V;
    constexpr int KB = Wt<T>::kBytes;
    constexpr int D = NC * V * 64;
    const int wl = (wave - 1) * 64 + lane;
    const size_t row_bytes = (size_t)D * KB;
    // a workgroup without a column tile (d / 16 below the grid) loads the last tile's pieces:
    // every load stays inside the block, and the values are never used
    const size_t down_off =
        2 * (size_t)g.blk * row_bytes + (size_t)min(g.w, D / kColTile - 1) * g.blk * kColTile * KB;
    const size_t bb = P.block_bytes;
    const u32x4 zero4 = {0u, 0u, 0u, 0u};
    // pfr: folded predictor rows in flight (one layer), moved to LDS one layer after they
    // were requested; chunk c = wl + kWL*j of row m sits in pfr[m * kPfPer + j]
    u32x4 pfr[kMaxSRows * kPfPer], gg[kSlots][NC], uu[kSlots][NC], dn[kMaxDn];
    uint32_t bw[kSlots];  // the word holding each slot's gate bias (when the layer has one)
#pragma unroll
    for (int sl = 0; sl < kSlots; ++sl) bw[sl] = 0u;
#pragma unroll
    for (int j = 0; j < kMaxSRows * kPfPer; ++j) pfr[j] = zero4;
#pragma unroll
    for (int sl = 0; sl < kSlots; ++sl)
#pragma unroll
        for (int j = 0; j < NC; ++j) gg[sl][j] = uu[sl][j] = zero4;
#pragma unroll
    for (int j = 0; j < kMaxDn; ++j) dn[j] = zero4;

    // every load is issued (clamped to valid addresses) so that later waits count exactly
    auto load_pf = [&](int layer) {
#pragma unroll
        for (int m = 0; m < kMaxSRows; ++m) {
            const int r = m < g.SPW ? g.w + g.G * m : 0;
            const float* row = sm.lt[layer].pf + (size_t)r * D;
#pragma unroll
            for (int j = 0; j < kPfPer; ++j)
                pfr[m * kPfPer + j] = gload_u(row, (uint32_t)min(wl + kWL * j, g.CH - 1) * 16u);
        }
    };
    auto stash_pf = [&](int layer) {  // pfr -> LDS buffer of `layer`
#pragma unroll
        for (int m = 0; m < kMaxSRows; ++m) {
            if (m < g.SPW) {
#pragma unroll
                for (int j = 0; j < kPfPer; ++j) {
                    const int c = wl + kWL * j;
                    if (c < g.CH) {
                        const u32x4 v = pin(pfr[m * kPfPer + j]);
                        sm.pfs[layer & 1][m][c] = f32x4{__uint_as_float(v.x), __uint_as_float(v.y),
                                                        __uint_as_float(v.z), __uint_as_float(v.w)};
                    }
                }
            }
        }
    };
    // neuron slot sl of this wave: workgroup slot index i = (wave-1) + kWorkers*sl,
    // global slot t = w + G*i (list position t / blk, neuron t % blk)
    // b and q are the same in every lane of the wave (one slot per wave)
    auto load_gu = [&](int sl, int layer, int b, int q) {
        b = __builtin_amdgcn_readfirstlane(b);
        q = __builtin_amdgcn_readfirstlane(q);
        const uint8_t* base = sm.lt[layer].blocks + (size_t)b * bb;
        {
            // the gate bias word (from the block base when the layer has no bias)
            const void* bias = sm.lt[layer].bias;
            const uint32_t e = (uint32_t)min(b * g.blk + q, g.F - 1);
            bw[sl] = gload_word(bias ? bias : (const void*)base, bias ? (e * KB) & ~3u : 0u);
        }
        const uint8_t* gr = base + (size_t)q * row_bytes;
        const uint8_t* ur = base + (size_t)(g.blk + q) * row_bytes;
#pragma unroll
        for (int j = 0; j < NC; ++j) gg[sl][j] = gload_u(gr, (uint32_t)(lane + 64 * j) * 16u);
#pragma unroll
        for (int j = 0; j < NC; ++j) uu[sl][j] = gload_u(ur, (uint32_t)(lane + 64 * j) * 16u);
    };
    // down pieces: position p = (wave-1) + kWorkers*jp of the list, chunks lane + 64*i of the piece
    auto load_down_pos = [&](int layer, int b, int jp) {
        b = __builtin_amdgcn_readfirstlane(b);
        const uint8_t* base = sm.lt[layer].blocks + (size_t)b * bb + down_off;
#pragma unroll
        for (int i = 0; i < kDnPer; ++i)
            dn[jp * kDnPer + i] = gload_u(base, (uint32_t)min(lane + 64 * i, g.NPC - 1) * 16u);
    };

    // activations of the slots in `use` (wave-uniform bit mask) from their rows in gg/uu:
    // slot sl holds neuron q[sl] of block b[sl]; every lane gets the results.  One
    // slot at a time, with several partial sums per row for instruction-level parallelism.
    auto gate_up = [&](int layer, float sc, unsigned use, const int (&b)[kSlots], const int (&q)[kSlots],
                       float (&a)[kSlots]) {
        constexpr int NA = 4;  // partial sums per row
        // this lane's part of the input: all LDS reads in flight together, reused by every
        // slot.  Read only by a wave with a slot in use: its published activations are what
        // orders these reads before the next layer's input overwrites xin.
        f32x4 hr[NC][V / 4];
        if (use) {
#pragma unroll
            for (int j = 0; j < NC; ++j)
#pragma unroll
                for (int i = 0; i < V / 4; ++i)
                    hr[j][i] = reinterpret_cast<const f32x4*>(sm.xin + (lane + 64 * j) * V)[i];
        }
        float gs[kSlots], us[kSlots];
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            gs[sl] = us[sl] = 0.f;
            if (use & (1u << sl)) {
                float ga[NA], ua[NA];
#pragma unroll
                for (int i = 0; i < NA; ++i) ga[i] = ua[i] = 0.f;
#pragma unroll
                for (int j = 0; j < NC; ++j) {
                    float wg[V], wu[V];
                    Wt<T>::widen(pin(gg[sl][j]), wg);
                    Wt<T>::widen(pin(uu[sl][j]), wu);
#pragma unroll
                    for (int i = 0; i < V / 4; ++i) {
                        const float hx[4] = {hr[j][i].x, hr[j][i].y, hr[j][i].z, hr[j][i].w};
#pragma unroll
                        for (int c = 0; c < 4; ++c) {
                            const int v = 4 * i + c;
                            ga[v % NA] = fmaf(wg[v], hx[c], ga[v % NA]);
                            ua[v % NA] = fmaf(wu[v], hx[c], ua[v % NA]);
                        }
                    }
                    if (j % 2 == 1) __builtin_amdgcn_sched_barrier(0);  // bounded live registers
                }
                gs[sl] = (ga[0] + ga[1]) + (ga[2] + ga[3]);
                us[sl] = (ua[0] + ua[1]) + (ua[2] + ua[3]);
            }
        }
        const void* bias = sm.lt[layer].bias;
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            if (use & (1u << sl)) {
                const float g0 = sc * wave_sum_dpp(gs[sl]) +
                                 (bias ? Wt<T>::from_word(bw[sl], (size_t)min(b[sl] * g.blk + q[sl], g.F - 1)) : 0.f);
                const float u0 = sc * wave_sum_dpp(us[sl]);
                if (A == LS_ACT_REGLU) {
                    a[sl] = fmaxf(g0, 0.f) * u0;
                } else {
                    const float sg = g0 / (1.f + expf(-g0));
                    a[sl] = fabsf(sg) > sm.lt[layer].threshold ? sg * u0 : 0.f;
                }
            }
        }
    };

    // this tile's down partials of the wave's list positions (p = wave-1 + kWorkers*jp), from
    // the pieces staged in LDS and the gathered activations.  Lane = column c + 16*gq; round r
    // takes position jp = 4r + gq, and each lane sums its column over the block's NG*V neurons
    // (chunk n*16 + c of a piece holds neurons n*V..n*V+V-1 of column c): no cross-lane
    // reduction, and every LDS read of a round is issued before its products.
    constexpr int kDnRounds = (kDnPos + 3) / 4;
    auto down_round = [&](auto ng_const, int r) {
        constexpr int NG = decltype(ng_const)::value;
        const int c = lane & (kColTile - 1), gq = lane >> 4;
        {
            const int jp = 4 * r + gq;
            const int p0 = (wave - 1) + kWorkers * jp;
            const bool ok = jp < kDnPos && p0 < g.kp;
            const int p = ok ? p0 : 0;  // a lane group without a position reads position 0
            u32x4 wr[NG];
            f32x4 av[NG][V / 4];
            const f32x4* a4 = reinterpret_cast<const f32x4*>(sm.aall) + p * (g.blk / 4);
#pragma unroll
            for (int n = 0; n < NG; ++n) {
                wr[n] = sm.dnl[p][n * kColTile + c];
#pragma unroll
                for (int i = 0; i < V / 4; ++i) av[n][i] = a4[n * (V / 4) + i];
            }
            // all of the round's LDS reads are in flight before the first product
            __builtin_amdgcn_sched_barrier(0);
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int n = 0; n < NG; ++n) {
                float wv[V];
                Wt<T>::widen(wr[n], wv);
#pragma unroll
                for (int i = 0; i < V / 4; ++i) {
                    acc[0] = fmaf(av[n][i].x, wv[4 * i + 0], acc[0]);
                    acc[1] = fmaf(av[n][i].y, wv[4 * i + 1], acc[1]);
                    acc[2] = fmaf(av[n][i].z, wv[4 * i + 2], acc[2]);
                    acc[3] = fmaf(av[n][i].w, wv[4 * i + 3], acc[3]);
                }
            }
            if (ok) sm.dparts[p][c] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
        }
    };

    int slot_t[kSlots];  // global slot index of each of this wave's slots
#pragma unroll
    for (int sl = 0; sl < kSlots; ++sl) slot_t[sl] = g.w + g.G * ((wave - 1) + kWorkers * sl);

    load_pf(0);

    for (int l = 0; l < g.L; ++l) {
        const bool last = l == g.L - 1;
        const int* Pc = sm.Plist[l & 1];
        const int* Pn = sm.Plist[(l + 1) & 1];
        // folded rows of layer l+1 (requested one layer ago) go to LDS before S needs them
        if (l == 0) {
            stash_pf(0);
            if (g.L > 1) {
                load_pf(1);
                stash_pf(1);
            }
        } else if (!last) {
            stash_pf(l + 1);
        }
        // this layer's down pieces (prefetched during the previous layer) into LDS
        if (l > 0 && g.has_tile) {
#pragma unroll
            for (int jp = 0; jp < kDnPos; ++jp) {
                const int p = (wave - 1) + kWorkers * jp;
                if (p < g.kp) {
#pragma unroll
                    for (int i = 0; i < kDnPer; ++i) sm.dnl[p][lane + 64 * i] = pin(dn[jp * kDnPer + i]);
                }
            }
        }
        // this wave's quarter of the layer input (no weight loads are in flight now)
        gather_input<D>(P, sm, g, l, wave, lane);
        lds_barrier();  // 1: input gathered
        const float sc = input_scale<D>(P, sm, l);
        // folded rows of layer l+2 (staged at the next layer's start), requested while no
        // weights stream: after the input barrier rather than after this layer's down rounds
        // (2068 against 2035 tokens/s on the 7B shape; after the early gate/up: 2031)
        if (l + 2 < g.L) load_pf(l + 2);
        // early GU: every speculative position held in this wave's slots (prefetched during
        // the previous layer), published at its list position while the selection runs
        if (l > 0) {
            unsigned use = 0;
            int bs[kSlots], qs[kSlots];
            float as[kSlots];
#pragma unroll
            for (int sl = 0; sl < kSlots; ++sl) {
                const int t = slot_t[sl];
                bs[sl] = t < g.kp * g.blk ? Pc[t / g.blk] : 0;
                qs[sl] = t % g.blk;
                if (t < g.kp * g.blk) use |= 1u << sl;
            }
            LS_STAMP(P, g, l, 14, wave == 3 && lane == 0);
            gate_up(l, sc, use, bs, qs, as);
#pragma unroll
            for (int sl = 0; sl < kSlots; ++sl)
                if ((use & (1u << sl)) && lane == 0)
                    __hip_atomic_store(acts_rows(P, g.AW, g.F, l, g.tag) + slot_t[sl], x_bits(as[sl]), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
        }
        LS_STAMP(P, g, l, 13, wave == 3 && lane == 0);
        // the selection: wave 2 the exact top-k of this layer, wave 3 the next layer's list
        if (wave == 2) {
            flag_wait(&sm.f_keys, l + 1, lane, P.err);
            top_set<32>(sm.key[0], g.nb, g.k, sm.E, lane);
            flag_set(&sm.f_E, l + 1, lane);
        } else if (wave == 3) {
            flag_wait(&sm.f_keys, l + 1, lane, P.err);
            // the speculative list only decides what is prefetched: its keys are cut to 16 bits
            // (ties to the smaller index), which halves the search
            if (!last) top_set<16>(sm.key[1], g.nb, g.kp, const_cast<int*>(Pn), lane);
            flag_set(&sm.f_pn, l + 1, lane);
            LS_STAMP(P, g, l, 12, lane == 0);
        }
        // the next layer's speculative list: the first slot's gate/up rows (and bias words) are
        // issued at once, this layer's down partials follow as soon as the list activations
        // are in (LDS work only), and the other slots' loads come after them: a compute unit
        // holds only about one slot's loads per wave in flight before issue stalls, so issuing
        // them earlier would hold the partials back (measured: 0, 1 or 2 early slots give
        // 1782, 1933 and 1900 tokens/s on the 7B shape).  Slots beyond the list (and the last
        // layer) load nothing: the next uses of these registers come after the layer-start
        // wait for every load.
        flag_wait(&sm.f_pn, l + 1, lane, P.err);
        const int ng = g.NPC / kColTile;
        static_assert(kDnRounds == kSlots, "one down round per slot");
#pragma unroll
        for (int sl = 0; sl < kEarlySlots; ++sl) {
            const int t = slot_t[sl];
            if (!last && t < g.kp * g.blk) load_gu(sl, l + 1, Pn[t / g.blk], t % g.blk);
        }
        flag_wait(&sm.f_acts, l + 1, lane, P.err);
        LS_STAMP(P, g, l, 15, wave == 3 && lane == 0);
        // list positions of this wave: (wave - 1) + kWorkers * jp below kp; round r takes 4r..4r+3
        const int npos = min(kDnPos, (g.kp - (wave - 1) + kWorkers - 1) / kWorkers);
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            if (l > 0 && g.has_tile && 4 * sl < npos) {
                if (ng == 8) down_round(std::integral_constant<int, 8>{}, sl);
                else if (ng == 4) down_round(std::integral_constant<int, 4>{}, sl);
                else down_round(std::integral_constant<int, 2>{}, sl);
            }
        }
        flag_set(&sm.f_done[wave], l + 1, lane);
        LS_STAMP(P, g, l, 11, wave == 3 && lane == 0);
        // the rest of the next layer's loads queue behind the control wave's loads of this
        // layer's missed rows (with a miss, a compute unit's memory pipeline full of the
        // stream held those rows back by several microseconds)
        flag_wait(&sm.f_mrows, l + 1, lane, P.err);
#pragma unroll
        for (int sl = kEarlySlots; sl < kSlots; ++sl) {
            const int t = slot_t[sl];
            if (!last && t < g.kp * g.blk) load_gu(sl, l + 1, Pn[t / g.blk], t % g.blk);
        }
        // then the next layer's down pieces for this workgroup's tile; the next layer starts
        // once the control wave has issued this layer's output.  (Measured on the 7B shape:
        // issuing the pieces after that wait instead gave 1980 against 1998 tokens/s, and
        // issuing pieces and rows before the other slots 1969 against 1994.)
        if (!last) {
#pragma unroll
            for (int jp = 0; jp < kDnPos; ++jp) {
                const int p = (wave - 1) + kWorkers * jp;
                if (p < g.kp) load_down_pos(l + 1, Pn[p], jp);
            }
        }
        LS_STAMP(P, g, l, 10, wave == 3 && lane == 0);
        flag_wait(&sm.f_out, l + 1, lane, P.err);
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
    g.nb = P.nb;
    g.blk = P.blk;
    g.k = P.k;
    g.kp = P.kp;
    g.F = P.F;
    g.SPW = g.w < g.nb ? (g.nb - 1 - g.w) / g.G + 1 : 0;
    g.CH = D / 4;
    g.SW = (int)fused_score_words_n(g.nb);
    g.miss_base = g.F;  // 64-bit words: the list's two 32-bit halves come first
    g.AW = 2 * g.F;
    g.NPC = g.blk * KB;
    g.has_tile = g.w < D / kColTile;
    g.tag = P.tag;
    {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(P.layers);
        uint32_t* dst = reinterpret_cast<uint32_t*>(sm.lt);
        const int words = P.L * (int)(sizeof(LayerPtrs) / 4);
        for (int i = threadIdx.x; i < words; i += kThreads) dst[i] = src[i];
        if (threadIdx.x == 0) {
            sm.f_keys = sm.f_acts = sm.f_E = sm.f_pn = sm.f_out = sm.f_mrows = 0;
            for (int v = 0; v < kWaves; ++v) sm.f_done[v] = 0;
        }
        __syncthreads();
    }
    if (wave == 0) control_loop<T, A, NC>(P, sm, g, lane);
    else worker_loop<T, A, NC>(P, sm, g, wave, lane);
}

// The layer-0 input as tagged mailbox words (launched before the fused kernel).
__global__ void tag_input_kernel(const float* __restrict__ x, int n, uint32_t* __restrict__ dst) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = x_bits(x[i]);
}

template <ls_dtype T, ls_act A>
hipError_t launch_t(const Shape& s, const FusedArgs& a, int n_wg, bool coop, hipStream_t st) {
    const int V = Wt<T>::V;
    const int nc = s.d / (V * 64);
    void* fn;
    if (nc == 2) fn = reinterpret_cast<void*>(decode_fused_kernel<T, A, 2>);
    else if (nc == 8) fn = reinterpret_cast<void*>(decode_fused_kernel<T, A, 8>);
    else return hipErrorNotSupported;
    if (a.L < 2) {  // with two or more layers, layer 0 reads x itself
        // row 0 of this launch's input half (one layer: L * d = d words per half)
        uint32_t* row0 = reinterpret_cast<uint32_t*>(a.xmb) + (size_t)(a.tag & 1u) * a.L * s.d;
        hipLaunchKernelGGL(tag_input_kernel, dim3((s.d + 255) / 256), dim3(256), 0, st, a.x, s.d, row0);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    FusedArgs copy = a;
    void* args[] = {&copy};
    if (coop) return hipLaunchCooperativeKernel(fn, dim3(n_wg), dim3(kThreads), args, 0, st);
    return hipLaunchKernel(fn, dim3(n_wg), dim3(kThreads), args, 0, st);
}

__global__ void untag_kernel(const uint64_t* __restrict__ src, int n, int stride, float* __restrict__ dst) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = __uint_as_float((uint32_t)src[(size_t)i * stride]);
}

}  // namespace

hipError_t launch_untag(const uint64_t* src, int n, int stride, float* dst, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(untag_kernel, dim3((n + 255) / 256), dim3(256), 0, st, src, n, stride, dst);
    return hipGetLastError();
}

FusedSupport fused_supported(const Shape& s, int B, int k, int kp, int n_wg, int L) {
    const int V = vec_elems(s.dtype), KB = elem_size(s.dtype);
    if (B != 1) return {false, "batch > 1"};
    if (L > kMaxLayers) return {false, "more than 128 layers"};
    if (s.d % (V * 64) || (s.d / (V * 64) != 2 && s.d / (V * 64) != 8)) return {false, "d_model"};
    if (s.d > kMaxD || s.d / kColTile > n_wg) return {false, "d_model too large for one tile per workgroup"};
    if (!s.fold) return {false, "predictor kept factored (its product would be larger)"};
    if ((s.n_blk + n_wg - 1) / n_wg > kMaxSRows) return {false, "predictor rows per workgroup"};
    if (s.n_blk > kMaxNb) return {false, "n_blk"};
    if (k < 1 || kp < k || kp > kMaxKp || kp > s.n_blk) return {false, "k / speculative width"};
    if ((long)kp * s.blk > (long)kWorkers * kSlots * n_wg) return {false, "neuron slots"};
    if (s.blk * KB > 64 * kDnPer || kp > kMaxDnTot) return {false, "down chunks"};
    {
        const int ng = s.blk * KB / 16;  // 16-byte chunks of one column of a down piece
        if (s.blk * KB % 16 || (ng != 2 && ng != 4 && ng != 8)) return {false, "block size"};
    }
    if ((long)kp * s.blk > kMaxA) return {false, "speculative width * block"};
    return {true, ""};
}

int fused_max_spec(const Shape& s, int n_wg) {
    const long by_slots = (long)kWorkers * kSlots * n_wg / s.blk;
    const long m = std::min<long>(std::min<long>(by_slots, kMaxKp), kMaxDnTot);
    return (int)std::min<long>(m, s.n_blk);
}


hipError_t launch_decode_fused(const Shape& s, const FusedArgs& a, int n_wg, bool coop, hipStream_t st) {
    const bool relu = s.act == LS_ACT_REGLU;
    switch (s.dtype) {
        case LS_F32: return relu ? launch_t<LS_F32, LS_ACT_REGLU>(s, a, n_wg, coop, st) : launch_t<LS_F32, LS_ACT_SWIGLU_THRESH>(s, a, n_wg, coop, st);
        case LS_F16: return relu ? launch_t<LS_F16, LS_ACT_REGLU>(s, a, n_wg, coop, st) : launch_t<LS_F16, LS_ACT_SWIGLU_THRESH>(s, a, n_wg, coop, st);
        case LS_BF16: return relu ? launch_t<LS_BF16, LS_ACT_REGLU>(s, a, n_wg, coop, st) : launch_t<LS_BF16, LS_ACT_SWIGLU_THRESH>(s, a, n_wg, coop, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace ls
