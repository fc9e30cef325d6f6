// ls_sparse.h - device bodies of the sparse FFN step shared by the per-call kernels and the
// stage-consuming persistent kernel: one neuron's gate/up dot products and gating (Eq. 1),
// one column tile of the down projection over a range of the priority list (the sum over
// hidden neurons of Sec. 3.2.2).  Both kernels run the same code, so their results agree bit
// for bit.
#pragma once

#include "ls_device.h"
#include "ls_internal.h"

namespace ls {

// Activation words.  COH: relaxed atomics at agent scope, coherent across the compute units
// of every XCD without cache maintenance (a persistent kernel that exchanges activations
// between its own workgroups); otherwise plain accesses (the next kernel launch orders them).
template <bool COH>
__device__ __forceinline__ void act_store(float* p, float v) {
    if (COH) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else *p = v;
}
template <bool COH>
__device__ __forceinline__ f32x4 act_load4(const float* p) {
    if (!COH) return *reinterpret_cast<const f32x4*>(p);
    f32x4 r;
    r.x = __hip_atomic_load(p + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    r.y = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    r.z = __hip_atomic_load(p + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    r.w = __hip_atomic_load(p + 3, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return r;
}

// A hook run once per wave by the bodies below before their first read of staged data
// (the callers that stage it in LDS pass a copy and a barrier); by default nothing.
struct NoPrep {
    __device__ void operator()() const {}
};

// ---- gate/up gather + gating (one wave per neuron) --------------------------------------------------------------
__device__ inline int list_end(const int32_t* count, int end, int n_blk) {
    int c = *count;
    c = c < 0 ? 0 : (c > n_blk ? n_blk : c);
    return end < c ? end : c;
}

// acc[i] += row . h[i] over this lane's 16-byte chunks (c = lane + 64 n), in the same order
// whether or not the row is read alone; SS also sums h[i]^2 into ss[i].  U chunks' loads are
// issued together (the order does not depend on U); prep() runs once, after the first loads.
template <ls_dtype T, int B, bool SS, int U = 4, typename Prep = NoPrep>
__device__ __forceinline__ void row_dot(const u32x4* row, const float* __restrict__ h, int d, int lane,
                                        float (&acc)[B], float (&ss)[B], Prep prep = Prep{}) {
    constexpr int V = Wt<T>::V;
    const int nchunk = d / V;
    if (nchunk <= 0) prep();
    for (int r0 = 0; r0 < nchunk; r0 += 64 * U) {
        const int c0 = r0 + lane;
        u32x4 rw[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + u * 64;
            rw[u] = c < nchunk ? ld_stream(row + c) : u32x4{0u, 0u, 0u, 0u};
        }
        if (r0 == 0) prep();
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + u * 64;
            if (c < nchunk) {
                float w[V];
                Wt<T>::widen(rw[u], w);
#pragma unroll
                for (int i = 0; i < B; ++i) {
                    const f32x4* hp = reinterpret_cast<const f32x4*>(h + (size_t)i * d + (size_t)c * V);
#pragma unroll
                    for (int qq = 0; qq < V / 4; ++qq) {
                        const f32x4 x4 = hp[qq];
                        acc[i] = fmaf(w[4 * qq + 0], x4.x, acc[i]);
                        acc[i] = fmaf(w[4 * qq + 1], x4.y, acc[i]);
                        acc[i] = fmaf(w[4 * qq + 2], x4.z, acc[i]);
                        acc[i] = fmaf(w[4 * qq + 3], x4.w, acc[i]);
                        if (SS) {
                            ss[i] = fmaf(x4.x, x4.x, ss[i]);
                            ss[i] = fmaf(x4.y, x4.y, ss[i]);
                            ss[i] = fmaf(x4.z, x4.z, ss[i]);
                            ss[i] = fmaf(x4.w, x4.w, ss[i]);
                        }
                    }
                }
            }
        }
    }
}

// Gate output of Eq. 1 before the up factor: ReLU(g), or SiLU(g) when |SiLU(g)| > thresh
// (thresholded SiLU), else 0.
template <ls_act A>
__device__ __forceinline__ float gate_out(float g, float thresh) {
    if (A == LS_ACT_REGLU) return fmaxf(g, 0.f);
    const float sg = g / (1.f + expf(-g));
    return fabsf(sg) > thresh ? sg : 0.f;
}

// Neuron q of list entry e (block b) for B tokens of h: a_buf[i F + e blk + q] = its
// activation.  Called by one whole wave.
// ZS (row-level zero skip): the gate row is read first and the up row only when the gate
// output of some token is nonzero; a neuron whose gate output is zero for every token then
// costs its gate row alone.  The activations equal those of the one-pass form (same
// accumulation order; a skipped product is an exact zero).
// U: 16-byte chunks per row and lane whose loads are issued together.  Each lane sums its
// chunks lane, lane + 64, ... in ascending order whatever U is, so U does not change results.
// prep() runs once before h is first read: after the first U chunks' loads are issued (at the
// start with ZS, and before returning for an entry that reads nothing).
template <ls_dtype T, ls_act A, int B, bool RMS, bool ZS, bool COH = false, int U = 4, typename Prep = NoPrep>
__device__ __forceinline__ void gateup_neuron(
    const uint8_t* __restrict__ blocks, size_t block_bytes, const int32_t* __restrict__ slot_table,
    const void* __restrict__ bias, float thresh, const float* __restrict__ h, int d, int blk,
    int n_blk, int F, int b, int e, int q, float* __restrict__ a_buf, int lane, Prep prep = Prep{}) {
    constexpr int V = Wt<T>::V;
    const size_t apos = (size_t)e * blk + q;
    if (b < 0 || b >= n_blk) {  // invalid id: the entry contributes nothing
        prep();
        if (lane < B) act_store<COH>(a_buf + (size_t)lane * F + apos, 0.f);
        return;
    }
    const int slot = slot_table ? slot_table[b] : b;
    if (slot < 0) {  // block not in the cache: contributes nothing
        prep();
        if (lane < B) act_store<COH>(a_buf + (size_t)lane * F + apos, 0.f);
        return;
    }
    const uint8_t* base = blocks + (size_t)slot * block_bytes;
    const size_t row_bytes = (size_t)d * Wt<T>::kBytes;
    const u32x4* grow = reinterpret_cast<const u32x4*>(base + (size_t)q * row_bytes);
    const u32x4* urow = reinterpret_cast<const u32x4*>(base + (size_t)(blk + q) * row_bytes);
    const int nchunk = d / V;
    float ag[B], au[B], ss[B];  // h here is the layer input x; ss its sum of squares
#pragma unroll
    for (int i = 0; i < B; ++i) ag[i] = au[i] = ss[i] = 0.f;
    const float bj = bias ? Wt<T>::scalar(bias, (size_t)b * blk + q) : 0.f;
    if (ZS) {
        prep();
        row_dot<T, B, RMS>(grow, h, d, lane, ag, ss);
        bool any = false;
#pragma unroll
        for (int i = 0; i < B; ++i) {
            const float sc = RMS ? rms_scale(wave_sum(ss[i]), d) : 1.f;
            ag[i] = gate_out<A>(sc * wave_sum(ag[i]) + bj, thresh);
            ss[i] = sc;
            any |= ag[i] != 0.f;
        }
        if (any) {  // wave-uniform: every lane holds the same sums
            float unused[B];
            row_dot<T, B, false>(urow, h, d, lane, au, unused);
        }
#pragma unroll
        for (int i = 0; i < B; ++i) {
            const float a = ag[i] != 0.f ? ag[i] * (ss[i] * wave_sum(au[i])) : 0.f;
            if (lane == 0) act_store<COH>(a_buf + (size_t)i * F + apos, a);
        }
        return;
    }
    // rounds of U chunks per lane (r0 is the same in every lane, so prep() is reached by the
    // whole wave); lane L takes chunks L, L + 64, ... in ascending order
    if (nchunk <= 0) prep();
    for (int r0 = 0; r0 < nchunk; r0 += 64 * U) {
        const int c0 = r0 + lane;
        u32x4 rg[U], ru[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + u * 64;
            const bool ok = c < nchunk;
            rg[u] = ok ? ld_stream(grow + c) : u32x4{0u, 0u, 0u, 0u};
            ru[u] = ok ? ld_stream(urow + c) : u32x4{0u, 0u, 0u, 0u};
        }
        if (r0 == 0) prep();
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + u * 64;
            if (c < nchunk) {
                float wg[V], wu[V];
                Wt<T>::widen(rg[u], wg);
                Wt<T>::widen(ru[u], wu);
#pragma unroll
                for (int i = 0; i < B; ++i) {
                    const f32x4* hp = reinterpret_cast<const f32x4*>(h + (size_t)i * d + (size_t)c * V);
#pragma unroll
                    for (int qq = 0; qq < V / 4; ++qq) {
                        const f32x4 x4 = hp[qq];
                        ag[i] = fmaf(wg[4 * qq + 0], x4.x, ag[i]);
                        ag[i] = fmaf(wg[4 * qq + 1], x4.y, ag[i]);
                        ag[i] = fmaf(wg[4 * qq + 2], x4.z, ag[i]);
                        ag[i] = fmaf(wg[4 * qq + 3], x4.w, ag[i]);
                        au[i] = fmaf(wu[4 * qq + 0], x4.x, au[i]);
                        au[i] = fmaf(wu[4 * qq + 1], x4.y, au[i]);
                        au[i] = fmaf(wu[4 * qq + 2], x4.z, au[i]);
                        au[i] = fmaf(wu[4 * qq + 3], x4.w, au[i]);
                        if (RMS) {
                            ss[i] = fmaf(x4.x, x4.x, ss[i]);
                            ss[i] = fmaf(x4.y, x4.y, ss[i]);
                            ss[i] = fmaf(x4.z, x4.z, ss[i]);
                            ss[i] = fmaf(x4.w, x4.w, ss[i]);
                        }
                    }
                }
            }
        }
    }
#pragma unroll
    for (int i = 0; i < B; ++i) {
        const float sc = RMS ? rms_scale(wave_sum(ss[i]), d) : 1.f;
        const float g = sc * wave_sum(ag[i]) + bj;
        const float u = sc * wave_sum(au[i]);
        float a;
        if (A == LS_ACT_REGLU) {
            a = fmaxf(g, 0.f) * u;  // exactly zero for g <= 0
        } else {
            const float sg = g / (1.f + expf(-g));
            a = fabsf(sg) > thresh ? sg * u : 0.f;
        }
        if (lane == 0) act_store<COH>(a_buf + (size_t)i * F + apos, a);
    }
}

// ---- down projection + residual -----------------------------------------------------------
// Column tile `tile` of the down projection over list entries [begin, n_end), by the NP waves
// (wave 0..NP-1) that own `part`; x_acc = (begin == 0 ? x_in : x_acc) + y for the tile's columns.
// The activation of neuron j of entry e is a_buf[i F + (e - a_off) blk + j].
// sync() is the barrier of the waves that share `part` (the workgroup's, or the group's);
// a group with active == false only takes part in it.
// The sum has one fixed order whatever NP and G are: kDnVirt virtual waves, virtual wave v
// taking the entries begin + v + kDnVirt j; its work is a sequence of items (entry j, chunk
// pair p: chunks lane + 64 (2p + r), r = 0, 1 of the entry's piece) in entry-major order,
// summed item by item per lane; then lanes l, l+16, l+32, l+48 (the same column) are added,
// and the column's total is the sum of the virtual waves' in order.  Physical wave w runs the
// virtual waves w, w + NP, ... one after the other; the loads of G items are issued together.
// So the per-call kernel (16 waves) and the stage-consuming kernel (a 4-wave group) agree
// bit for bit.
// ZS (row-level zero skip): a lane's 16-byte vector holds V neurons of one column; it is read
// only when one of those neurons has a nonzero activation for some token.  The sums equal
// those of the full read (a skipped product is an exact zero).
constexpr int kDnVirt = 16;

template <ls_dtype T, int B, bool ZS, bool COH, int G, int NP, typename Sync, typename Prep = NoPrep>
__device__ __forceinline__ void down_tile(
    const uint8_t* __restrict__ blocks, size_t block_bytes, const int32_t* __restrict__ slot_table,
    const float* __restrict__ a_buf, int F, int d, int blk, int n_blk,
    const int32_t* __restrict__ idx, int begin, int n_end,
    const float* __restrict__ x_in, float* __restrict__ x_acc, int tile, int wave, int lane, bool active,
    float (&part)[kDnVirt][kMaxBatch][kColTile], Sync sync, int a_off = 0, Prep prep = Prep{}) {
    static_assert(kDnVirt % NP == 0, "whole virtual waves per physical wave");
    constexpr int V = Wt<T>::V;
    if (!active) n_end = begin;
    const int nchunk = blk * Wt<T>::kBytes;  // 16-byte chunks of one (block, tile) piece
    const int npair = (nchunk + 127) / 128;  // chunk pairs per lane and entry
    const size_t down_off = (size_t)2 * blk * d * Wt<T>::kBytes +
                            (size_t)tile * blk * kColTile * Wt<T>::kBytes;
    bool prepped = false;
    if (ZS) {
        prep();
        prepped = true;
    }
    for (int vw = wave; vw < kDnVirt; vw += NP) {
        const int n_mine = n_end > begin + vw ? (n_end - begin - vw + kDnVirt - 1) / kDnVirt : 0;
        const int n_items = n_mine * npair;
        float acc[B];
#pragma unroll
        for (int i = 0; i < B; ++i) acc[i] = 0.f;
        for (int it0 = 0; it0 < n_items; it0 += G) {
            const u32x4* src[G];
            int ent[G], c0[G], bv[G];
            // the items' list entries, then (host-resident weights) their cache slots: every load
            // of a kind issued before the first use, entries past the list clamped to a valid one
            // (a per-item branch had made each load wait for the one before)
#pragma unroll
            for (int u = 0; u < G; ++u) {
                const int it = it0 + u;
                bv[u] = it < n_items ? idx[begin + vw + kDnVirt * (it / npair)] : -1;
            }
#pragma unroll
            for (int u = 0; u < G; ++u) bv[u] = bv[u] < n_blk ? bv[u] : -1;
            if (slot_table) {
#pragma unroll
                for (int u = 0; u < G; ++u) {
                    const int sl = slot_table[bv[u] < 0 ? 0 : bv[u]];
                    bv[u] = bv[u] < 0 ? -1 : sl;
                }
            }
#pragma unroll
            for (int u = 0; u < G; ++u) {
                const int it = it0 + u;
                const int j = it / npair, pr = it - j * npair;
                const int e = begin + vw + kDnVirt * j;
                const int slot = bv[u];
                ent[u] = slot < 0 ? -1 : e;
                c0[u] = lane + 128 * pr;
                src[u] = reinterpret_cast<const u32x4*>(blocks + (size_t)(slot < 0 ? 0 : slot) * block_bytes +
                                                        down_off);
            }
            bool use[G][2];
#pragma unroll
            for (int u = 0; u < G; ++u)
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const int c = c0[u] + 64 * r;
                    use[u][r] = ent[u] >= 0 && c < nchunk;
                    if (ZS && use[u][r]) {
                        const float* ap = a_buf + (size_t)(ent[u] - a_off) * blk + (size_t)(c / kColTile) * V;
                        bool nz = false;
#pragma unroll
                        for (int i = 0; i < B; ++i) {
#pragma unroll
                            for (int qq = 0; qq < V / 4; ++qq) {
                                const f32x4 av = act_load4<COH>(ap + (size_t)i * F + 4 * qq);
                                nz |= (av.x != 0.f) | (av.y != 0.f) | (av.z != 0.f) | (av.w != 0.f);
                            }
                        }
                        use[u][r] = nz;
                    }
                }
            u32x4 raw[G][2];
#pragma unroll
            for (int u = 0; u < G; ++u)
#pragma unroll
                for (int r = 0; r < 2; ++r)
                    raw[u][r] = use[u][r] ? ld_stream(src[u] + c0[u] + 64 * r) : u32x4{0u, 0u, 0u, 0u};
            if (!prepped) {
                prep();
                prepped = true;
            }
#pragma unroll
            for (int u = 0; u < G; ++u)
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const int c = c0[u] + 64 * r;
                    if (use[u][r]) {
                        float w[V];
                        Wt<T>::widen(raw[u][r], w);
                        const int grp = c / kColTile;  // this lane's V neurons
                        const float* ap = a_buf + (size_t)(ent[u] - a_off) * blk + (size_t)grp * V;
#pragma unroll
                        for (int i = 0; i < B; ++i) {
#pragma unroll
                            for (int qq = 0; qq < V / 4; ++qq) {
                                const f32x4 av = act_load4<COH>(ap + (size_t)i * F + 4 * qq);
                                acc[i] = fmaf(av.x, w[4 * qq + 0], acc[i]);
                                acc[i] = fmaf(av.y, w[4 * qq + 1], acc[i]);
                                acc[i] = fmaf(av.z, w[4 * qq + 2], acc[i]);
                                acc[i] = fmaf(av.w, w[4 * qq + 3], acc[i]);
                            }
                        }
                    }
                }
        }
        // lanes l, l+16, l+32, l+48 hold the same column
#pragma unroll
        for (int i = 0; i < B; ++i) {
            float v = acc[i];
            v += __shfl_xor(v, 16, 64);
            v += __shfl_xor(v, 32, 64);
            if (lane < kColTile) part[vw][i][lane] = v;
        }
    }
    if (!prepped) prep();
    sync();
    const int tid = wave * 64 + lane;
    if (active && tid < B * kColTile) {
        const int i = tid / kColTile, col = tid % kColTile;
        float y = 0.f;
#pragma unroll
        for (int v = 0; v < kDnVirt; ++v) y += part[v][i][col];
        const size_t m = (size_t)i * d + (size_t)tile * kColTile + col;
        x_acc[m] = (begin == 0 ? x_in[m] : x_acc[m]) + y;
    }
}


}  // namespace ls
