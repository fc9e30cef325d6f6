// ls_stage.hip - persistent consumer of one streamed layer's copy stages: the device side of
// the paper's flag coordination (Sec. 3.2.1, Alg. 1) on one MI355X.
//
// The blocks of a layer's priority list are copied into the HBM cache in K stages on the
// copy stream; after the copies of stage s the copy stream writes the call's tag into the
// arrival word arrive[s] (fine-grained device memory).  One launch of this kernel computes the
// whole layer with two kinds of waves in every workgroup:
//   gate/up waves (12): for s = 0..K-1, wait for stage s's arrival word, compute the gate/up
//     activations of the stage's neurons (one wave per neuron, spread over every gate/up wave
//     of the grid), and add the workgroup to the stage's count once all its gate/up waves
//     have stored theirs;
//   down group (4 waves): for s = 0..K-1, wait until every workgroup has counted stage s, add
//     the stage's down projection to the output tiles this workgroup owns (Eq. 1 partial
//     outputs summed into the refined feature of Eq. 2), and count itself done; the workgroup
//     that completes a stage's done count writes the tag into the host-visible done word (one
//     signal for many workgroups).
// So the gate/up of later stages runs while the down projection of earlier ones does, and
// each stage starts as soon as its own copies have landed.  Activations are exchanged as
// agent-scope atomic words (no cache write-back or invalidation); after an arrival one wave
// per workgroup takes a system-scope acquire so the copy engine's writes are seen.  Every wait
// is bounded by the wall clock: a wait that runs out writes the host-visible status word and
// ends the kernel, so a missing arrival fails the call instead of hanging (the counters are
// then left for the host to clear).
//
// The per-neuron and per-tile arithmetic is the per-call kernels' own (ls_sparse.h), so the
// result is bitwise that of the same stages run as separate launches.
#include "ls_sparse.h"

namespace ls {
namespace {

constexpr int kStageWaves = 16;  // waves 0-3: the down group; waves 4-15 gate/up
constexpr int kGuWaves = kStageWaves - 4;
constexpr int kStageActs = 8192;  // activations of one stage staged in LDS (larger stages read them from HBM)

__device__ inline uint64_t ticks() { return __builtin_amdgcn_s_memrealtime(); }

// *w == tag, read at system scope (the copy stream writes it); false once `limit` ticks pass
__device__ bool wait_tag(const uint32_t* w, uint32_t tag, uint64_t limit) {
    const uint64_t t0 = ticks();
    while (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != tag) {
        if (ticks() - t0 > limit) return false;
        __builtin_amdgcn_s_sleep(2);
    }
    return true;
}

// *c >= target, read at agent scope (this kernel's workgroups count into it)
__device__ bool wait_count(const uint32_t* c, uint32_t target, uint64_t limit) {
    const uint64_t t0 = ticks();
    while (__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        if (ticks() - t0 > limit) return false;
        __builtin_amdgcn_s_sleep(1);
    }
    return true;
}

// LDS word *c >= target (workgroup scope, acquire); false once `limit` ticks pass
__device__ bool wait_lds(const int* c, int target, uint64_t limit) {
    const uint64_t t0 = ticks();
    while (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < target) {
        if (ticks() - t0 > limit) return false;
        __builtin_amdgcn_s_sleep(1);
    }
    return true;
}

struct Lds {
    float acts[kStageActs];
    float part[kDnVirt][kMaxBatch][kColTile];
    int arrived;      // gate/up waves: stages whose arrival word was seen (and acquired)
    int gu_done[kMaxStages];  // gate/up waves done with each stage
    int dn_bar;       // down group: barrier arrivals
    int abort;        // a wait of this workgroup ran out
};

template <ls_dtype T, ls_act A, bool RMS>
__global__ __launch_bounds__(64 * kStageWaves) void stage_consumer_kernel(StageArgs p) {
    __shared__ Lds sh;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int G = gridDim.x;
    if (threadIdx.x == 0) sh.arrived = sh.dn_bar = sh.abort = 0;
    for (int i = threadIdx.x; i < kMaxStages; i += blockDim.x) sh.gu_done[i] = 0;
    __syncthreads();
    auto fail = [&](uint32_t code) {
        if (lane == 0) {
            __hip_atomic_store(p.status, code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            __hip_atomic_store(&sh.abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
    };
    if (wave >= 4) {
        // ---- gate/up waves ----
        const int gw = wave - 4;
        for (int s = 0; s < p.K; ++s) {
            const int lo = (int)((int64_t)s * p.n / p.K), hi = (int)((int64_t)(s + 1) * p.n / p.K);
            if (gw == 0) {  // one wave per workgroup watches the arrival word
                bool ok = true;
                // a stage that copied nothing was covered by an earlier stage's word
                const bool fresh = p.arrive != nullptr && p.wait_on[s] == s;
                if (lane == 0) {
                    ok = !fresh || wait_tag(p.arrive + s, p.tag, p.limit);
                    // system-scope acquire: this compute unit's L1 and its XCD's L2 drop lines the
                    // copy engine has since overwritten
                    if (ok && fresh) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
                    if (ok) __hip_atomic_store(&sh.arrived, s + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
                }
                ok = __shfl(ok ? 1 : 0, 0) != 0;
                if (!ok) { fail(2u); return; }
            } else if (!wait_lds(&sh.arrived, s + 1, p.limit)) {
                if (__hip_atomic_load(&sh.abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == 0) fail(2u);
                return;
            }
            if (__hip_atomic_load(&sh.abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) return;
            // neuron j of the whole list (j = lo blk + t) goes to gate/up wave j mod W of the grid,
            // so consecutive stages keep every workgroup busy
            const int tasks = (hi - lo) * p.blk;
            const int W = G * kGuWaves, g = blockIdx.x * kGuWaves + gw;
            for (int t = ((g - (lo * p.blk) % W) % W + W) % W; t < tasks; t += W) {
                const int e = lo + t / p.blk, q = t % p.blk;
                gateup_neuron<T, A, 1, RMS, false, true>(p.blocks, p.block_bytes, p.slot_table, p.bias, p.thresh,
                                                         p.x_in, p.d, p.blk, p.n_blk, p.F, p.idx[e], e, q, p.a_buf,
                                                         lane);
            }
            // this wave's activation stores are complete before it is counted
            __builtin_amdgcn_s_waitcnt(0);
            if (lane == 0) {
                const int c = __hip_atomic_fetch_add(&sh.gu_done[s], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP) + 1;
                if (c == kGuWaves) atomicAdd(p.cnt + kMaxStages + s, 1u);  // the workgroup's last gate/up wave of stage s
            }
        }
        return;
    }
    // ---- down group (waves 0-3) ----
    const int ntiles = p.d / kColTile;
    int bar = 0;
    bool alive = true;
    auto group_sync = [&] {
        bar += 4;
        if (lane == 0) __hip_atomic_fetch_add(&sh.dn_bar, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        bool ok = true;
        if (lane == 0) ok = wait_lds(&sh.dn_bar, bar, p.limit);
        if (!__shfl(ok ? 1 : 0, 0)) alive = false;
    };
    for (int s = 0; s < p.K && alive; ++s) {
        const int lo = (int)((int64_t)s * p.n / p.K), hi = (int)((int64_t)(s + 1) * p.n / p.K);
        const bool work = hi > lo || s == 0;
        bool ok = true;
        if (lane == 0) ok = wait_count(p.cnt + kMaxStages + s, (uint32_t)G, p.limit);
        if (!__shfl(ok ? 1 : 0, 0)) {
            if (__hip_atomic_load(&sh.abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == 0) fail(4u);
            return;
        }
        // the stage's activations: into LDS with one coalesced pass of agent-scope atomic loads
        // (pairs of words; lo blk and the count are even), or read from HBM by every tile
        const int n_act = (hi - lo) * p.blk;
        const bool staged = n_act <= kStageActs;
        if (staged) {
            const uint64_t* src = reinterpret_cast<const uint64_t*>(p.a_buf + (size_t)lo * p.blk);
            uint64_t* dst = reinterpret_cast<uint64_t*>(sh.acts);
            for (int i = threadIdx.x; i < n_act / 2; i += 256)
                dst[i] = __hip_atomic_load(src + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            group_sync();
        }
        for (int tile = blockIdx.x; tile < ntiles && alive; tile += G) {
            if (staged)
                down_tile<T, 1, false, false, 4, 4>(p.blocks, p.block_bytes, p.slot_table, sh.acts, p.F, p.d, p.blk,
                                              p.n_blk, p.idx, lo, hi, p.x_in, p.x_acc, tile, wave, lane, work,
                                              sh.part, group_sync, lo);
            else
                down_tile<T, 1, false, true, 4, 4>(p.blocks, p.block_bytes, p.slot_table, p.a_buf, p.F, p.d, p.blk,
                                             p.n_blk, p.idx, lo, hi, p.x_in, p.x_acc, tile, wave, lane, work,
                                             sh.part, group_sync);
            group_sync();  // the tile's partials (and the staged activations) are read before reuse
        }
        if (!alive) { fail(4u); return; }
        if (wave == 0 && lane == 0) {
            const uint32_t done = atomicAdd(p.cnt + s, 1u) + 1u;
            if (done == (uint32_t)G) {  // the last workgroup to finish stage s
                if (p.done) __hip_atomic_store(p.done + s, p.tag, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
                // after the last stage every wave of the grid is past every wait (a down group
                // finishes its stages in order): reset for the next call
                if (s == p.K - 1)
                    for (int i = 0; i < p.K; ++i) {
                        __hip_atomic_store(p.cnt + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        __hip_atomic_store(p.cnt + kMaxStages + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
            }
        }
    }
}

// The copy stream's own small kernels must find room on some compute unit while this kernel
// occupies every one of them (the arrival words wait for them): a build whose waves would
// leave fewer than 64 of a SIMD's 512 registers free is refused.
constexpr int kFreeRegsPerSimd = 64;

template <ls_dtype T, ls_act A>
hipError_t launch_t(const Shape& s, const StageArgs& p, int grid, bool cooperative, hipStream_t st) {
    const void* fn = s.prenorm ? reinterpret_cast<const void*>(&stage_consumer_kernel<T, A, true>)
                               : reinterpret_cast<const void*>(&stage_consumer_kernel<T, A, false>);
    hipFuncAttributes fa{};
    hipError_t e = hipFuncGetAttributes(&fa, fn);
    if (e != hipSuccess) return e;
    const int regs = (fa.numRegs + 7) / 8 * 8;  // allocation granule of 8
    if (regs * (kStageWaves / 4) > 512 - kFreeRegsPerSimd) return hipErrorInvalidConfiguration;
    StageArgs arg = p;
    void* args[] = {&arg};
    if (cooperative) return hipLaunchCooperativeKernel(fn, dim3(grid), dim3(64 * kStageWaves), args, 0, st);
    return hipLaunchKernel(fn, dim3(grid), dim3(64 * kStageWaves), args, 0, st);
}

}  // namespace

hipError_t launch_stage_consumer(const Shape& s, const StageArgs& p, int grid, bool cooperative, hipStream_t st) {
    if (p.K < 1 || p.K > kMaxStages || p.n < 0 || grid < 1 || p.d % kColTile) return hipErrorInvalidValue;
    const bool relu = s.act == LS_ACT_REGLU;
    switch (s.dtype) {
        case LS_F32: return relu ? launch_t<LS_F32, LS_ACT_REGLU>(s, p, grid, cooperative, st)
                                 : launch_t<LS_F32, LS_ACT_SWIGLU_THRESH>(s, p, grid, cooperative, st);
        case LS_F16: return relu ? launch_t<LS_F16, LS_ACT_REGLU>(s, p, grid, cooperative, st)
                                 : launch_t<LS_F16, LS_ACT_SWIGLU_THRESH>(s, p, grid, cooperative, st);
        case LS_BF16: return relu ? launch_t<LS_BF16, LS_ACT_REGLU>(s, p, grid, cooperative, st)
                                  : launch_t<LS_BF16, LS_ACT_SWIGLU_THRESH>(s, p, grid, cooperative, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace ls
