// ls_kernels.hip - gfx950 kernels of one sparse-FFN decode step.
//
//  gemv_rows  predictor projections (Sec. 3.3.3): z = P1 h and scores = P2 z.
//             One wave per output row; 16-byte nontemporal loads of the row,
//             the fp32 input vector read through the L1, butterfly row sum.
//  select     priority list (Sec. 2.1): deterministic top-k / threshold /
//             batch union over fp32 scores, one workgroup, rank by counting.
//  gateup     gate/up row gather for the selected blocks plus the gating of
//             Eq. 1, one wave per neuron; writes a in priority-list order.
//  down       down projection as the sum over hidden neurons (Sec. 3.2.2) plus
//             the residual of Eq. 2, one workgroup per 16-column tile over all
//             selected blocks, so no partial sums leave the workgroup.
//
// Every reduction has a fixed order: results are bitwise reproducible.
#include <atomic>

#include "ls_device.h"
#include "ls_internal.h"
#include "ls_sparse.h"

namespace ls {
namespace {

// ---- GEMV over rows: out[b, row] = c_b * sum_c W[row, c] * v[b, c] ------------------------
// c_b = rms_scale of v[b, :] when RMS (the MLP input of a prenorm stack), else 1.
// One workgroup of NW waves per R rows; the waves split the rows' 16-byte chunks, then a
// fixed-order sum of the wave totals.  The R rows share the input reads (with B tokens the
// input is B times the bytes of a row); every row's dot product is summed in the same order
// for any R.  U: 16-byte loads in flight per lane and row; a lane sums its chunks in ascending
// order whatever U is.
template <ls_dtype T, int B, bool RMS, int R, int NW, int U>
__global__ __launch_bounds__(64 * NW) void gemv_rows_kernel(const uint8_t* __restrict__ W, int rows,
                                                        int cols, int G, int rpw,
                                                        const float* __restrict__ v,
                                                        float* __restrict__ out) {
    constexpr int V = Wt<T>::V;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int row0 = blockIdx.x * R;
    const int nchunk = cols / V;
    const u32x4* wr[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int row = min(row0 + r, rows - 1);  // rows past the end repeat the last one, unstored
        const int srow = (row % G) * rpw + row / G;
        wr[r] = reinterpret_cast<const u32x4*>(W + (size_t)srow * cols * Wt<T>::kBytes);
    }
    float acc[R][B], ss[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
        ss[b] = 0.f;
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r][b] = 0.f;
    }
    // PRE (up to 3 tokens): the input chunks are requested with the weights, so the products
    // wait for one round trip; otherwise each chunk's input read is issued at its first use
    // (measured at 8 tokens, requesting them early was slower: 2260 against 2272 tokens/s on
    // the 13B shape), and so it is where they would take more than 32 registers of 16 bytes
    constexpr bool PRE = B <= 3 && U * B * (V / 4) <= 32;
    constexpr int UX = PRE ? U : 1;
    for (int c0 = threadIdx.x; c0 < nchunk; c0 += 64 * NW * U) {
        u32x4 raw[U][R];
        f32x4 xin[UX][PRE ? B : 1][V / 4];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + u * 64 * NW;
#pragma unroll
            for (int r = 0; r < R; ++r) raw[u][r] = c < nchunk ? ld_stream(wr[r] + c) : u32x4{0u, 0u, 0u, 0u};
        }
        if constexpr (PRE) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int c = min(c0 + u * 64 * NW, nchunk - 1);
#pragma unroll
                for (int b = 0; b < B; ++b)
#pragma unroll
                    for (int q = 0; q < V / 4; ++q)
                        xin[u][b][q] = reinterpret_cast<const f32x4*>(v + (size_t)b * cols + (size_t)c * V)[q];
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + u * 64 * NW;
            if (c < nchunk) {
                float w[R][V];
#pragma unroll
                for (int r = 0; r < R; ++r) Wt<T>::widen(raw[u][r], w[r]);
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    const f32x4* vp = reinterpret_cast<const f32x4*>(v + (size_t)b * cols + (size_t)c * V);
#pragma unroll
                    for (int q = 0; q < V / 4; ++q) {
                        const f32x4 x4 = PRE ? xin[PRE ? u : 0][PRE ? b : 0][q] : vp[q];
#pragma unroll
                        for (int r = 0; r < R; ++r) {
                            acc[r][b] = fmaf(w[r][4 * q + 0], x4.x, acc[r][b]);
                            acc[r][b] = fmaf(w[r][4 * q + 1], x4.y, acc[r][b]);
                            acc[r][b] = fmaf(w[r][4 * q + 2], x4.z, acc[r][b]);
                            acc[r][b] = fmaf(w[r][4 * q + 3], x4.w, acc[r][b]);
                        }
                        if (RMS) {
                            ss[b] = fmaf(x4.x, x4.x, ss[b]);
                            ss[b] = fmaf(x4.y, x4.y, ss[b]);
                            ss[b] = fmaf(x4.z, x4.z, ss[b]);
                            ss[b] = fmaf(x4.w, x4.w, ss[b]);
                        }
                    }
                }
            }
        }
    }
    __shared__ float part[NW][R][B], pss[NW][B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float s = wave_sum_dpp(acc[r][b]);
            if (lane == 0) part[wave][r][b] = s;
        }
        const float q = RMS ? wave_sum_dpp(ss[b]) : 0.f;
        if (lane == 0) pss[wave][b] = q;
    }
    __syncthreads();
    if (threadIdx.x < R * B) {
        const int r = threadIdx.x / B, b = threadIdx.x % B;
        float dot = 0.f, q = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) dot += part[w][r][b], q += pss[w][b];
        const float sc = RMS ? rms_scale(q, cols) : 1.f;
        if (row0 + r < rows) out[(size_t)b * rows + row0 + r] = dot * sc;
    }
}

// ---- block selection --------------------------------------------------------------------
// One workgroup.  Wave w selects for tokens w, w + waves, ...: the keys of a token sit in
// registers (Q per lane); top-k finds the k-th largest key T by a bitwise search with wave
// ballots (the largest T with at least k keys >= T) and takes every key > T plus the first
// keys equal to T by index; the threshold test is key > key(tau) on non-NaN scores.  Members
// are compacted by ballot prefix, then ranked among themselves (key descending, index
// ascending) so the output is in priority order.  Union: the OR of the tokens' sets, ranked
// by each block's largest key over all tokens.
// Ranking packs (key, 0xffff - index) into one 64-bit word, so the priority order is the
// descending order of distinct words and a member's rank is the count of larger words; the
// lists are padded with zero words (below every member) to a multiple of 8 so the count
// runs 8 independent LDS reads at a time.
// Q: keys per lane (n <= 64 Q); small lists get a small unrolled body.
__device__ inline uint64_t rank_word(uint32_t key, int i) {
    return ((uint64_t)key << 32) | (uint32_t)(0xffff - i);
}

__device__ inline int rank_in(const uint64_t* __restrict__ w, int n_pad, uint64_t mine) {
    int rank = 0;
#pragma unroll 1
    for (int j = 0; j < n_pad; j += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u) rank += w[j + u] > mine;
    }
    return rank;
}

// One token's selection by one wave.  With a union: fold the members into bkey (largest key
// per block) and umask (OR of the member sets); otherwise rank them through mk (an LDS row of
// at least n + 8 words) and write out_idx[rank] = block index and out_count[0].
template <int Q>
__device__ __forceinline__ void select_token(const float* __restrict__ row, int n, int mode, int k, float tau,
                                             int lane, bool UNION, uint64_t* mk, uint32_t* bkey, uint32_t* umask,
                                             int32_t* __restrict__ out_idx, int32_t* __restrict__ out_count) {
    const uint64_t below = (1ull << lane) - 1ull;
    const int Qn = (n + 63) / 64;
    // all Q loads in flight before the first use (indices past n re-read entry n - 1, n >= 1)
    float sv[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) sv[q] = row[min(q * 64 + lane, n - 1)];
    // entries past n get key 0: below every search candidate (>= 1) and never > T
    uint32_t ok[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int i = q * 64 + lane;
        ok[q] = i < n ? order_key(sv[q]) : 0u;
        if (UNION && i < n) atomicMax(&bkey[i], ok[q]);
    }
    // membership rule: key > T, or key == T among the first `rem` such by index
    uint32_t T = 0u;
    int rem = 0;
    const bool thr_mode = mode != LS_SEL_TOPK;
    if (!thr_mode) {
        auto step = [&](int bit) {
            const uint32_t c = T | (1u << bit);
            int cnt = 0;
#pragma unroll
            for (int q = 0; q < Q; ++q) cnt += __popcll(__ballot(ok[q] >= c));
            if (cnt >= k) T = c;
        };
        int bit = 31;
        for (; bit >= 16; --bit) step(bit);
        // top 16 bits decided: with exactly k keys at or above them the members are every
        // such key whatever T's low bits become (ties at T are then all taken), so the low
        // steps are skipped; T != 0 keeps the padding out of the count
        int ge = 0;
        if (T != 0u) {
#pragma unroll
            for (int q = 0; q < Q; ++q) ge += __popcll(__ballot(ok[q] >= T));
        }
        if (ge != k)
            for (; bit >= 0; --bit) step(bit);
        int gt = 0;
#pragma unroll
        for (int q = 0; q < Q; ++q) gt += __popcll(__ballot(ok[q] > T));
        rem = k - gt;
    }
    const uint32_t ktau = isnan(tau) ? 0xffffffffu : order_key(tau);
    int m = 0, eq_before = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        if (q < Qn) {
            const int i = q * 64 + lane;
            const bool valid = i < n;
            bool mem;
            if (thr_mode) {
                mem = valid && ok[q] != 0u && ok[q] > ktau;
            } else {
                const bool eq = valid && ok[q] == T;
                const uint64_t eqb = __ballot(eq);
                mem = valid && (ok[q] > T || (eq && eq_before + __popcll(eqb & below) < rem));
                eq_before += __popcll(eqb);
            }
            const uint64_t mb = __ballot(mem);
            if (mem) {
                if (UNION)
                    atomicOr(&umask[i >> 5], 1u << (i & 31));
                else
                    mk[m + __popcll(mb & below)] = rank_word(ok[q], i);
            }
            m += __popcll(mb);
        }
    }
    if (!UNION) {
        const int m_pad = (m + 7) & ~7;
        if (lane < m_pad - m) mk[m + lane] = 0ull;
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront", "local");
        for (int p = lane; p < m; p += 64) {
            const uint64_t mine = mk[p];
            out_idx[rank_in(mk, m_pad, mine)] = 0xffff - (int)(uint32_t)mine;
        }
        if (lane == 0) out_count[0] = m;
    }
}

template <int Q>
__global__ __launch_bounds__(Q > 8 ? 512 : 1024) void select_kernel(const float* __restrict__ scores, int B,
                                                      int n, int mode, int k, float tau,
                                                      int union_batch, int cap,
                                                      int32_t* __restrict__ idx,
                                                      int32_t* __restrict__ count) {
    // per token: its members' rank words; with a union, row 0 holds the union's instead
    __shared__ uint64_t mk[kMaxBatch][kMaxBlocks];
    __shared__ uint32_t bkey[kMaxBlocks];           // union: largest key of block i over all tokens
    __shared__ uint32_t umask[kMaxBlocks / 32];     // union: OR of the tokens' member sets
    __shared__ int ucount;
    const int tid = threadIdx.x, nt = blockDim.x;
    const int wave = tid >> 6, lane = tid & 63, nwaves = nt >> 6;
    const bool do_union = union_batch && B > 1;
    const uint64_t below = (1ull << lane) - 1ull;
    const int Qn = (n + 63) / 64;
    if (do_union) {
        for (int i = tid; i < n; i += nt) bkey[i] = 0u;
        for (int i = tid; i < (n + 31) / 32; i += nt) umask[i] = 0u;
        __syncthreads();
    }
    for (int b = wave; b < B; b += nwaves) {
        select_token<Q>(scores + (size_t)b * n, n, mode, k, tau, lane, do_union, mk[b], bkey, umask,
                        idx + (size_t)b * cap, count + b);
    }
    if (!do_union) return;
    __syncthreads();
    // union members with their largest keys, compacted by wave 0 into row 0
    if (wave == 0) {
        int u = 0;
        for (int q = 0; q < Qn; ++q) {
            const int i = q * 64 + lane;
            const bool in = i < n && ((umask[i >> 5] >> (i & 31)) & 1u);
            const uint64_t ub = __ballot(in);
            if (in) mk[0][u + __popcll(ub & below)] = rank_word(bkey[i], i);
            u += __popcll(ub);
        }
        const int u_pad = (u + 7) & ~7;
        if (lane < u_pad - u) mk[0][u + lane] = 0ull;
        if (lane == 0) ucount = u;
    }
    __syncthreads();
    const int U = ucount, U_pad = (U + 7) & ~7;
    for (int p = tid; p < U; p += nt) {
        const uint64_t mine = mk[0][p];
        idx[rank_in(mk[0], U_pad, mine)] = 0xffff - (int)(uint32_t)mine;
    }
    if (tid == 0) count[0] = U;
}

// ---- gate/up gather + gating: one wave per neuron of list entries [begin, end) ------------
// HS: the B x d input is first copied to LDS (dynamic shared memory of B d floats), once per
// workgroup instead of once per wave from L2; the copy starts once the first row loads are in
// flight.  The sums are the same either way.
template <ls_dtype T, ls_act A, int B, bool RMS, bool ZS, int U, bool HS>
__global__ __launch_bounds__(256) void gateup_kernel(
    const uint8_t* __restrict__ blocks, size_t block_bytes, const int32_t* __restrict__ slot_table,
    const void* __restrict__ bias, float thresh, const float* __restrict__ h, int d, int blk,
    int n_blk, int F, const int32_t* __restrict__ idx, const int32_t* __restrict__ count, int begin,
    int end, float* __restrict__ a_buf) {
    const long t = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int e = begin + (int)(t / blk);
    const int q = (int)(t % blk);
    const int lane = threadIdx.x & 63;
    if constexpr (HS) {
        extern __shared__ f32x4 hs[];
        auto prep = [&] {
            const f32x4* src = reinterpret_cast<const f32x4*>(h);
            for (int i = threadIdx.x; i < B * d / 4; i += 256) hs[i] = src[i];
            // a barrier that orders LDS only: the row loads already issued stay in flight
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        };
        if (e >= list_end(count, end, n_blk)) {  // a wave past the list still joins the barrier
            prep();
            return;
        }
        gateup_neuron<T, A, B, RMS, ZS, false, U>(blocks, block_bytes, slot_table, bias, thresh,
                                                  reinterpret_cast<const float*>(hs), d, blk, n_blk, F, idx[e], e, q,
                                                  a_buf, lane, prep);
    } else {
        if (e >= list_end(count, end, n_blk)) return;
        gateup_neuron<T, A, B, RMS, ZS, false, U>(blocks, block_bytes, slot_table, bias, thresh, h, d, blk, n_blk, F,
                                                  idx[e], e, q, a_buf, lane);
    }
}

// ---- batch 1: the selection and the gate/up gather in one launch --------------------------
// Wave 0 of every workgroup ranks the token's scores into LDS with the selection kernel's own
// code (so the list is the same) while the other waves copy the input to LDS; after one barrier
// each wave takes its neuron of the list, exactly as gateup_kernel with the input in LDS.
// Workgroup 0 also writes the list and its length for the down projection.  Every workgroup
// repeats the ranking of a few hundred keys, which costs about what the separate selection
// launch did and saves that launch.
template <ls_dtype T, ls_act A, bool RMS, int U, int Q>
__global__ __launch_bounds__(256) void gateup_select_kernel(
    const uint8_t* __restrict__ blocks, size_t block_bytes, const void* __restrict__ bias, float thresh,
    const float* __restrict__ h, int d, int blk, int n_blk, int F, const float* __restrict__ scores, int k,
    int32_t* __restrict__ idx, int32_t* __restrict__ count, float* __restrict__ a_buf) {
    extern __shared__ f32x4 hs[];
    __shared__ uint64_t mk[Q * 64 + 8];
    __shared__ int32_t list[Q * 64];
    __shared__ int32_t lcount;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (wave == 0) {
        select_token<Q>(scores, n_blk, LS_SEL_TOPK, k, 0.f, lane, false, mk, nullptr, nullptr, list, &lcount);
    } else {
        const f32x4* src = reinterpret_cast<const f32x4*>(h);
        for (int i = (int)threadIdx.x - 64; i < d / 4; i += 192) hs[i] = src[i];
    }
    __syncthreads();
    const int n = lcount;
    if (blockIdx.x == 0) {
        for (int i = threadIdx.x; i < n; i += 256) idx[i] = list[i];
        if (threadIdx.x == 0) count[0] = n;
    }
    const long t = (long)blockIdx.x * 4 + wave;
    const int e = (int)(t / blk), q = (int)(t % blk);
    if (e >= n) return;
    gateup_neuron<T, A, 1, RMS, false, false, U>(blocks, block_bytes, nullptr, bias, thresh,
                                                 reinterpret_cast<const float*>(hs), d, blk, n_blk, F, list[e], e,
                                                 q, a_buf, lane);
}

// ---- down projection + residual: one workgroup of kDnWaves waves per 16-column tile ------
// G: (entry, chunk pair) items whose loads each wave issues together.
// AS: the range's activations (B (end - begin) blk floats, at most kDownActs) are first copied
// to LDS, so the products read them there instead of from L2; the copy starts once the first
// weight loads are in flight.  The sums are the same either way.
constexpr int kDownActs = 12288;
constexpr int kDnWaves = 16;  // a compute unit needs about 16 waves of scattered reads to stream

// OCC: workgroups that must fit in a compute unit together (2: at most 64 registers a lane),
// for a tile count above the CU count, so that the extra tiles run beside the others.
template <ls_dtype T, int B, bool ZS, int G, bool AS, int OCC>
__global__ __launch_bounds__(64 * kDnWaves) __attribute__((amdgpu_waves_per_eu(OCC * kDnWaves / 4))) void down_kernel(
    const uint8_t* __restrict__ blocks, size_t block_bytes, const int32_t* __restrict__ slot_table,
    const float* __restrict__ a_buf, int F, int d, int blk, int n_blk,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ count, int begin, int end,
    const float* __restrict__ x_in, float* __restrict__ x_acc) {
    __shared__ float part[kDnVirt][kMaxBatch][kColTile];
    const int n_end = list_end(count, end, n_blk);
    auto sync = [] { __syncthreads(); };
    if constexpr (AS) {
        __shared__ f32x4 acts[kDownActs / 4];
        const int n4 = (n_end > begin ? n_end - begin : 0) * blk / 4;  // vectors per token
        auto prep = [&] {
            const f32x4* src = reinterpret_cast<const f32x4*>(a_buf + (size_t)begin * blk);
            for (int i = threadIdx.x; i < B * n4; i += 64 * kDnWaves) {
                const int tok = i / n4, j = i - tok * n4;
                acts[i] = src[(size_t)tok * (F / 4) + j];
            }
            // a barrier that orders LDS only: the weight loads already issued stay in flight
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        };
        down_tile<T, B, ZS, false, G, kDnWaves>(blocks, block_bytes, slot_table, reinterpret_cast<const float*>(acts),
                                                4 * n4, d, blk, n_blk, idx, begin, n_end, x_in, x_acc, blockIdx.x,
                                                threadIdx.x >> 6, threadIdx.x & 63, true, part, sync, begin, prep);
    } else {
        down_tile<T, B, ZS, false, G, kDnWaves>(blocks, block_bytes, slot_table, a_buf, F, d, blk, n_blk, idx, begin,
                                                n_end, x_in, x_acc, blockIdx.x, threadIdx.x >> 6, threadIdx.x & 63,
                                                true, part, sync);
    }
}

}  // namespace

template <ls_dtype T, ls_act A>
static hipError_t gateup_select_t(const Shape& s, const LayerDev& L, const float* h, const float* scores, int k,
                                  int32_t* idx, int32_t* count, float* a_buf, hipStream_t st) {
    const long tasks = (long)k * s.blk;
    const dim3 grid((unsigned)((tasks + 3) / 4)), blk(256);
    const size_t bb = s.block_elems * elem_size(s.dtype);
    const size_t hs_bytes = (size_t)s.d * sizeof(float);
    const int per_lane = (s.d / Wt<T>::V + 63) / 64;
#define LS_GS_K(RMS, U, Q)                                                                                    \
    hipLaunchKernelGGL((gateup_select_kernel<T, A, RMS, U, Q>), grid, blk, hs_bytes, st, L.blocks, bb, L.bias, \
                       L.threshold, h, s.d, s.blk, s.n_blk, s.F, scores, k, idx, count, a_buf)
#define LS_GS_Q(RMS, U)                                     \
    do {                                                    \
        if (s.n_blk <= 128) LS_GS_K(RMS, U, 2);             \
        else if (s.n_blk <= 192) LS_GS_K(RMS, U, 3);        \
        else if (s.n_blk <= 256) LS_GS_K(RMS, U, 4);        \
        else LS_GS_K(RMS, U, 8);                            \
    } while (0)
#define LS_GS_U(RMS)                                        \
    do {                                                    \
        if (per_lane <= 4) LS_GS_Q(RMS, 4);                 \
        else if (per_lane <= 8) LS_GS_Q(RMS, 8);            \
        else if (per_lane <= 12) LS_GS_Q(RMS, 12);          \
        else LS_GS_Q(RMS, 16);                              \
    } while (0)
    if (s.prenorm) LS_GS_U(true); else LS_GS_U(false);
#undef LS_GS_U
#undef LS_GS_Q
#undef LS_GS_K
    return hipGetLastError();
}

bool gateup_select_ok(const Shape& s, int B, int k) {
    return B == 1 && !s.zero_skip && k >= 1 && k <= s.n_blk && s.n_blk <= 512 &&
           (size_t)s.d * sizeof(float) <= 32768;
}

hipError_t launch_gateup_select(const Shape& s, const LayerDev& L, const float* h, const float* scores, int k,
                                int32_t* idx, int32_t* count, float* a_buf, hipStream_t st) {
    if (k < 1) return hipSuccess;
    const bool relu = s.act == LS_ACT_REGLU;
    switch (s.dtype) {
        case LS_F32:
            return relu ? gateup_select_t<LS_F32, LS_ACT_REGLU>(s, L, h, scores, k, idx, count, a_buf, st)
                        : gateup_select_t<LS_F32, LS_ACT_SWIGLU_THRESH>(s, L, h, scores, k, idx, count, a_buf, st);
        case LS_F16:
            return relu ? gateup_select_t<LS_F16, LS_ACT_REGLU>(s, L, h, scores, k, idx, count, a_buf, st)
                        : gateup_select_t<LS_F16, LS_ACT_SWIGLU_THRESH>(s, L, h, scores, k, idx, count, a_buf, st);
        case LS_BF16:
            return relu ? gateup_select_t<LS_BF16, LS_ACT_REGLU>(s, L, h, scores, k, idx, count, a_buf, st)
                        : gateup_select_t<LS_BF16, LS_ACT_SWIGLU_THRESH>(s, L, h, scores, k, idx, count, a_buf, st);
    }
    return hipErrorInvalidValue;
}



template <ls_dtype T, bool RMS>
static hipError_t gemv_t(const void* W, int rows, int cols, int G, int rpw, const float* v, int B,
                         float* out, hipStream_t st) {
    // four rows and eight waves per workgroup once the batch makes the input reads dominate;
    // one row per workgroup below, on eight waves at batch 1 (against four: 7B shape 1664 ->
    // 1681 tokens/s, 13B 1106 -> 1114 on the per-kernel path) and four at B = 2, 3
    const int R = B >= 4 ? 4 : 1, NW = B >= 4 || B == 1 ? 8 : 4;
    const dim3 grid((unsigned)((rows + R - 1) / R)), blk(64 * NW);
    const uint8_t* w = static_cast<const uint8_t*>(W);
    // a row longer than 4 loads per lane is read in one round of 8
    const bool wide = cols / Wt<T>::V > 64 * NW * 4;
#define LS_GEMV_U(NB, NR, NWV, U) hipLaunchKernelGGL((gemv_rows_kernel<T, NB, RMS, NR, NWV, U>), grid, blk, 0, st, w, rows, cols, G, rpw, v, out)
#define LS_GEMV(NB, NR, NWV) LS_GEMV_U(NB, NR, NWV, 4)
    switch (B) {
        case 1: if (wide) LS_GEMV_U(1, 1, 8, 8); else LS_GEMV(1, 1, 8); break;
        case 2: if (wide) LS_GEMV_U(2, 1, 4, 8); else LS_GEMV(2, 1, 4); break;
        case 3: if (wide) LS_GEMV_U(3, 1, 4, 8); else LS_GEMV(3, 1, 4); break;
        case 4: LS_GEMV(4, 4, 8); break;
        case 5: LS_GEMV(5, 4, 8); break;
        case 6: LS_GEMV(6, 4, 8); break;
        case 7: LS_GEMV(7, 4, 8); break;
        case 8: LS_GEMV(8, 4, 8); break;
        default: return hipErrorInvalidValue;
    }
#undef LS_GEMV
#undef LS_GEMV_U
    return hipGetLastError();
}

hipError_t launch_gemv_rows(ls_dtype t, const void* W, int rows, int cols, int G, int rpw,
                            const float* v, int B, bool rms, float* out, hipStream_t st) {
    switch (t) {
        case LS_F32: return rms ? gemv_t<LS_F32, true>(W, rows, cols, G, rpw, v, B, out, st)
                                : gemv_t<LS_F32, false>(W, rows, cols, G, rpw, v, B, out, st);
        case LS_F16: return rms ? gemv_t<LS_F16, true>(W, rows, cols, G, rpw, v, B, out, st)
                                : gemv_t<LS_F16, false>(W, rows, cols, G, rpw, v, B, out, st);
        case LS_BF16: return rms ? gemv_t<LS_BF16, true>(W, rows, cols, G, rpw, v, B, out, st)
                                 : gemv_t<LS_BF16, false>(W, rows, cols, G, rpw, v, B, out, st);
    }
    return hipErrorInvalidValue;
}

// Folding the predictor factors: a workgroup owns 8 rows of the product and 256 columns;
// the 8 x 64 tile of P2 for the current m-range is shared through LDS.
template <ls_dtype T>
__global__ __launch_bounds__(256) void fold_predictor_kernel(const void* __restrict__ P1,
                                                             const void* __restrict__ P2, int r,
                                                             int d, int n_blk,
                                                             float* __restrict__ out) {
    constexpr int R = 8, M = 64;
    __shared__ double p2s[R][M];
    const int j = blockIdx.x * 256 + threadIdx.x;
    const int i0 = blockIdx.y * R;
    double acc[R];
#pragma unroll
    for (int ii = 0; ii < R; ++ii) acc[ii] = 0.0;
    for (int m0 = 0; m0 < r; m0 += M) {
        for (int t = threadIdx.x; t < R * M; t += 256) {
            const int ii = t / M, m = m0 + t % M;
            p2s[ii][t % M] = (i0 + ii < n_blk && m < r) ? (double)Wt<T>::scalar(P2, (size_t)(i0 + ii) * r + m) : 0.0;
        }
        __syncthreads();
        if (j < d) {
            const int mend = min(M, r - m0);
            for (int mm = 0; mm < mend; ++mm) {
                const double pv = (double)Wt<T>::scalar(P1, (size_t)(m0 + mm) * d + j);
#pragma unroll
                for (int ii = 0; ii < R; ++ii) acc[ii] = fma(p2s[ii][mm], pv, acc[ii]);
            }
        }
        __syncthreads();
    }
    if (j < d) {
#pragma unroll
        for (int ii = 0; ii < R; ++ii)
            if (i0 + ii < n_blk) out[(size_t)(i0 + ii) * d + j] = (float)acc[ii];
    }
}

hipError_t launch_fold_predictor(ls_dtype t, const void* P1, const void* P2, int r, int d, int n_blk,
                                 float* out, hipStream_t st) {
    if (r < 1 || d < 1 || n_blk < 1) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((d + 255) / 256), (unsigned)((n_blk + 7) / 8)), blk(256);
    switch (t) {
        case LS_F32: hipLaunchKernelGGL(fold_predictor_kernel<LS_F32>, grid, blk, 0, st, P1, P2, r, d, n_blk, out); break;
        case LS_F16: hipLaunchKernelGGL(fold_predictor_kernel<LS_F16>, grid, blk, 0, st, P1, P2, r, d, n_blk, out); break;
        case LS_BF16: hipLaunchKernelGGL(fold_predictor_kernel<LS_BF16>, grid, blk, 0, st, P1, P2, r, d, n_blk, out); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_select(const float* scores, int B, int n_blk, int mode, int k, float tau,
                         int union_batch, int cap, int32_t* idx, int32_t* count, hipStream_t st) {
    // one wave per token; more waves share the union ranking
    int waves = (n_blk + 63) / 64;
    waves = waves < B ? B : waves;
    const int max_waves = n_blk <= 512 ? 16 : 8;  // the widest body needs 256 registers a lane
    waves = waves > max_waves ? max_waves : waves;
    const int threads = 64 * waves;
    // key slots per lane: only as many as n_blk needs (the search's time follows its
    // instruction count)
    auto fn = n_blk <= 128   ? select_kernel<2>
              : n_blk <= 192 ? select_kernel<3>
              : n_blk <= 256 ? select_kernel<4>
              : n_blk <= 512 ? select_kernel<8>
                             : select_kernel<kMaxBlocks / 64>;
    hipLaunchKernelGGL(fn, dim3(1), dim3(threads), 0, st, scores, B, n_blk, mode, k, tau,
                       union_batch, cap, idx, count);
    return hipGetLastError();
}

// compute units of the current device (0 when unknown), queried once per device
static int cu_count() {
    static std::atomic<int> cached[64];
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (dev >= 0 && dev < 64 && (cus = cached[dev].load(std::memory_order_relaxed)) > 0) return cus;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) return 0;
    if (dev >= 0 && dev < 64) cached[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

template <ls_dtype T, ls_act A>
static hipError_t gateup_t(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                           const float* h, int B, const int32_t* idx, const int32_t* count,
                           int begin, int end, float* a_buf, hipStream_t st) {
    const long tasks = (long)(end - begin) * s.blk;
    if (tasks <= 0) return hipSuccess;
    const dim3 grid((unsigned)((tasks + 3) / 4)), blk(256);
    const size_t bb = s.block_elems * elem_size(s.dtype);
    // the input goes through LDS while it takes at most 32 KB (five or more workgroups per CU)
    const size_t hs_bytes = (size_t)B * s.d * sizeof(float);
    const bool hs = hs_bytes <= 32768;
#define LS_GU_KU(NB, RMS, ZS, U)                                                                          \
    do {                                                                                                  \
        if (hs)                                                                                           \
            hipLaunchKernelGGL((gateup_kernel<T, A, NB, RMS, ZS, U, true>), grid, blk, hs_bytes, st, L.blocks, bb, \
                               slot_table, L.bias, L.threshold, h, s.d, s.blk, s.n_blk, s.F, idx, count, begin, end, \
                               a_buf);                                                                    \
        else                                                                                              \
            hipLaunchKernelGGL((gateup_kernel<T, A, NB, RMS, ZS, U, false>), grid, blk, 0, st, L.blocks, bb, \
                               slot_table, L.bias, L.threshold, h, s.d, s.blk, s.n_blk, s.F, idx, count, begin, end, \
                               a_buf);                                                                    \
    } while (0)
    // at batch 1 a wave issues every load of its two rows at once (up to 16 chunks per lane)
    const int per_lane = (s.d / Wt<T>::V + 63) / 64;
#define LS_GU_K(NB, RMS, ZS)                                                  \
    do {                                                                      \
        if (NB > 1 || ZS || per_lane <= 4) LS_GU_KU(NB, RMS, ZS, 4);          \
        else if (per_lane <= 8) LS_GU_KU(NB, RMS, ZS, (NB > 1 || ZS ? 4 : 8));  \
        else if (per_lane <= 12) LS_GU_KU(NB, RMS, ZS, (NB > 1 || ZS ? 4 : 12)); \
        else LS_GU_KU(NB, RMS, ZS, (NB > 1 || ZS ? 4 : 16));                   \
    } while (0)
#define LS_GU(NB)                                                                 \
    do {                                                                          \
        if (s.prenorm) {                                                          \
            if (s.zero_skip) LS_GU_K(NB, true, true); else LS_GU_K(NB, true, false);   \
        } else {                                                                  \
            if (s.zero_skip) LS_GU_K(NB, false, true); else LS_GU_K(NB, false, false); \
        }                                                                         \
    } while (0)
    switch (B) {
        case 1: LS_GU(1); break;
        case 2: LS_GU(2); break;
        case 3: LS_GU(3); break;
        case 4: LS_GU(4); break;
        case 5: LS_GU(5); break;
        case 6: LS_GU(6); break;
        case 7: LS_GU(7); break;
        case 8: LS_GU(8); break;
        default: return hipErrorInvalidValue;
    }
#undef LS_GU
#undef LS_GU_K
#undef LS_GU_KU
    return hipGetLastError();
}

hipError_t launch_gateup(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                         const float* h, int B, const int32_t* idx, const int32_t* count,
                         int begin, int end, float* a_buf, hipStream_t st) {
    if (s.batch_mfma && !s.zero_skip && mfma_path(s, B))
        return launch_gateup_mfma(s, L, slot_table, h, B, idx, count, begin, end, a_buf, st);
    const bool relu = s.act == LS_ACT_REGLU;
    switch (s.dtype) {
        case LS_F32:
            return relu ? gateup_t<LS_F32, LS_ACT_REGLU>(s, L, slot_table, h, B, idx, count, begin, end, a_buf, st)
                        : gateup_t<LS_F32, LS_ACT_SWIGLU_THRESH>(s, L, slot_table, h, B, idx, count, begin, end, a_buf, st);
        case LS_F16:
            return relu ? gateup_t<LS_F16, LS_ACT_REGLU>(s, L, slot_table, h, B, idx, count, begin, end, a_buf, st)
                        : gateup_t<LS_F16, LS_ACT_SWIGLU_THRESH>(s, L, slot_table, h, B, idx, count, begin, end, a_buf, st);
        case LS_BF16:
            return relu ? gateup_t<LS_BF16, LS_ACT_REGLU>(s, L, slot_table, h, B, idx, count, begin, end, a_buf, st)
                        : gateup_t<LS_BF16, LS_ACT_SWIGLU_THRESH>(s, L, slot_table, h, B, idx, count, begin, end, a_buf, st);
    }
    return hipErrorInvalidValue;
}

// Items of loads in flight per wave (an item: 2 vectors of 16 bytes per lane): 2 up to B = 3
// (zero skip: at batch 1), where each wave then reaches its first products sooner (with 8:
// Mistral-7B shape at batch 1 751 against 768 tokens/s, 7B shape 1587 against 1662 on the
// per-kernel path, 13B shape at B = 2 1192 against 1288, 7B shape with zero skip 1473 against
// 1578; 3 and 4 in between); 4 where the per-token sums (B >= 4) or the zero-skip tests
// (B >= 2) take the registers.
constexpr int down_items(int B, bool ZS) { return (ZS ? B == 1 : B <= 3) ? 2 : 4; }

template <ls_dtype T, int NB, bool ZS, bool AS>
static void down_launch(const Shape& s, const LayerDev& L, const int32_t* slot_table, const float* a_buf,
                        const int32_t* idx, const int32_t* count, int begin, int end, const float* x_in,
                        float* x_acc, bool two, hipStream_t st) {
    const dim3 grid(s.d / kColTile), blk(64 * kDnWaves);
    const size_t bb = s.block_elems * elem_size(s.dtype);
    if constexpr (NB == 1 && !ZS) {
        if (two) {
            hipLaunchKernelGGL((down_kernel<T, NB, ZS, 2, AS, 2>), grid, blk, 0, st, L.blocks, bb, slot_table, a_buf,
                               s.F, s.d, s.blk, s.n_blk, idx, count, begin, end, x_in, x_acc);
            return;
        }
    }
    hipLaunchKernelGGL((down_kernel<T, NB, ZS, down_items(NB, ZS), AS, 1>), grid, blk, 0, st, L.blocks, bb,
                       slot_table, a_buf, s.F, s.d, s.blk, s.n_blk, idx, count, begin, end, x_in, x_acc);
}

template <ls_dtype T>
static hipError_t down_t(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                         const float* a_buf, int B, const int32_t* idx, const int32_t* count,
                         int begin, int end, const float* x_in, float* x_acc, hipStream_t st) {
    const bool as = (long)B * (end - begin) * s.blk <= kDownActs && s.F % 4 == 0;
    // more tiles than CUs (d = 5120: 320 tiles): at batch 1, two workgroups per CU with 2 items
    // of loads in flight per wave instead of one with 8, so the extra tiles run beside the others
    const bool two = B == 1 && !s.zero_skip && s.d / kColTile > cu_count();
#define LS_DN_K(NB, ZS, AS) \
    down_launch<T, NB, ZS, AS>(s, L, slot_table, a_buf, idx, count, begin, end, x_in, x_acc, two, st)
#define LS_DN(NB)                                                                                   \
    do {                                                                                            \
        if (s.zero_skip) {                                                                          \
            if (as) LS_DN_K(NB, true, true); else LS_DN_K(NB, true, false);                         \
        } else {                                                                                    \
            if (as) LS_DN_K(NB, false, true); else LS_DN_K(NB, false, false);                       \
        }                                                                                           \
    } while (0)
    switch (B) {
        case 1: LS_DN(1); break;
        case 2: LS_DN(2); break;
        case 3: LS_DN(3); break;
        case 4: LS_DN(4); break;
        case 5: LS_DN(5); break;
        case 6: LS_DN(6); break;
        case 7: LS_DN(7); break;
        case 8: LS_DN(8); break;
        default: return hipErrorInvalidValue;
    }
#undef LS_DN
#undef LS_DN_K
    return hipGetLastError();
}

hipError_t launch_down(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                       const float* a_buf, int B, const int32_t* idx, const int32_t* count,
                       int begin, int end, const float* x_in, float* x_acc, float* part,
                       hipStream_t st) {
    if (s.batch_mfma && !s.zero_skip && mfma_path(s, B))
        return launch_down_mfma(s, L, slot_table, a_buf, B, idx, count, begin, end, x_in, x_acc, part, st);
    switch (s.dtype) {
        case LS_F32: return down_t<LS_F32>(s, L, slot_table, a_buf, B, idx, count, begin, end, x_in, x_acc, st);
        case LS_F16: return down_t<LS_F16>(s, L, slot_table, a_buf, B, idx, count, begin, end, x_in, x_acc, st);
        case LS_BF16: return down_t<LS_BF16>(s, L, slot_table, a_buf, B, idx, count, begin, end, x_in, x_acc, st);
    }
    return hipErrorInvalidValue;
}

// ---- streaming-read ceiling (measurement) ------------------------------------------------
// Workgroup w reads the contiguous vector range [w n / G, (w + 1) n / G) of 16-byte vectors,
// eight loads in flight per thread, and folds them with XOR; each wave writes one word so the
// loads cannot be dropped.  out holds 4 words per workgroup.
__global__ __launch_bounds__(256) void read_probe_kernel(const u32x4* __restrict__ p, size_t n_vec,
                                                         uint32_t* __restrict__ out) {
    const size_t lo = (size_t)blockIdx.x * n_vec / gridDim.x;
    const size_t hi = (size_t)(blockIdx.x + 1) * n_vec / gridDim.x;
    uint32_t acc = 0;
    size_t i = lo + threadIdx.x;
    for (; i + 7 * 256 < hi; i += 8 * 256) {
        u32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = ld_stream(p + i + (size_t)u * 256);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < hi; i += 256) {
        const u32x4 v = ld_stream(p + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, off, 64);
    if ((threadIdx.x & 63) == 0) out[(size_t)blockIdx.x * 4 + (threadIdx.x >> 6)] = acc;
}

hipError_t launch_read_probe(const void* buf, size_t bytes, uint32_t* out, int grid, hipStream_t st) {
    hipLaunchKernelGGL(read_probe_kernel, dim3(grid), dim3(256), 0, st, static_cast<const u32x4*>(buf),
                       bytes / 16, out);
    return hipGetLastError();
}

}  // namespace ls
