// ls_mfma.hip - batched (B >= 4) gate/up and down kernels on the matrix cores of gfx950.
//
// With B tokens the gather GEMVs become small dense contractions: for a group of
// 16 neurons, [16 x d] weight rows times [d x B] activations.  These kernels run them as
// v_mfma_f32_16x16x32_{f16,bf16}: the weights are the A operand, loaded straight from
// their rows (one 16-byte load per lane per step), and the activations are the B operand,
// padded with zeros to 16 token columns.  Activations are fp32, so each one is split into
// a 16-bit "hi" part and the 16-bit rounding of the remainder ("lo"); W.hi + W.lo carries
// about 22 (f16) or 16 (bf16) significant bits of the activation, with fp32
// accumulation in the matrix cores.  Results match the VALU kernels to fp32 rounding
// (Eq. 1 of the paper, union over tokens as for the VALU path).
//
// Lane layout of v_mfma_f32_16x16x32 (lane l, i < 8 / i < 4):
//   A[l % 16][8 (l / 16) + i],  B[8 (l / 16) + i][l % 16],  C[4 (l / 16) + i][l % 16].
#include "ls_device.h"
#include "ls_internal.h"

namespace ls {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

// fp32 -> bfloat16 bits, round to nearest even (NaN stays a quiet NaN)
__device__ inline unsigned short bf16_rne(float x) {
    const unsigned u = __float_as_uint(x);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (unsigned short)((u >> 16) | 0x40u);
    return (unsigned short)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Split 8 fp32 values into hi and lo 16-bit operands of type T.
template <ls_dtype T>
struct Split;

template <>
struct Split<LS_F16> {
    typedef f16x8 vec;
    __device__ static inline void run(const float* x, vec& hi, vec& lo) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const _Float16 h = (_Float16)x[i];
            hi[i] = h;
            lo[i] = (_Float16)(x[i] - (float)h);
        }
    }
    __device__ static inline vec from_raw(const u32x4& r) {
        vec v;
        __builtin_memcpy(&v, &r, 16);
        return v;
    }
    __device__ static inline f32x4v mfma(const vec& a, const vec& b, const f32x4v& c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};

template <>
struct Split<LS_BF16> {
    typedef s16x8 vec;
    __device__ static inline void run(const float* x, vec& hi, vec& lo) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const unsigned short h = bf16_rne(x[i]);
            hi[i] = (short)h;
            lo[i] = (short)bf16_rne(x[i] - __uint_as_float((unsigned)h << 16));
        }
    }
    __device__ static inline vec from_raw(const u32x4& r) {
        vec v;
        __builtin_memcpy(&v, &r, 16);
        return v;
    }
    __device__ static inline f32x4v mfma(const vec& a, const vec& b, const f32x4v& c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

__device__ inline int list_end_m(const int32_t* count, int end, int n_blk) {
    int c = *count;
    c = c < 0 ? 0 : (c > n_blk ? n_blk : c);
    return end < c ? end : c;
}

constexpr int kWaves = 4;     // gate/up: waves per workgroup
constexpr int kRowsW = 32 / kWaves;  // gate/up: staged rows loaded by each wave per chunk
constexpr int kUnroll = 8;    // gate/up: K steps in flight per wave
constexpr int kUnrollDn = 4;  // down: (entry, K step) items in flight per wave, at most
constexpr int kWavesDn = 16;  // down: waves per workgroup (one 16-column tile)

// One workgroup per group of 16 neurons (rows r0..r0+15 of one list entry).  The gate and up
// rows of the group stream through LDS in chunks of 512 K values: each load instruction reads
// one kilobyte of one row (row-contiguous reads stream far better than the 16-row x 64-byte
// pattern of an MFMA operand), the 4 waves write them to LDS rows padded to 1040 bytes (so
// that the 16 lanes reading one fragment column hit different banks), and each wave then runs
// a quarter of the chunk's K steps from LDS while the next chunk's loads are in flight.
// a_buf[tok * F + e * blk + q] as the VALU kernel writes it.  x is the layer input; with RMS
// each lane also sums the squares of the x values it loads (every (token, k) exactly once per
// workgroup) and the dot products are scaled at the end.
constexpr int kChunkK = 512;                 // K values per chunk (1 KB of a 16-bit row)
constexpr int kLpr = 2 * kChunkK / 1024;     // 1 KB loads per staged row and chunk
constexpr int kRowPitch = 2 * kChunkK + 16;  // LDS bytes per staged row
// three waves per SIMD (at most 168 registers a lane): three workgroups per CU
constexpr int kGuWavesPerEu = 3;
template <ls_dtype T, ls_act A, bool RMS>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(kGuWavesPerEu))) void gateup_mfma_kernel(
    const uint8_t* __restrict__ blocks, size_t block_bytes, const int32_t* __restrict__ slot_table,
    const void* __restrict__ bias, float thresh, const float* __restrict__ h, int B, int d, int blk,
    int n_blk, int F, const int32_t* __restrict__ idx, const int32_t* __restrict__ count, int begin,
    int end, float* __restrict__ a_buf) {
    using S = Split<T>;
    __shared__ __attribute__((aligned(16))) uint8_t stage[32 * kRowPitch];  // rows 0-15 gate, 16-31 up
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int groups_per_entry = blk / 16;
    const int e = begin + (int)blockIdx.x / groups_per_entry;
    const int r0 = ((int)blockIdx.x % groups_per_entry) * 16;
    if (e >= list_end_m(count, end, n_blk)) return;
    const int b = idx[e];
    const int slot = (b < 0 || b >= n_blk) ? -1 : (slot_table ? slot_table[b] : b);
    if (slot < 0) {  // invalid id or block not in the cache: the entry contributes nothing
        if (threadIdx.x < 16 * B) {
            const int tok = threadIdx.x / 16, r = threadIdx.x % 16;
            a_buf[(size_t)tok * F + (size_t)e * blk + r0 + r] = 0.f;
        }
        return;
    }
    const size_t row_bytes = (size_t)d * 2;
    const uint8_t* base = blocks + (size_t)slot * block_bytes;
    const int tok = lane & 15;
    const bool tok_ok = tok < B;
    const float* hrow = h + (size_t)(tok_ok ? tok : 0) * d;
    // staged row j of this wave's loads: gate row r0 + j (j < 16) or up row r0 + j - 16
    auto row_ptr = [&](int j) {
        return base + (size_t)(j < 16 ? r0 + j : blk + r0 + j - 16) * row_bytes;
    };
    auto load_chunk = [&](int c0, u32x4 (&rw)[kRowsW * kLpr]) {
        const int bytes = 2 * min(kChunkK, d - c0);
#pragma unroll
        for (int i = 0; i < kRowsW; ++i) {
            const int j = wave + kWaves * i;
#pragma unroll
            for (int h = 0; h < kLpr; ++h) {
                const int off = 1024 * h + lane * 16;
                rw[i * kLpr + h] = off < bytes ? ld_stream(reinterpret_cast<const u32x4*>(row_ptr(j) + (size_t)c0 * 2 + off))
                                               : u32x4{0u, 0u, 0u, 0u};
            }
        }
    };
    // x of this wave's K steps of a chunk (s0 = wave + kWaves j), requested once the wave is
    // done with the previous chunk's (after the next chunk's weights: a wave waits for both
    // at the top of the chunk anyway)
    constexpr int kStepsW = kChunkK / 32 / kWaves;
    auto load_x = [&](int c0, f32x4 (&hx)[kStepsW][2]) {
        const int steps = min(kChunkK, d - c0) / 32;
#pragma unroll
        for (int j = 0; j < kStepsW; ++j) {
            const int s0 = wave + kWaves * j;
            const int kc = 32 * s0 + 8 * (lane >> 4);  // this lane's 8 K values in the chunk
            const f32x4 z = {0.f, 0.f, 0.f, 0.f};
            const bool ok = tok_ok && s0 < steps;
            hx[j][0] = ok ? reinterpret_cast<const f32x4*>(hrow + c0 + kc)[0] : z;
            hx[j][1] = ok ? reinterpret_cast<const f32x4*>(hrow + c0 + kc)[1] : z;
        }
    };
    f32x4v cg = {0.f, 0.f, 0.f, 0.f}, cu = {0.f, 0.f, 0.f, 0.f};
    float ss = 0.f;
    u32x4 rw[kRowsW * kLpr];
    f32x4 hx[kStepsW][2];
    load_chunk(0, rw);
    load_x(0, hx);
    for (int c0 = 0; c0 < d; c0 += kChunkK) {
        const int steps = min(kChunkK, d - c0) / 32;
        const bool more = c0 + kChunkK < d;
#pragma unroll
        for (int i = 0; i < kRowsW; ++i)
#pragma unroll
            for (int h = 0; h < kLpr; ++h)
                *reinterpret_cast<u32x4*>(stage + (wave + kWaves * i) * kRowPitch + 1024 * h + lane * 16) = rw[i * kLpr + h];
        __syncthreads();
        if (more) load_chunk(c0 + kChunkK, rw);  // in flight while this chunk runs
#pragma unroll
        for (int j = 0; j < kStepsW; ++j) {
            const int s0 = wave + kWaves * j;
            if (s0 >= steps) break;
            const int kc = 32 * s0 + 8 * (lane >> 4);
            const f32x4 h0 = hx[j][0], h1 = hx[j][1];
            const float xv[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
            if (RMS) {
#pragma unroll
                for (int i = 0; i < 8; ++i) ss = fmaf(xv[i], xv[i], ss);
            }
            typename S::vec hi, lo;
            S::run(xv, hi, lo);
            const u32x4 wg4 = *reinterpret_cast<const u32x4*>(stage + (lane & 15) * kRowPitch + kc * 2);
            const u32x4 wu4 = *reinterpret_cast<const u32x4*>(stage + (16 + (lane & 15)) * kRowPitch + kc * 2);
            const typename S::vec wg = S::from_raw(wg4), wu = S::from_raw(wu4);
            cg = S::mfma(wg, hi, cg);
            cg = S::mfma(wg, lo, cg);
            cu = S::mfma(wu, hi, cu);
            cu = S::mfma(wu, lo, cu);
        }
        if (more) load_x(c0 + kChunkK, hx);
        __syncthreads();  // every wave is done with the chunk before it is overwritten
    }
    // lane l holds rows 4 (l / 16) + i, token l % 16 of this wave's partial sums
    // the partial sums reuse the staging buffer (every wave is past the last chunk), so that
    // four workgroups fit in a compute unit's LDS
    static_assert(sizeof(float) * (2 * kWaves * 16 * 16 + kWaves * 16) <= sizeof(stage), "epilogue fits the stage");
    float (&pg)[kWaves][16][16] = *reinterpret_cast<float (*)[kWaves][16][16]>(stage);
    float (&pu)[kWaves][16][16] = *reinterpret_cast<float (*)[kWaves][16][16]>(stage + sizeof(float) * kWaves * 16 * 16);
    float (&pss)[kWaves][16] = *reinterpret_cast<float (*)[kWaves][16]>(stage + 2 * sizeof(float) * kWaves * 16 * 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        pg[wave][4 * (lane >> 4) + i][lane & 15] = cg[i];
        pu[wave][4 * (lane >> 4) + i][lane & 15] = cu[i];
    }
    if (RMS) {  // lanes l, l+16, l+32, l+48 hold the same token
        ss += __shfl_xor(ss, 16, 64);
        ss += __shfl_xor(ss, 32, 64);
        if (lane < 16) pss[wave][lane] = ss;
    }
    __syncthreads();
    if (threadIdx.x < 16 * B) {
        const int t = threadIdx.x / 16, r = threadIdx.x % 16;
        float sq = 0.f, gs = 0.f, us = 0.f;  // the waves' partial sums in wave order
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            sq += pss[w][t];
            gs += pg[w][r][t];
            us += pu[w][r][t];
        }
        const float sc = RMS ? rms_scale(sq, d) : 1.f;
        const float g = sc * gs +
                        (bias ? Wt<T>::scalar(bias, (size_t)b * blk + r0 + r) : 0.f);
        const float u = sc * us;
        float a;
        if (A == LS_ACT_REGLU) {
            a = fmaxf(g, 0.f) * u;
        } else {
            const float sg = g / (1.f + expf(-g));
            a = fabsf(sg) > thresh ? sg * u : 0.f;
        }
        a_buf[(size_t)t * F + (size_t)e * blk + r0 + r] = a;
    }
}

// One workgroup per NT adjacent 16-column tiles of y and part of the list; its waves split
// that part's entries.  The down piece of a block for one 16-column tile is [blk/8][16][8]:
// K step s of an entry is the contiguous kilobyte of chunks 64 s .. 64 s + 63, exactly one A
// fragment, and the pieces of adjacent tiles are adjacent.  A wave loads the activations of
// a work item once for its NT fragments: every workgroup reads the whole part's activations
// (L2 hits, but through the same per-CU memory path as the weights, which bounds these
// kernels), so NT tiles per workgroup divide those reads by NT.
// With splits > 1 the list range is cut into `splits` equal parts (workgroup
// tile + n_tiles * part) so that the workgroup count is a multiple of the CU count even when
// the tile count is not; each part's sum goes to part_out[part][token][column] and
// down_finish_kernel adds the parts in order.  The wave count is blockDim.x / 64 (at most
// kWavesDn, and at most kWavesDn / NT with NT > 1).
template <ls_dtype T, int NT, int KU>
__global__ __launch_bounds__(64 * kWavesDn) void down_mfma_kernel(
    const uint8_t* __restrict__ blocks, size_t block_bytes, const int32_t* __restrict__ slot_table,
    const float* __restrict__ a_buf, int B, int F, int d, int blk, int n_blk,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ count, int begin, int end,
    const float* __restrict__ x_in, float* __restrict__ x_acc, int splits,
    float* __restrict__ part_out) {
    using S = Split<T>;
    static_assert(KU >= 1 && KU <= kUnrollDn, "items in flight per wave");
    constexpr int kU = KU;
    const int n_tiles = d / (kColTile * NT);
    const int tile = (int)blockIdx.x % n_tiles, sp = (int)blockIdx.x / n_tiles;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int n_waves = (int)(blockDim.x >> 6);
    const int len = max(0, list_end_m(count, end, n_blk) - begin);
    const int e0 = begin + (int)((long)len * sp / splits);
    const int e1 = begin + (int)((long)len * (sp + 1) / splits);
    const size_t down_off = (size_t)2 * blk * d * 2 + (size_t)tile * NT * blk * kColTile * 2;
    const int piece_v = blk * kColTile * 2 / 16;  // 16-byte vectors of one tile's piece
    const int ksteps = blk / 32;
    const int tok = lane & 15;
    const bool tok_ok = tok < B;
    // the cache slot of every entry of the part (-1: invalid id or absent), resolved once so
    // that each work item waits only for its weight load
    __shared__ int slots[kMaxBlocks];
    for (int e = e0 + (int)threadIdx.x; e < e1; e += (int)blockDim.x) {
        const int b = idx[e];
        slots[e - e0] = (b < 0 || b >= n_blk) ? -1 : (slot_table ? slot_table[b] : b);
    }
    __syncthreads();
    f32x4v c[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) c[j] = f32x4v{0.f, 0.f, 0.f, 0.f};
    // work items (entry, K step) of the part, dealt to the waves round-robin; kU items per
    // wave are in flight together
    const long items = (long)(e1 - e0) * ksteps;
    for (long i0 = wave; i0 < items; i0 += (long)n_waves * kU) {
        const u32x4* src[kU];
        const float* arow[kU];
        bool live[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const long it = i0 + (long)n_waves * u;
            const int e = e0 + (int)(it / ksteps), s = (int)(it % ksteps);
            live[u] = it < items;
            const int slot = live[u] ? slots[e - e0] : -1;
            live[u] = live[u] && slot >= 0;  // an invalid or absent block contributes nothing
            src[u] = reinterpret_cast<const u32x4*>(blocks + (size_t)(slot < 0 ? 0 : slot) * block_bytes +
                                                    down_off) + 64 * s + lane;
            arow[u] = a_buf + (size_t)(tok_ok ? tok : 0) * F + (size_t)e * blk + 32 * s + 8 * (lane >> 4);
        }
        u32x4 w[kU][NT];
        f32x4 av[kU][2];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < NT; ++j) w[u][j] = live[u] ? ld_stream(src[u] + j * piece_v) : u32x4{0u, 0u, 0u, 0u};
            av[u][0] = live[u] && tok_ok ? reinterpret_cast<const f32x4*>(arow[u])[0] : z;
            av[u][1] = live[u] && tok_ok ? reinterpret_cast<const f32x4*>(arow[u])[1] : z;
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const float xv[8] = {av[u][0].x, av[u][0].y, av[u][0].z, av[u][0].w,
                                 av[u][1].x, av[u][1].y, av[u][1].z, av[u][1].w};
            typename S::vec hi, lo;
            S::run(xv, hi, lo);
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const typename S::vec wv = S::from_raw(w[u][j]);
                c[j] = S::mfma(wv, hi, c[j]);
                c[j] = S::mfma(wv, lo, c[j]);
            }
        }
    }
    // lane l holds columns 4 (l / 16) + i of tile j for token l % 16
    __shared__ float part[NT == 1 ? kWavesDn : kWavesDn / NT][NT][16][16];
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) part[wave][j][4 * (lane >> 4) + i][lane & 15] = c[j][i];
    __syncthreads();
    for (int q = (int)threadIdx.x; q < NT * 16 * B; q += (int)blockDim.x) {
        const int j = q / (16 * B), t = (q / 16) % B, col = q % 16;
        float y = 0.f;
        for (int w = 0; w < n_waves; ++w) y += part[w][j][col][t];
        const size_t m = (size_t)t * d + (size_t)(tile * NT + j) * kColTile + col;
        if (splits == 1)
            x_acc[m] = (begin == 0 ? x_in[m] : x_acc[m]) + y;
        else
            part_out[(size_t)sp * B * d + m] = y;
    }
}

// x_acc[m] = (x_in or x_acc)[m] + the parts' sums for m in order of part
__global__ __launch_bounds__(256) void down_finish_kernel(const float* __restrict__ part, int splits,
                                                          int n, const float* __restrict__ x_in,
                                                          float* __restrict__ x_acc, int first) {
    const int m = (int)blockIdx.x * 256 + (int)threadIdx.x;
    if (m >= n) return;
    float y = 0.f;
    for (int p = 0; p < splits; ++p) y += part[(size_t)p * n + m];
    x_acc[m] = (first ? x_in[m] : x_acc[m]) + y;
}

}  // namespace

bool mfma_path(const Shape& s, int B) {
    return B >= kMfmaMinBatch && B <= 16 && s.dtype != LS_F32 && s.blk % 32 == 0 && s.d % 32 == 0;
}

hipError_t launch_gateup_mfma(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                              const float* x, int B, const int32_t* idx, const int32_t* count,
                              int begin, int end, float* a_buf, hipStream_t st) {
    const long groups = (long)(end - begin) * (s.blk / 16);
    if (groups <= 0) return hipSuccess;
    const size_t bb = s.block_elems * elem_size(s.dtype);
    const dim3 grid((unsigned)groups), blk(64 * kWaves);
    const bool relu = s.act == LS_ACT_REGLU;
#define LS_GUM(TT, AA)                                                                            \
    do {                                                                                          \
        if (s.prenorm)                                                                            \
            hipLaunchKernelGGL((gateup_mfma_kernel<TT, AA, true>), grid, blk, 0, st, L.blocks, bb, \
                               slot_table, L.bias, L.threshold, x, B, s.d, s.blk, s.n_blk, s.F,   \
                               idx, count, begin, end, a_buf);                                    \
        else                                                                                      \
            hipLaunchKernelGGL((gateup_mfma_kernel<TT, AA, false>), grid, blk, 0, st, L.blocks,   \
                               bb, slot_table, L.bias, L.threshold, x, B, s.d, s.blk, s.n_blk,    \
                               s.F, idx, count, begin, end, a_buf);                               \
    } while (0)
    if (s.dtype == LS_F16) {
        if (relu) LS_GUM(LS_F16, LS_ACT_REGLU);
        else LS_GUM(LS_F16, LS_ACT_SWIGLU_THRESH);
    } else if (s.dtype == LS_BF16) {
        if (relu) LS_GUM(LS_BF16, LS_ACT_REGLU);
        else LS_GUM(LS_BF16, LS_ACT_SWIGLU_THRESH);
    } else {
        return hipErrorInvalidValue;
    }
#undef LS_GUM
    return hipGetLastError();
}

DownLayout down_layout(const Shape& s, int B) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    // Chosen from launch times over list lengths on the three model shapes (B = 4 and 8):
    // 32 columns per workgroup wherever the activation reads are a large share of a
    // workgroup's bytes; tiles that do not fill whole rounds of the CUs (d = 5120) and 128-row
    // blocks (one block's piece of a tile is 4 KB) take 8 list parts of 4 waves; 64-row blocks
    // at d = 4096 take 2 parts of 8 waves at B = 8 and one 16-column tile per workgroup, no
    // parts, below.
    if ((s.d / kColTile) % cus != 0 || s.blk >= 128) return DownLayout{2, 8, 4};
    if (B >= 8 && (s.d / (2 * kColTile)) * 2 % cus == 0) return DownLayout{2, 2, 8};
    return DownLayout{1, 1, kWavesDn};
}

hipError_t launch_down_mfma(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                            const float* a_buf, int B, const int32_t* idx, const int32_t* count,
                            int begin, int end, const float* x_in, float* x_acc, float* part,
                            hipStream_t st) {
    const size_t bb = s.block_elems * elem_size(s.dtype);
    DownLayout lay = down_layout(s, B);
    if (!part) lay = DownLayout{1, 1, kWavesDn};
    const dim3 grid((unsigned)(s.d / (kColTile * lay.nt) * lay.splits)), blk(64 * lay.waves);
    // items in flight per wave: 4 with eight waves per workgroup, else 2 (measured at B = 4 and
    // 8 on the three shapes: 2 against 4 gave the 13B shape at B = 8 2357 -> 2367 tokens/s, the
    // Mistral-7B shape at B = 4 1208 -> 1230, the 7B shape at B = 4 2719 -> 2757, and lost 1.5%
    // on the 7B shape at B = 8, the eight-wave layout; 6 lost everywhere)
    const int ku = lay.waves == 8 ? 4 : 2;
#define LS_DNM(TT, NT, KU)                                                                                   \
    hipLaunchKernelGGL((down_mfma_kernel<TT, NT, KU>), grid, blk, 0, st, L.blocks, bb, slot_table, a_buf, B, \
                       s.F, s.d, s.blk, s.n_blk, idx, count, begin, end, x_in, x_acc, lay.splits, part)
#define LS_DNT(TT)                                     \
    do {                                               \
        if (lay.nt == 1) LS_DNM(TT, 1, 2);             \
        else if (ku == 4) LS_DNM(TT, 2, 4);            \
        else LS_DNM(TT, 2, 2);                         \
    } while (0)
    if (s.dtype == LS_F16)
        LS_DNT(LS_F16);
    else if (s.dtype == LS_BF16)
        LS_DNT(LS_BF16);
    else
        return hipErrorInvalidValue;
#undef LS_DNT
#undef LS_DNM
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || lay.splits == 1) return e;
    const int n = B * s.d;
    hipLaunchKernelGGL(down_finish_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, part, lay.splits, n,
                       x_in, x_acc, begin == 0 ? 1 : 0);
    return hipGetLastError();
}

}  // namespace ls
