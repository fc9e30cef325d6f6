// ls_hash.hip - stacked learnable hashing predictor at inference (Sec. 3.3.1, Eq. hash_layer,
// Eq. hashfunc_layer): an alternative block scorer to the low-rank predictor.
//
// Five hashing layers with 8 hash bits each and 256-wide binary features between them.  Layer
// 1 hashes the real input with 8 real hyperplanes (8 dot products over d); layers 2-5 hash the
// previous table row with binary hyperplanes, the signed products taken as XNOR + bitcount
// (x.w = 256 - 2 popcount(x XOR w)).  A code's bucket is the code read as an 8-bit number, first
// hash bit most significant, +1 -> 1 (the paper's sign-pattern order); sign(0) = +1.  The last
// layer's bucket selects a row of 8-bit block-priority levels, the block scores.
//
// One workgroup per token.  The binary layers' tables and hyperplanes (33 KB) are copied into
// LDS while the first layer runs, so the four dependent lookups after it do not go to memory.
// The dot products are the only floating-point work: each of the 256 threads sums j = t,
// t + 256, ... with fused multiply-adds in order, then a pairwise halving sum in LDS gives each
// hash bit (a fixed order, so the codes are reproducible).  The four binary layers run in one
// wave (lane b evaluates hash bit b; a ballot forms the bucket).
#include "ls_internal.h"

namespace ls {
namespace {

constexpr int kTau = 8;                // hash bits per layer
constexpr int kDh = 256;               // binary feature width
constexpr int kDhWords = kDh / 32;
constexpr int kHashLayers = 5;
constexpr int kThreads = 256;

// bucket of a code whose bit b (hash bit b, 1 = +1) sits in bit b of `mask`: bit b has weight
// 2^(7 - b)
__device__ __forceinline__ int bucket_of(uint64_t mask) {
    return (int)(__brev((uint32_t)(mask & 0xffu)) >> 24);
}

__global__ __launch_bounds__(kThreads) void hash_predict_kernel(int d, int nblk, const float* __restrict__ x,
                                                               const float* __restrict__ w1,
                                                               const uint32_t* __restrict__ w_bin,
                                                               const uint32_t* __restrict__ tables,
                                                               const uint8_t* __restrict__ head,
                                                               float* __restrict__ scores) {
    __shared__ float part[kTau][kThreads];
    __shared__ uint32_t tab[(kHashLayers - 1) * kDh * kDhWords];
    __shared__ uint32_t wb[(kHashLayers - 1) * kTau * kDhWords];
    __shared__ int last_bucket;
    const int t = threadIdx.x;
    {
        // 16-byte copies: tables 2048, hyperplanes 64
        const uint4* src = reinterpret_cast<const uint4*>(tables);
        uint4* dst = reinterpret_cast<uint4*>(tab);
        constexpr int n_tab = (kHashLayers - 1) * kDh * kDhWords / 4;
#pragma unroll
        for (int i = 0; i < n_tab / kThreads; ++i) dst[t + kThreads * i] = src[t + kThreads * i];
        constexpr int n_wb = (kHashLayers - 1) * kTau * kDhWords / 4;
        if (t < n_wb) reinterpret_cast<uint4*>(wb)[t] = reinterpret_cast<const uint4*>(w_bin)[t];
    }
    const float* xt = x + (size_t)blockIdx.x * d;
    float acc[kTau];
#pragma unroll
    for (int b = 0; b < kTau; ++b) acc[b] = 0.f;
    for (int j = t; j < d; j += kThreads) {
        const float xv = xt[j];
        const float4 lo = *reinterpret_cast<const float4*>(w1 + (size_t)j * kTau);
        const float4 hi = *reinterpret_cast<const float4*>(w1 + (size_t)j * kTau + 4);
        acc[0] = fmaf(xv, lo.x, acc[0]);
        acc[1] = fmaf(xv, lo.y, acc[1]);
        acc[2] = fmaf(xv, lo.z, acc[2]);
        acc[3] = fmaf(xv, lo.w, acc[3]);
        acc[4] = fmaf(xv, hi.x, acc[4]);
        acc[5] = fmaf(xv, hi.y, acc[5]);
        acc[6] = fmaf(xv, hi.z, acc[6]);
        acc[7] = fmaf(xv, hi.w, acc[7]);
    }
#pragma unroll
    for (int b = 0; b < kTau; ++b) part[b][t] = acc[b];
    __syncthreads();
    for (int s = kThreads / 2; s >= 1; s >>= 1) {
        if (t < s) {
#pragma unroll
            for (int b = 0; b < kTau; ++b) part[b][t] = part[b][t] + part[b][t + s];
        }
        __syncthreads();
    }
    if (t < 64) {
        int idx = bucket_of(__ballot(t < kTau && part[t & (kTau - 1)][0] >= 0.f));
        for (int k = 1; k < kHashLayers; ++k) {
            const uint32_t* y = tab + ((k - 1) * kDh + idx) * kDhWords;  // y_k = T_k[idx]
            int mismatch = 0;
            if (t < kTau) {
                const uint32_t* w = wb + ((k - 1) * kTau + t) * kDhWords;
#pragma unroll
                for (int m = 0; m < kDhWords; ++m) mismatch += __popc(y[m] ^ w[m]);
            }
            idx = bucket_of(__ballot(t < kTau && kDh - 2 * mismatch >= 0));
        }
        if (t == 0) last_bucket = idx;
    }
    __syncthreads();
    const uint8_t* row = head + (size_t)last_bucket * nblk;
    for (int b = t; b < nblk; b += kThreads) scores[(size_t)blockIdx.x * nblk + b] = (float)row[b];
}

}  // namespace

hipError_t launch_hash_predict(int d, int nblk, const float* x, int B, const HashDev& h, float* scores,
                               hipStream_t st) {
    if (B <= 0) return hipSuccess;
    hipLaunchKernelGGL(hash_predict_kernel, dim3(B), dim3(kThreads), 0, st, d, nblk, x, h.w1, h.w_bin,
                       h.tables, h.head, scores);
    return hipGetLastError();
}

}  // namespace ls
