// ls_decode.h - the fused decode-step kernel (one persistent launch per token).
#pragma once

#include "ls_internal.h"

namespace ls {

// Device view of one layer for the fused kernel.
struct LayerPtrs {
    const uint8_t* blocks;  // n_blk blocks of block_bytes
    const void* bias;       // [F] or null
    const float* pf;        // [n_blk, d] folded predictor P2 P1
    float threshold;
    float pad_;
};

struct FusedArgs {
    const LayerPtrs* layers;  // device [L]
    int L, d, nb, blk, F, k, kp, prenorm;
    size_t block_bytes;
    float* x;                 // [d]: input at entry, output at exit
    uint64_t* xmb;            // [L][d]      as 2 x [L][d] 32-bit words: the layer inputs of
                              //             launches with even / odd tag (row 0: the input,
                              //             unused when L >= 2: layer 0 then reads x itself)
    uint64_t* smb;            // [L][2 n_blk] tagged scores (exact | speculative)
    uint64_t* amb;            // [L][2F]     tagged activations: list positions, then misses
    uint32_t tag;             // launch epoch (>= 1)
    int* err;                 // set to 1 when a wait exceeded its spin limit
    uint64_t* trace;          // null, or [L][kTracePoints] wall-clock stamps of one workgroup
    int trace_wg;
};

constexpr int kTracePoints = 16;

// Shapes the fused kernel handles (others use the per-kernel path).
struct FusedSupport {
    bool ok;
    const char* why;
};
FusedSupport fused_supported(const Shape& s, int B, int k, int kp, int n_wg, int L);

// Largest speculative width (blocks prefetched for the next layer) the fused kernel holds.
int fused_max_spec(const Shape& s, int n_wg);

// Mailbox layout of the fused kernel: the layer inputs (L * d 64-bit words, used as two halves
// of [L][d] bare 32-bit words selected by the parity of the launch's tag, each word 0xffffffff
// until published; workgroup w writes its 16-column tile of a row, one 64-byte line), then per
// layer the scores (kScoreStride words per workgroup, a
// 64-byte line of its own: exact at +0, speculative at +1; when many workgroups write into
// one line the exchange takes about twice as long), then per layer 2F words of activations:
// the list's activations in list order as two halves of F bare 32-bit words (by the tag's
// parity, each word 0xffffffff until published, as for the inputs), then the misses' tagged
// words (k*blk <= F).
constexpr int kScoreStride = 8;
__host__ __device__ inline size_t fused_score_words_n(int n_blk) { return (size_t)n_blk * kScoreStride; }
inline size_t fused_score_words(const Shape& s) { return fused_score_words_n(s.n_blk); }
inline size_t fused_input_words(const Shape& s, int L) { return (size_t)L * s.d; }
inline size_t fused_acts_offset(const Shape& s, int L) { return (size_t)L * (s.d + fused_score_words(s)); }
inline size_t fused_mailbox_words(const Shape& s, int L, int /*n_wg*/) {
    return (size_t)L * ((size_t)s.d + fused_score_words(s) + 2 * (size_t)s.F);
}

// dst[i] = value bits of the tagged words src[i * stride], i < n
hipError_t launch_untag(const uint64_t* src, int n, int stride, float* dst, hipStream_t st);

// cooperative: hipLaunchCooperativeKernel (guaranteed co-residency), else a plain launch
hipError_t launch_decode_fused(const Shape& s, const FusedArgs& a, int n_wg, bool cooperative,
                               hipStream_t st);

}  // namespace ls
