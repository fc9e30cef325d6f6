// ls_internal.h - shared declarations of the gfx950 sparse-FFN library.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/ls_ffn.h"

namespace ls {

// Down-projection column tile: a block's down weights are stored as
// [d/kColTile][block/V][kColTile][V] with V = 16 bytes / element size, so one
// 16-byte lane load holds V neurons of one output column and a wave's load
// instruction covers a contiguous kilobyte.
constexpr int kColTile = 16;
constexpr int kMaxBatch = 8;
constexpr int kMaxBlocks = 2048;  // n_blk limit of the selection kernel

inline int elem_size(ls_dtype t) { return t == LS_F32 ? 4 : 2; }
inline int vec_elems(ls_dtype t) { return 16 / elem_size(t); }

// Device views of one layer.
struct LayerDev {
    const uint8_t* blocks = nullptr;  // n_blk blocks of block_bytes (resident mode)
    const void* bias = nullptr;       // [F] or null
    const void* p1 = nullptr;         // [r, d] in the grouped row order (factored predictor)
    const void* p2 = nullptr;         // [n_blk, r] in the grouped row order (factored predictor)
    const float* pf = nullptr;        // [n_blk, d] fp32 product P2 P1 (folded predictor)
    float threshold = 0.f;
};

struct Shape {
    int d, F, blk, r, n_blk;
    ls_dtype dtype;
    ls_act act;
    int prenorm;
    size_t block_elems;  // 3 * blk * d
    // Predictor rows are stored grouped by workgroup: logical row i of P1 (P2) sits at
    // storage row (i % G) * p1_rpw + i / G  ((i % G) * p2_rpw + i / G).
    int G, p1_rpw, p2_rpw;
    // 1: the predictor is kept as the fp32 product P2 P1 (one n_blk x d GEMV), chosen
    // when that matrix is no larger than the two factors in the weight type.
    int fold;
    // 1: batches of kMfmaMinBatch or more tokens use the matrix-core gate/up and down
    // kernels when the shape allows (16-bit weights, block a multiple of 32).
    int batch_mfma = 1;
    // 1: row-level zero skip in the vector-ALU gate/up and down kernels (up rows only for
    // neurons with a nonzero gate output; down vectors only for groups with a nonzero
    // activation); the batch then always runs on those kernels.
    int zero_skip = 0;
};

constexpr int kMfmaMinBatch = 4;

// Fold decision: the product costs 4 n_blk d bytes, the factors (r d + n_blk r) elem bytes.
inline int predictor_folds(int d, int r, int n_blk, ls_dtype t) {
    return 4.0 * n_blk * d <= (double)elem_size(t) * ((double)r * d + (double)n_blk * r) ? 1 : 0;
}

// ---- kernel launchers (ls_kernels.hip) -------------------------------------------------
// The MLP input h = x / sqrt(mean(x^2) + 1e-6) is never materialised: a kernel that reads x
// for a dot product also sums x^2 and scales the dot product (h.w = scale * (x.w)).
//
// out[b, i] = c_b * W[s(i), :] . v[b, :] with s(i) = (i % G) * rpw + i / G (the grouped row
// order); c_b = the RMS scale of v[b, :] when rms, else 1.
hipError_t launch_gemv_rows(ls_dtype t, const void* W, int rows, int cols, int G, int rpw,
                            const float* v, int B, bool rms, float* out, hipStream_t st);
// out[i, j] = sum_m P2[i, m] P1[m, j] (fp64 accumulation in m order, rounded once to
// fp32); P1 [r, d], P2 [n_blk, r] row-major in the weight type.
hipError_t launch_fold_predictor(ls_dtype t, const void* P1, const void* P2, int r, int d, int n_blk,
                                 float* out, hipStream_t st);
// Stacked hashing predictor of one layer (ls_hash.hip): device copies of its weights.
struct HashDev {
    float* w1 = nullptr;          // [d][8]
    uint32_t* w_bin = nullptr;    // [4][8][8]
    uint32_t* tables = nullptr;   // [4][256][8]
    uint8_t* head = nullptr;      // [256][n_blk]
};
// scores[b, :] = the hashing predictor's block scores of token b of x [B, d]
hipError_t launch_hash_predict(int d, int nblk, const float* x, int B, const HashDev& h, float* scores,
                               hipStream_t st);
hipError_t launch_select(const float* scores, int B, int n_blk, int mode, int k, float tau,
                         int union_batch, int cap, int32_t* idx, int32_t* count, hipStream_t st);
// slot_table: null in resident mode (block b lives at blocks + b*block_bytes); else
// device int32 [n_blk] giving the cache slot of block b, relative to `blocks`.
// x: the layer input [B, d]; the RMS scale is applied when s.prenorm
hipError_t launch_gateup(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                         const float* x, int B, const int32_t* idx, const int32_t* count,
                         int begin, int end, float* a_buf, hipStream_t st);
// Batch 1, resident weights: the top-k selection of `scores` (as launch_select with
// LS_SEL_TOPK, k, no union) and the gate/up gather of its list in one launch; writes idx[0..n)
// and count[0] = n for launch_down.  gateup_select_ok: whether the shape allows it.
bool gateup_select_ok(const Shape& s, int B, int k);
hipError_t launch_gateup_select(const Shape& s, const LayerDev& L, const float* x, const float* scores, int k,
                                int32_t* idx, int32_t* count, float* a_buf, hipStream_t st);
// part: [kDownPartsMax, B, d] floats of scratch for the matrix-core path's split list (may be
// null: no split)
hipError_t launch_down(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                       const float* a_buf, int B, const int32_t* idx, const int32_t* count,
                       int begin, int end, const float* x_in, float* x_acc, float* part,
                       hipStream_t st);

// Streaming read of `bytes` (a multiple of 16) at buf by `grid` workgroups of 256 threads;
// out: 4 * grid words of scratch.
hipError_t launch_read_probe(const void* buf, size_t bytes, uint32_t* out, int grid, hipStream_t st);

// ---- persistent consumer of a streamed layer's copy stages (ls_stage.hip) ----------------
constexpr int kMaxStages = 64;
struct StageArgs {
    const uint8_t* blocks;       // HBM cache arena
    size_t block_bytes;
    const int32_t* slot_table;   // device [n_blk]: cache slot of each block of the layer
    const void* bias;
    float thresh;
    const float* x_in;           // [d] layer input
    float* x_acc;                // [d] x_in + the partial outputs of the stages so far
    float* a_buf;                // [F] activations in list order
    const int32_t* idx;          // device priority list, n entries
    int n, K;                    // list length, stages (stage s: entries [s n / K, (s+1) n / K))
    int d, blk, n_blk, F;
    const uint32_t* arrive;      // [K] arrival words (fine-grained device memory), or null
    uint8_t wait_on[kMaxStages]; // stage s waits for arrive[wait_on[s]] (wait_on[s] <= s)
    uint32_t* done;              // [K] host-visible done words, or null
    uint32_t* cnt;               // device [2][kMaxStages]: per-stage done counts, then gate/up counts; zero between calls
    uint32_t* status;            // host-visible: 0, or 2 / 4 when an arrival / barrier wait ran out
    uint32_t tag;                // this call's arrival / done value
    uint64_t limit;              // wall-clock ticks (100 MHz) any one wait may take
};
// One launch of `grid` workgroups (one per compute unit; cooperative when asked) consuming
// the stages in order (B = 1).
hipError_t launch_stage_consumer(const Shape& s, const StageArgs& p, int grid, bool cooperative, hipStream_t st);

// ---- matrix-core variants for B >= kMfmaMinBatch (ls_mfma.hip) ---------------------------
bool mfma_path(const Shape& s, int B);
hipError_t launch_gateup_mfma(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                              const float* x, int B, const int32_t* idx, const int32_t* count,
                              int begin, int end, float* a_buf, hipStream_t st);
constexpr int kDownPartsMax = 8;  // list parts of the matrix-core down projection, at most
// Layout of the matrix-core down projection: nt adjacent 16-column tiles per workgroup, the
// list cut into `splits` parts (partial sums in the part buffer, added by a finish kernel),
// `waves` waves per workgroup.
struct DownLayout {
    int nt, splits, waves;
};
DownLayout down_layout(const Shape& s, int B);
hipError_t launch_down_mfma(const Shape& s, const LayerDev& L, const int32_t* slot_table,
                            const float* a_buf, int B, const int32_t* idx, const int32_t* count,
                            int begin, int end, const float* x_in, float* x_acc, float* part,
                            hipStream_t st);

}  // namespace ls
