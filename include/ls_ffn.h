/*
 * ls_ffn.h - C ABI of the MI355X (gfx950) sparse-FFN decode library.
 *
 * One decode step of the activation-sparse gated FFN of LeanStream's
 * speculate-and-refine decode (arxiv 2609.03079): a low-rank predictor scores
 * neuron blocks, the blocks are selected in descending predicted priority,
 * and only the selected blocks' gate/up/down weights are read and computed.
 *
 * Conventions (every entry point):
 *  - Every call returns ls_status; nothing aborts, throws or exits.
 *  - Pointers marked "dev" are device pointers (HBM) owned by the caller;
 *    pointers marked "host" are host pointers.  Weight storage is owned by the
 *    context.
 *  - Activations (x, h, scores, y) are fp32; weights are in the context dtype;
 *    accumulation is fp32.  Row-major ("C") layouts throughout.
 *  - Compute calls enqueue on the context's stream and return; argument
 *    validation is synchronous.  A HIP failure makes the context sticky in
 *    LS_E_DEVICE until ls_ffn_destroy.
 *  - One host thread per context.  ls_last_error() describes the last failure.
 *  - Every call that the library accepts for a given context, shape and
 *    selection computes the same bits on every run (fixed reduction orders,
 *    no floating-point atomics).
 */
#ifndef LS_FFN_H
#define LS_FFN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ls_ffn ls_ffn; /* opaque context; owns all weight storage */

typedef enum {
    LS_OK = 0,
    LS_E_INVAL = 1,       /* bad argument (null pointer, shape, range, cap too small) */
    LS_E_NOMEM = 2,       /* host or device allocation failed */
    LS_E_DEVICE = 3,      /* a HIP call failed; sticky until ls_ffn_destroy */
    LS_E_STATE = 4,       /* call not valid in the context's state (e.g. layer not set) */
    LS_E_UNSUPPORTED = 5, /* valid request the library does not implement */
    LS_E_CAPACITY = 6     /* request larger than the HBM block cache */
} ls_status;

typedef enum { LS_F32 = 0, LS_F16 = 1, LS_BF16 = 2 } ls_dtype;

/* Gating of the gate branch (Eq. 1, Sec. 2.1):
 *  REGLU:          a_j = max(g_j, 0) * u_j
 *  SWIGLU_THRESH:  s_j = g_j / (1 + exp(-g_j));  a_j = s_j * u_j if |s_j| > t_l else 0 */
typedef enum { LS_ACT_REGLU = 0, LS_ACT_SWIGLU_THRESH = 1 } ls_act;

/* Where the FFN blocks live: resident in HBM, or in pinned host memory with a
 * bounded HBM block cache filled by ls_stream_weights. */
typedef enum { LS_WEIGHTS_HBM = 0, LS_WEIGHTS_HOST = 1 } ls_residency;

/* Block selection: top-k by score, or every score strictly above tau. */
typedef enum { LS_SEL_TOPK = 0, LS_SEL_THRESHOLD = 1 } ls_sel_mode;

typedef struct {
    int32_t n_layers;
    int32_t d_model;      /* d; multiple of 64 */
    int32_t d_ff;         /* F; multiple of block */
    int32_t block;        /* neurons per block; multiple of 8 */
    int32_t rank;         /* predictor rank r; multiple of 64 */
    int32_t max_batch;    /* 1..8 tokens per call */
    ls_dtype dtype;       /* weight storage type */
    ls_act act;
    ls_residency residency;
    int32_t prenorm_rms;  /* 0: h = x;  1: h = x / sqrt(mean(x^2) + 1e-6) */
    uint64_t hbm_cache_bytes; /* LS_WEIGHTS_HOST only: HBM block-cache budget */
    void* stream;         /* hipStream_t borrowed for all compute (NULL: the null stream);
                             must outlive the context */
    uint32_t debug_flags; /* reserved, 0 */
} ls_ffn_desc;

/* One layer's weights, host pointers in the context dtype, nn.Linear layouts.
 * Copied by ls_ffn_set_layer; the caller may free them afterwards. */
typedef struct {
    const void* w_gate; /* [F, d] */
    const void* w_up;   /* [F, d] */
    const void* w_down; /* [d, F] (nn.Linear down_proj.weight) */
    const void* b_gate; /* [F] or NULL (gate-branch bias) */
    const void* p1;     /* [r, d]      predictor input projection (Sec. 3.3.3) */
    const void* p2;     /* [n_blk, r]  predictor head scoring neuron blocks */
    float threshold;    /* t_l of LS_ACT_SWIGLU_THRESH; ignored for ReGLU */
} ls_layer_weights;

typedef struct {
    int64_t hits;       /* requested blocks already in the HBM cache */
    int64_t misses;     /* requested blocks copied host -> HBM */
    int64_t bytes;      /* bytes copied host -> HBM by this call */
    int64_t evictions;  /* cache slots reassigned by this call */
} ls_stream_stats;

/* Create a context on the current HIP device.  Allocates the weight arena
 * (HBM, or pinned host + HBM cache) and the workspaces.
 * The context is the holder of the model's FFN weights in the problem setting
 * of Sec. 1: weights kept in a large tier (here HBM, or pinned host memory
 * standing in for the paper's storage) of which each decode step reads only the
 * predicted sub-matrices.  desc is read during the call only.  On success *out
 * receives a context the caller owns and releases with ls_ffn_destroy; on
 * failure *out is set to NULL and ls_last_error(NULL) describes it.
 * LS_E_INVAL on a bad descriptor; LS_E_NOMEM if an allocation fails (for
 * instance an hbm_cache_bytes the device cannot hold). */
ls_status ls_ffn_create(const ls_ffn_desc* desc, ls_ffn** out);

/* Copy one layer's weights (host, nn.Linear layouts) into the context's own
 * layout: per block of `block` neurons one contiguous chunk
 * [gate rows | up rows | down columns], which serves coalesced 128-bit loads
 * and one copy per block (Sec. 3.2.2: blocks appended in arrival order form a
 * contiguous buffer).  Synchronous.  LS_E_INVAL on null pointers or layer out
 * of range. */
ls_status ls_ffn_set_layer(ls_ffn* ctx, int32_t layer, const ls_layer_weights* w);

/* Release everything the context owns (the counterpart of ls_ffn_create,
 * Sec. 1 problem setting).  Synchronises the stream and the copy stream first.
 * LS_E_INVAL for a NULL ctx.  ctx is invalid afterwards. */
ls_status ls_ffn_destroy(ls_ffn* ctx);

/* Predictor (Sec. 3.3.3): h = prenorm(x); scores = P2 (P1 h).
 * x: dev fp32 [B, d]; scores: dev fp32 [B, n_blk].  1 <= B <= max_batch.
 * When the product is no larger than the factors (4 n_blk d bytes against
 * (r d + n_blk r) weight-type bytes) the context keeps Pf = P2 P1, formed once
 * by ls_ffn_set_layer with fp64 accumulation and rounded to fp32, and applies
 * it as one GEMV; otherwise it applies P1, then P2.  Either way the scores are
 * the same function of x up to fp32 rounding. */
ls_status ls_predict(ls_ffn* ctx, int32_t layer, const float* x, int32_t B, float* scores);

/* Block selection over dev fp32 scores [B, n_blk] (priority list, Sec. 2.1).
 * Total order: a before b iff key(a) > key(b), or keys equal and a < b, where
 * key puts NaN below every number, treats -0 == +0, and is IEEE order
 * otherwise.  TOPK: the first k entries.  THRESHOLD: every non-NaN score > tau,
 * in the same order.  union_batch != 0 and B > 1: the union of the tokens'
 * selections, ordered by the largest key over all B tokens, then by index.
 * Output, dev int32: per token idx [B, cap], count [B]; union idx [cap], count [1].
 * cap must be >= k (TOPK), >= min(n_blk, B*k) (TOPK union) or >= n_blk
 * (THRESHOLD); 1 <= k <= n_blk for TOPK.  LS_E_INVAL otherwise. */
ls_status ls_select_blocks(ls_ffn* ctx, const float* scores, int32_t B, ls_sel_mode mode,
                           int32_t k, float tau, int32_t union_batch, int32_t cap, int32_t* idx,
                           int32_t* count);

/* Sparse FFN over entries [begin, min(end, *count)) of the priority list idx
 * (dev int32, one list shared by all B tokens) for layer `layer`:
 *   h = prenorm(x_in);  for every neuron j of those blocks:
 *   g_j = Wg[j,:] h + b_j, u_j = Wu[j,:] h, a_j = gate(g_j, u_j)   (Eq. 1)
 *   y = sum_j a_j Wd[:, j]                                          (Sec. 3.2.2)
 *   begin == 0: x_acc = x_in + y;   begin > 0: x_acc += y            (Eq. 2)
 * so after the stages [0,e1), [e1,e2), ... x_acc holds the refined feature
 * x_tilde of Eq. 2.  x_in, x_acc: dev fp32 [B, d], must not alias.
 * count: dev int32 [1].  0 <= begin <= end.  An entry that is not a valid
 * block id (or, with host-resident weights, not in the block cache)
 * contributes nothing. */
ls_status ls_sparse_ffn_step(ls_ffn* ctx, int32_t layer, const float* x_in, int32_t B,
                             const int32_t* idx, const int32_t* count, int32_t begin, int32_t end,
                             float* x_acc);

/* For callers that cannot allocate memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): ls_sparse_ffn_step with the
 * same arguments, kernels and results, whose scratch (the activations
 * [B, d_ff] and the split down projection's parts [8, B, d_model], fp32) lives
 * in a fixed device array of LS_STATIC_SCRATCH_BYTES that the library defines
 * instead of in the context's workspace.  Each GPU holds its own copy of that
 * array from the first ls_ffn_create on it until the process ends.  The call
 * allocates nothing and never brackets its launches with timing events.
 * Nothing in the array needs to start at zero (every element read is written
 * earlier in the same call), but every call on one GPU shares the array and it
 * keeps the last call's contents: calls that overlap on one GPU (other streams,
 * other contexts, other host threads) race, so the caller must order them.
 * LS_E_CAPACITY if B * (d_ff + 8 d_model) floats exceed the array; otherwise
 * the errors of ls_sparse_ffn_step.  ls_debug_last_activations then reads the
 * activations from the array. */
#define LS_STATIC_SCRATCH_BYTES (4u << 20)
ls_status ls_sparse_ffn_step_static(ls_ffn* ctx, int32_t layer, const float* x_in, int32_t B,
                                    const int32_t* idx, const int32_t* count, int32_t begin,
                                    int32_t end, float* x_acc);

/* The I/O side of Sec. 3.2.1 (Alg. 1: weight blocks loaded in priority order
 * while the GPU computes the blocks already present) with the block layout of
 * Sec. 3.2.2 (one contiguous chunk per block, so one copy per block).
 * LS_WEIGHTS_HOST: make blocks idx_host[0..n) of `layer` (host int32 list, in
 * priority order, read during the call only) resident in the HBM cache, copying
 * misses from pinned host memory in priority order on a copy stream, in
 * n_stages equal contiguous stages; the following ls_sparse_ffn_step calls of
 * this layer wait for the stages they read.  No block of this request is
 * evicted to make room for another of it.  Blocks of other layers that it
 * evicts drop out of those layers' slot tables: their later steps treat them
 * as not resident.  LS_WEIGHTS_HBM: no copy, all hits.  LS_E_INVAL on a block
 * id out of range, n < 0 or n_stages < 1; LS_E_CAPACITY if n exceeds the cache
 * slots.  stats may be NULL. */
ls_status ls_stream_weights(ls_ffn* ctx, int32_t layer, const int32_t* idx_host, int32_t n,
                            int32_t n_stages, ls_stream_stats* stats);

/* Stacked learnable hashing predictor of one layer (Sec. 3.3.1, Eq. hash_layer,
 * Eq. hashfunc_layer): five hashing layers of 8 hash bits with 256-wide binary
 * features, an alternative block scorer to ls_predict.  Binary {-1,+1}
 * vectors are bit-packed: element e is bit (e & 31) of word e >> 5, 1 = +1. */
typedef struct {
    const float* w1;        /* [d][8] real hyperplanes of the first layer */
    const uint32_t* w_bin;  /* [4][8][8] binary hyperplanes of layers 2..5 (hash bit b: 256 signs) */
    const uint32_t* tables; /* [4][256][8] feature tables T_1..T_4 (bucket i: 256 signs) */
    const uint8_t* head;    /* [256][n_blk] block-priority levels of the last layer's bucket */
} ls_hash_weights;

/* Copy one layer's hashing predictor (host pointers) into the context.
 * Synchronous.  LS_E_INVAL on null pointers or layer out of range. */
ls_status ls_set_hash_predictor(ls_ffn* ctx, int32_t layer, const ls_hash_weights* w);

/* Block scores of the hashing predictor for B tokens:
 *   layer 1:    c = sign(x W_1)              (8 products over d, binary32)
 *   layers 2-5: c = sign(y W_k), y = T_{k-1}[i], products as XNOR + bitcount
 *   i = the code read as an 8-bit number, first hash bit most significant,
 *       +1 -> 1; sign(0) = +1
 *   scores[b] = head[i_5][b].
 * The input is used as given (the codes are invariant to a positive scale, so
 * no prenorm).  The first layer's products are summed in a fixed order (per
 * hash bit: 256 partial sums of x_j W_1[j] over j = t, t + 256, ... with fused
 * multiply-adds in increasing j, then pairwise halving), so the codes are
 * reproducible.  x: dev fp32 [B, d]; scores: dev fp32 [B, n_blk] (integral
 * values 0..255; rank them with ls_select_blocks).  1 <= B <= max_batch.
 * LS_E_STATE if the layer has no hashing predictor. */
ls_status ls_hash_predict(ls_ffn* ctx, int32_t layer, const float* x, int32_t B, float* scores);

/* Cross-layer prefetch policy of ls_decode_step_streamed. */
typedef enum {
    LS_PREFETCH_NONE = 0,    /* a layer's blocks are requested once its own list is known */
    LS_PREFETCH_ONESHOT = 1, /* while layer n runs, layer n+1 is scored once on x_n (the
                                input of layer n) and its list is prefetched */
    LS_PREFETCH_REFINE = 2   /* after every stage j of layer n, layer n+1 is re-scored on the
                                refined feature x~_n^(j) (Sec. 2.1, Eq. 2) and the blocks of
                                its new list that are not yet resident are prefetched */
} ls_prefetch_mode;

typedef struct {
    int64_t final_bytes;   /* block bytes of every layer's final list (k blocks per layer) */
    int64_t copied_bytes;  /* all bytes copied host -> HBM by the step */
    int64_t late_bytes;    /* copied after the layer's own list was known: its compute waits */
    int64_t spec_bytes;    /* copied ahead of time for the next layer */
    int64_t wasted_bytes;  /* of spec_bytes: blocks the next layer's final list did not hold */
} ls_stream_report;

/* One decode step (B = 1) over every layer with host-resident weights, staged
 * (Sec. 2.1, Eq. 1-2).  Layer n's final list is topk(predict(n, x_n), k), from
 * its complete input exactly as in ls_decode_step; its blocks are requested
 * (misses copied in priority order in n_stages stages) and the layer runs as
 * n_stages sparse steps over equal parts of the list, each waiting only for its
 * own copies.  mode adds prefetch of layer n+1 during layer n (k_spec blocks per
 * prediction), with layer n's blocks protected from eviction meanwhile.  The
 * result depends only on the final lists, so every mode gives the same x
 * bitwise; the modes differ in when and how many bytes cross the host link.
 * How a stage's compute learns that its copies landed is LS_CFG_STREAM_SYNC:
 * events and one gate/up + down launch pair per stage (default); device flags
 * (Sec. 3.2.1, Alg. 1): the copy stream writes an arrival word after each
 * stage and ONE persistent launch per layer consumes the stages as they land,
 * the last workgroup to finish a stage writing a host-visible done word (then
 * at most 64 stages, and LS_PREFETCH_REFINE, which re-scores between stage
 * launches, is LS_E_UNSUPPORTED); or a host synchronisation after every stage
 * launch (the device-wide synchronisation the paper compares against).  All
 * three give the same x bitwise.
 * x: dev fp32 [d], updated in place.  report may be NULL.
 * LS_E_UNSUPPORTED with HBM-resident weights; LS_E_INVAL on bad arguments;
 * LS_E_CAPACITY if the cache cannot hold a layer's list (plus, while
 * prefetching, the next layer's) with the running layer's blocks protected;
 * LS_E_DEVICE if a wait of the stage-consuming kernel ran out
 * (LS_CFG_STAGE_WAIT_US; reported by the next flagged layer or by
 * ls_ffn_sync; the context then stays failed). */
ls_status ls_decode_step_streamed(ls_ffn* ctx, float* x, int32_t k, int32_t n_stages, int32_t mode,
                                  int32_t k_spec, ls_stream_report* report);

/* Debug: after a streamed step with device flags, the number of stages of
 * `layer`'s latest request whose done word carries that request's tag (all of
 * them once the layer's kernel has finished).  Synchronises the stream.
 * LS_E_STATE if no flagged step has run the layer. */
ls_status ls_debug_stages_done(ls_ffn* ctx, int32_t layer, int32_t* n_done);

/* One decode step over every layer (Sec. 2.1, Eq. 1 for every layer, the
 * priority list predicted from each layer's complete input): for l in 0..L-1:
 *   scores = predict(l, x); idx = topk(scores, k) (union over the B tokens if B > 1);
 *   x = x + sparse_ffn(l, x, idx[0..count)).
 * x: dev fp32 [B, d], updated in place.  1 <= k <= n_blk, 1 <= B <= max_batch
 * (LS_E_INVAL otherwise); LS_E_STATE if a layer was never set; with host-
 * resident weights LS_E_UNSUPPORTED (use ls_decode_step_streamed).  Equal to
 * composing the calls above.  The fused path's device-side failures (a bounded
 * wait that ran out) are reported by the next ls_ffn_sync. */
ls_status ls_decode_step(ls_ffn* ctx, float* x, int32_t B, int32_t k);

/* Debug: copy the activations a [B, n_sel * block] (fp32, priority-list order)
 * of the most recent ls_sparse_ffn_step into dst (dev), n_sel = that step's
 * end.  Positions at or past the list's device count (*count) are not written
 * by the step: they hold whatever the activation buffer held before.
 * LS_E_INVAL if cap is smaller than what the last step produced; *n_out
 * receives n_sel * block. */
ls_status ls_debug_last_activations(ls_ffn* ctx, float* dst, int64_t cap, int64_t* n_out);

/* Per-kernel timing (tracing aid).  While enabled, every kernel launch the
 * context makes is bracketed by a pair of HIP events recorded on the context's
 * stream.  enable: 0 off; 1 or -1 every kernel; otherwise a mask with bit
 * (1 << id) set for each kernel id to bracket, the others run unbracketed.  ls_kernel_timing synchronises the stream, folds the finished event
 * pairs into per-kernel totals and returns the total milliseconds and launch
 * count of one kernel id since the last reset; reset != 0 clears all totals.
 * Kernel ids: 0 MLP input (the RMS prenorm is computed inside the predictor and
 * gate/up kernels, so nothing is launched under this id), 1 predictor projection
 * (or the folded predictor),
 * 2 predictor head (not launched when the predictor is folded),
 * 3 selection, 4 gate/up gather, 5 down projection, 6 fused decode step,
 * 7 stacked hashing predictor, 8 stage-consuming kernel of the streamed step. */
enum { LS_K_PRENORM = 0, LS_K_PRED_P1, LS_K_PRED_P2, LS_K_SELECT, LS_K_GATEUP, LS_K_DOWN,
       LS_K_DECODE, LS_K_HASH, LS_K_STAGE, LS_K_COUNT };
ls_status ls_set_kernel_timing(ls_ffn* ctx, int32_t enable);
ls_status ls_kernel_timing(ls_ffn* ctx, int32_t kernel, int32_t reset, double* total_ms,
                           int64_t* launches);

/* Tuning knobs of ls_decode_step.
 *  LS_CFG_DECODE_PATH: 0 auto (fused kernel when the shape allows it, else the
 *    per-kernel sequence), 1 per-kernel sequence, 2 fused kernel only
 *    (ls_decode_step then returns LS_E_UNSUPPORTED for shapes it cannot run).
 *  LS_CFG_SPEC_BLOCKS: blocks of the next layer the fused kernel prefetches
 *    speculatively (its top-kp by scores predicted from the current layer's
 *    input, Eq. 2); 0 = automatic (k + ceil(k/4), or fewer when the kernel's
 *    neuron slots or down positions hold fewer).  Never changes results.
 *  LS_CFG_COOPERATIVE: 1 (default) launch the fused kernel with
 *    hipLaunchCooperativeKernel, which guarantees that its one-workgroup-per-
 *    compute-unit grid is resident at once; 0 a plain launch of the same grid
 *    (residency then depends on the device being otherwise idle; every wait in
 *    the kernel is bounded, so a workgroup that never starts makes the step fail
 *    with LS_E_DEVICE at ls_ffn_sync instead of hanging).
 *  LS_CFG_BATCH_MFMA: 1 (default) batches of 4 or more tokens run the
 *    gate/up and down kernels on the matrix cores when the weights are 16-bit
 *    and the block is a multiple of 32 (activations split into 16-bit hi and lo
 *    parts, fp32 accumulation); 0 always uses the vector-ALU kernels.
 *  LS_CFG_TRACE_WG: -1 (default) off; otherwise the fused kernel records
 *    per-layer phase timestamps of that workgroup (see ls_debug_phase_trace).
 *  LS_CFG_ZERO_SKIP: 0 (default) off; 1 row-level zero skip within the
 *    selected blocks (the zero outputs of ReLU-family and thresholded-SiLU
 *    gates that Sec. 2.1 builds on: a neuron whose gate output is zero adds
 *    nothing to Eq. 1): the gate row is read first, the up row only when the gate output is nonzero for
 *    some token of the batch, and a 16-byte down vector (V = 16 / element-size
 *    neurons of one output column) only when one of its neurons has a nonzero
 *    activation.  Results are equal to those with the knob off.  It applies to
 *    the per-kernel sequence (ls_sparse_ffn_step, the streamed step, and
 *    ls_decode_step on the per-kernel path), which then runs the vector-ALU
 *    kernels at every batch size; the fused kernel reads rows before their
 *    gate outputs are known and ignores it.
 *  LS_CFG_STREAM_SYNC: how ls_decode_step_streamed orders a stage's compute
 *    after its copies: 0 (default) events, one launch pair per stage; 1 device
 *    flags and one persistent launch per layer (allocates the flag words at
 *    the first use); 2 a host synchronisation after every stage.  The
 *    persistent launch is cooperative when LS_CFG_COOPERATIVE is 1.
 *  LS_CFG_STAGE_WAIT_US: how long any one wait of the stage-consuming kernel
 *    may take, in microseconds (default 2000000, range 1 .. 60000000); a wait
 *    that runs out ends the kernel and the call fails with LS_E_DEVICE.
 * LS_E_INVAL on an unknown key or value. */
enum { LS_CFG_DECODE_PATH = 0, LS_CFG_SPEC_BLOCKS = 1, LS_CFG_TRACE_WG = 2, LS_CFG_COOPERATIVE = 3,
       LS_CFG_BATCH_MFMA = 4, LS_CFG_ZERO_SKIP = 5, LS_CFG_STREAM_SYNC = 6, LS_CFG_STAGE_WAIT_US = 7 };
ls_status ls_configure(ls_ffn* ctx, int32_t key, int64_t value);

/* Debug: after a fused ls_decode_step (B = 1), copy what it exchanged for
 * `layer`: the layer input x_l (dev fp32 [d]; layer 0 is not kept, pass NULL)
 * and the layer's predicted block scores (dev fp32 [n_blk]).  Either pointer
 * may be NULL.  Valid until the next ls_decode_step.  LS_E_STATE if the last
 * ls_decode_step did not run the fused kernel. */
ls_status ls_debug_decode_trace(ls_ffn* ctx, int32_t layer, float* x_in, float* scores);

/* Debug: phase timestamps of the traced workgroup from the last fused
 * ls_decode_step, host int64 [n_layers][16] in wall-clock ticks (100 MHz):
 * control wave: 0 layer start, 1 input gathered, 2 scores published,
 * 3 all scores gathered, 4 list activations gathered, 5 exact top-k ready,
 * 6 slot map, 7 misses done, 8 all down partials ready, 9 output published;
 * last worker wave (it also ranks the next layer's list): 14 past the input
 * barrier, 13 speculative gate/up done, 12 next layer's list ranked, 15 list
 * activations seen, 11 down partials done, 10 next layer's loads issued.
 * Synchronises the stream.
 * *n receives n_layers * 16. */
ls_status ls_debug_phase_trace(ls_ffn* ctx, int64_t* host_out, int64_t cap, int64_t* n);

/* Wait for all work enqueued on the context's stream and report a device-side
 * failure of the fused kernel (a bounded wait that timed out) as LS_E_DEVICE. */
ls_status ls_ffn_sync(ls_ffn* ctx);

/* Text of the last failure on ctx (or of the last failed ls_ffn_create when
 * ctx is NULL); valid until the next call on ctx.  The status-code contract
 * of the boundary (Sec. 1 problem setting: the library is called from a
 * serving loop that must not abort). */
const char* ls_last_error(const ls_ffn* ctx);

/* Measurement: the HBM streaming-read ceiling of the device.  Reads buf
 * (dev, `bytes` bytes, a multiple of 16, at least 1 MiB) reps times with a
 * kernel of 16-byte nontemporal loads over 8 workgroups per compute unit, each
 * workgroup a contiguous range, on the context's stream, and returns the
 * fastest and the median read rate in GB/s (1e9 bytes per second) from HIP
 * events around each launch.  Synchronises the stream.  Allocates a small
 * device result buffer per call.  LS_E_INVAL on bad arguments. */
ls_status ls_measure_read_bandwidth(ls_ffn* ctx, const void* buf, int64_t bytes, int32_t reps,
                                    double* best_gbs, double* median_gbs);

/* Digest (hex sha256) of the library sources this binary was built from, or
 * "unknown".  The Python binding refuses a library whose digest differs from
 * the sources beside it. */
const char* ls_build_digest(void);

#ifdef __cplusplus
}
#endif
#endif /* LS_FFN_H */
