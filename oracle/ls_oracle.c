/*
 * ls_oracle.c - plain, slow, obviously correct CPU reference for one decode
 * step of the activation-sparse gated FFN (LeanStream, "speculate-and-refine"
 * decode).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  It shares no code, header,
 * table or helper with the GPU library; both sides only consume the same
 * seeded inputs.
 *
 * Precision: weights are decoded exactly from their storage type (binary32,
 * binary16 or bfloat16) to double; all arithmetic is double; loops run in the
 * textbook order with no blocking or fusion.
 *
 * What each function follows:
 *   orc_mlp_input     the MLP input h_n, as distinct from the residual x_n
 *                     (Sec. 2.1, before Eq. 1); RMS prenorm is a reading.
 *   orc_predict       the predictor's PCA-style input projection (Sec. 3.3.3)
 *                     followed by a linear head that scores neuron blocks.
 *   orc_select        priority list = blocks in descending predicted priority
 *                     (Sec. 2.1; Sec. 3.3.3), with a deterministic total order.
 *   orc_activations   gate/up projections and the gating of Eq. 1.
 *   orc_down          the down projection of Eq. 1, written as the sum over
 *                     hidden neurons of Sec. 3.2.2 (permutation invariance).
 *   orc_ffn_masked_dense  dense FFN with the activations of unselected
 *                     neurons zeroed (a second code path for the masked FFN).
 *
 * Parity pins: every function is pinned by the non-GPU tests (library
 * routines, closed forms, brute force, invariants); none is "parity unpinned".
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_F32 = 0, ORC_F16 = 1, ORC_BF16 = 2 };
enum { ORC_ACT_REGLU = 0, ORC_ACT_SWIGLU_THRESH = 1 };
enum { ORC_SEL_TOPK = 0, ORC_SEL_THRESHOLD = 1 };

/* ---------------------------------------------------------------------------
 * Exact decoding of the storage types (IEEE 754 binary16 / binary32, bfloat16).
 * ------------------------------------------------------------------------- */
static double decode_f16(uint16_t b) {
    int sign = (b >> 15) & 1;
    int e = (b >> 10) & 0x1f;
    int m = b & 0x3ff;
    double v;
    if (e == 0) {
        v = ldexp((double)m, -24); /* subnormal: m * 2^-24 */
    } else if (e == 31) {
        v = (m == 0) ? INFINITY : NAN;
    } else {
        v = ldexp((double)(1024 + m), e - 25); /* (1 + m/1024) * 2^(e-15) */
    }
    return sign ? -v : v;
}

static double decode_bf16(uint16_t b) {
    uint32_t bits = (uint32_t)b << 16; /* bfloat16 is the top half of a binary32 */
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

double orc_decode(const void* w, int dtype, size_t i) {
    if (dtype == ORC_F32) return (double)((const float*)w)[i];
    if (dtype == ORC_F16) return decode_f16(((const uint16_t*)w)[i]);
    return decode_bf16(((const uint16_t*)w)[i]);
}

/* ---------------------------------------------------------------------------
 * MLP input: h = x, or h = x / sqrt(mean(x^2) + 1e-6) (parameter-free RMS
 * prenorm of the residual state).
 * ------------------------------------------------------------------------- */
void orc_mlp_input(int d, const float* x, int rms, double* h) {
    if (!rms) {
        for (int c = 0; c < d; ++c) h[c] = (double)x[c];
        return;
    }
    double ss = 0.0;
    for (int c = 0; c < d; ++c) ss += (double)x[c] * (double)x[c];
    double scale = 1.0 / sqrt(ss / (double)d + 1e-6);
    for (int c = 0; c < d; ++c) h[c] = (double)x[c] * scale;
}

/* ---------------------------------------------------------------------------
 * Predictor: z_i = sum_c P1[i,c] h_c (P1 is [r, d]); s_b = sum_i P2[b,i] z_i
 * (P2 is [n_blk, r]).  Scores are handed out rounded to binary32, which is the
 * score interface both sides agree on.
 * ------------------------------------------------------------------------- */
static void predict_z_rows(int d, const void* p1, int dtype, const double* h, int lo, int hi,
                           double* z) {
    for (int i = lo; i < hi; ++i) {
        double acc = 0.0;
        for (int c = 0; c < d; ++c) acc += orc_decode(p1, dtype, (size_t)i * d + c) * h[c];
        z[i] = acc;
    }
}

static void predict_s_rows(int r, const void* p2, int dtype, const double* z, int lo, int hi,
                           float* scores) {
    for (int b = lo; b < hi; ++b) {
        double acc = 0.0;
        for (int i = 0; i < r; ++i) acc += orc_decode(p2, dtype, (size_t)b * r + i) * z[i];
        scores[b] = (float)acc;
    }
}

void orc_predict(int d, int r, int nblk, const void* p1, const void* p2, int dtype,
                 const double* h, double* z_out, float* scores) {
    double* z = z_out ? z_out : (double*)malloc(sizeof(double) * (size_t)r);
    predict_z_rows(d, p1, dtype, h, 0, r, z);
    predict_s_rows(r, p2, dtype, z, 0, nblk, scores);
    if (!z_out) free(z);
}

/* ---------------------------------------------------------------------------
 * Selection.  Total order on (score, block index):
 *   a ranks before b  iff  key(a) > key(b), or key(a) == key(b) and index(a) < index(b);
 *   key: NaN is below every number (including -inf); -0 equals +0; otherwise
 *   IEEE order.
 * Top-k is the first k entries in that order, so the output order is the
 * priority order.  Threshold mode keeps every non-NaN score strictly above tau,
 * in the same order.  With union_batch and B > 1: the union of the tokens'
 * selections, ordered by the largest key over all B tokens, then by index.
 * ------------------------------------------------------------------------- */

/* +1 if key(a) > key(b), -1 if key(a) < key(b), 0 if equal. */
static int key_cmp(float a, float b) {
    int na = isnan(a), nb = isnan(b);
    if (na && nb) return 0;
    if (na) return -1;
    if (nb) return 1;
    if (a > b) return 1; /* IEEE comparison: -0 == +0 */
    if (a < b) return -1;
    return 0;
}

/* Does (sa, ia) rank before (sb, ib)? */
static int ranks_before(float sa, int ia, float sb, int ib) {
    int c = key_cmp(sa, sb);
    if (c != 0) return c > 0;
    return ia < ib;
}

/* Sort `n` block ids in place by the total order on vals[id] (selection sort). */
static void order_ids(int* ids, int n, const float* vals) {
    for (int p = 0; p < n; ++p) {
        int best = p;
        for (int q = p + 1; q < n; ++q)
            if (ranks_before(vals[ids[q]], ids[q], vals[ids[best]], ids[best])) best = q;
        int t = ids[p];
        ids[p] = ids[best];
        ids[best] = t;
    }
}

/* One token's selection: writes the selected ids in priority order into out
 * and returns their number. */
static int select_one(const float* s, int nblk, int mode, int k, float tau, int* out) {
    int* ids = (int*)malloc(sizeof(int) * (size_t)nblk);
    int n = 0;
    for (int b = 0; b < nblk; ++b) {
        if (mode == ORC_SEL_THRESHOLD) {
            if (!isnan(s[b]) && s[b] > tau) ids[n++] = b;
        } else {
            ids[n++] = b;
        }
    }
    order_ids(ids, n, s);
    int m = (mode == ORC_SEL_TOPK) ? (k < n ? k : n) : n;
    for (int p = 0; p < m; ++p) out[p] = ids[p];
    free(ids);
    return m;
}

/* scores: [B, nblk] binary32.  Per-token (union_batch == 0 or B == 1): idx is
 * [B, cap], count is [B].  Union: idx is [cap], count is [1].
 * Returns 0, or -1 if the output does not fit in cap. */
int orc_select(const float* scores, int B, int nblk, int mode, int k, float tau,
               int union_batch, int cap, int* idx, int* count) {
    int* tmp = (int*)malloc(sizeof(int) * (size_t)nblk);
    if (!union_batch || B == 1) {
        for (int b = 0; b < B; ++b) {
            int m = select_one(scores + (size_t)b * nblk, nblk, mode, k, tau, tmp);
            if (m > cap) { free(tmp); return -1; }
            for (int p = 0; p < m; ++p) idx[(size_t)b * cap + p] = tmp[p];
            count[b] = m;
        }
        free(tmp);
        return 0;
    }
    unsigned char* member = (unsigned char*)calloc((size_t)nblk, 1);
    for (int b = 0; b < B; ++b) {
        int m = select_one(scores + (size_t)b * nblk, nblk, mode, k, tau, tmp);
        for (int p = 0; p < m; ++p) member[tmp[p]] = 1;
    }
    /* largest key of each block over all B tokens */
    float* best = (float*)malloc(sizeof(float) * (size_t)nblk);
    for (int i = 0; i < nblk; ++i) {
        float m = scores[i];
        for (int b = 1; b < B; ++b)
            if (key_cmp(scores[(size_t)b * nblk + i], m) > 0) m = scores[(size_t)b * nblk + i];
        best[i] = m;
    }
    int n = 0;
    for (int i = 0; i < nblk; ++i)
        if (member[i]) tmp[n++] = i;
    order_ids(tmp, n, best);
    int rc = 0;
    if (n > cap) {
        rc = -1;
    } else {
        for (int p = 0; p < n; ++p) idx[p] = tmp[p];
        count[0] = n;
    }
    free(best);
    free(member);
    free(tmp);
    return rc;
}

/* ---------------------------------------------------------------------------
 * Gate/up projections and gating (Eq. 1), for a list of hidden neurons.
 *   g_j = sum_c Wg[j,c] h_c + bias_j,   u_j = sum_c Wu[j,c] h_c
 *   ReGLU:            a_j = max(g_j, 0) * u_j
 *   SwiGLU-threshold: sigma_j = g_j / (1 + exp(-g_j));
 *                     a_j = sigma_j * u_j if |sigma_j| > t, else 0
 * Wg, Wu are [F, d] (nn.Linear layout); bias is [F] or NULL.
 * ------------------------------------------------------------------------- */
void orc_activations(int d, int F, const void* wg, const void* wu, const void* bias, int dtype,
                     int act, double thresh, const double* h, int n, const int* neurons,
                     double* g_out, double* u_out, double* a_out) {
    (void)F;
    for (int t = 0; t < n; ++t) {
        int j = neurons[t];
        double g = 0.0, u = 0.0;
        for (int c = 0; c < d; ++c) g += orc_decode(wg, dtype, (size_t)j * d + c) * h[c];
        for (int c = 0; c < d; ++c) u += orc_decode(wu, dtype, (size_t)j * d + c) * h[c];
        if (bias) g += orc_decode(bias, dtype, (size_t)j);
        double a;
        if (act == ORC_ACT_REGLU) {
            a = (g > 0.0 ? g : 0.0) * u;
        } else {
            double sig = g / (1.0 + exp(-g));
            a = (fabs(sig) > thresh) ? sig * u : 0.0;
        }
        if (g_out) g_out[t] = g;
        if (u_out) u_out[t] = u;
        a_out[t] = a;
    }
}

/* ---------------------------------------------------------------------------
 * Down projection (Eq. 1; Sec. 3.2.2): y_m = sum_t a_t * Wd[m, neurons[t]],
 * Wd is [d, F] (nn.Linear layout), summed in list order.
 * ------------------------------------------------------------------------- */
static void down_cols(int F, const void* wd, int dtype, int n, const int* neurons, const double* a,
                      int lo, int hi, double* y) {
    for (int m = lo; m < hi; ++m) {
        double acc = 0.0;
        for (int t = 0; t < n; ++t)
            acc += a[t] * orc_decode(wd, dtype, (size_t)m * F + neurons[t]);
        y[m] = acc;
    }
}

void orc_down(int d, int F, const void* wd, int dtype, int n, const int* neurons,
              const double* a, double* y) {
    down_cols(F, wd, dtype, n, neurons, a, 0, d, y);
}

/* ---------------------------------------------------------------------------
 * Masked dense FFN (second code path): every neuron's activation is computed
 * in index order, then a_j := 0 wherever mask[j] == 0, then y = Wd a.
 * mask == NULL means the dense FFN.
 * ------------------------------------------------------------------------- */
void orc_ffn_masked_dense(int d, int F, const void* wg, const void* wu, const void* wd,
                          const void* bias, int dtype, int act, double thresh, const double* h,
                          const unsigned char* mask, double* y) {
    double* a = (double*)malloc(sizeof(double) * (size_t)F);
    for (int j = 0; j < F; ++j) {
        double g = 0.0, u = 0.0;
        for (int c = 0; c < d; ++c) {
            g += orc_decode(wg, dtype, (size_t)j * d + c) * h[c];
            u += orc_decode(wu, dtype, (size_t)j * d + c) * h[c];
        }
        if (bias) g += orc_decode(bias, dtype, (size_t)j);
        if (act == ORC_ACT_REGLU) {
            a[j] = (g > 0.0 ? g : 0.0) * u;
        } else {
            double sig = g / (1.0 + exp(-g));
            a[j] = (fabs(sig) > thresh) ? sig * u : 0.0;
        }
        if (mask && !mask[j]) a[j] = 0.0;
    }
    for (int m = 0; m < d; ++m) {
        double acc = 0.0;
        for (int j = 0; j < F; ++j) acc += a[j] * orc_decode(wd, dtype, (size_t)m * F + j);
        y[m] = acc;
    }
    free(a);
}

/* ---------------------------------------------------------------------------
 * One whole layer of one decode step for one token, composed from the steps
 * above (used for the CPU baseline timing and by the tests):
 *   h = mlp_input(x); s = predict(h); idx = topk(s, k);
 *   neurons = blocks idx[0..count) expanded in list order;
 *   a = activations(neurons); y = down(a); x_out = x + y.
 * Writes scores [nblk], idx [k], y [d] (double) and x_out [d] (float).
 * ------------------------------------------------------------------------- */
int orc_layer_step(int d, int F, int r, int blk, const void* wg, const void* wu, const void* wd,
                   const void* bias, const void* p1, const void* p2, int dtype, int act,
                   double thresh, int rms, int k, const float* x, float* scores, int* idx,
                   double* y, float* x_out) {
    int nblk = F / blk;
    double* h = (double*)malloc(sizeof(double) * (size_t)d);
    orc_mlp_input(d, x, rms, h);
    orc_predict(d, r, nblk, p1, p2, dtype, h, NULL, scores);
    int count = 0;
    if (orc_select(scores, 1, nblk, ORC_SEL_TOPK, k, 0.0f, 0, k, idx, &count) != 0) {
        free(h);
        return -1;
    }
    int n = count * blk;
    int* neurons = (int*)malloc(sizeof(int) * (size_t)n);
    double* a = (double*)malloc(sizeof(double) * (size_t)n);
    for (int p = 0; p < count; ++p)
        for (int q = 0; q < blk; ++q) neurons[p * blk + q] = idx[p] * blk + q;
    orc_activations(d, F, wg, wu, bias, dtype, act, thresh, h, n, neurons, NULL, NULL, a);
    orc_down(d, F, wd, dtype, n, neurons, a, y);
    for (int m = 0; m < d; ++m) x_out[m] = (float)((double)x[m] + y[m]);
    free(a);
    free(neurons);
    free(h);
    return count;
}

/* ---------------------------------------------------------------------------
 * The same layer step with its loops over output elements split into n_threads
 * contiguous ranges on POSIX threads (predictor rows, then block scores, then
 * neurons, then output columns; the selection stays on the calling thread).
 * Every output element is the same sum in the same order as in orc_layer_step,
 * so the results are identical; only the wall time changes.  Used to time the
 * oracle on every host core.
 * ------------------------------------------------------------------------- */
typedef struct {
    int phase, lo, hi;
    int d, F, r, dtype, act, nblk;
    const void *wg, *wu, *wd, *bias, *p1, *p2;
    double thresh;
    const double* h;
    double* z;
    float* scores;
    const int* neurons;
    double* a;
    double* y;
    int n;
} mt_job;

static void* mt_run(void* arg) {
    mt_job* j = (mt_job*)arg;
    if (j->phase == 0) {
        predict_z_rows(j->d, j->p1, j->dtype, j->h, j->lo, j->hi, j->z);
    } else if (j->phase == 1) {
        predict_s_rows(j->r, j->p2, j->dtype, j->z, j->lo, j->hi, j->scores);
    } else if (j->phase == 2) {
        orc_activations(j->d, j->F, j->wg, j->wu, j->bias, j->dtype, j->act, j->thresh, j->h,
                        j->hi - j->lo, j->neurons + j->lo, NULL, NULL, j->a + j->lo);
    } else {
        down_cols(j->F, j->wd, j->dtype, j->n, j->neurons, j->a, j->lo, j->hi, j->y);
    }
    return NULL;
}

/* runs one phase over [0, total) split into nt contiguous ranges */
static void mt_phase(const mt_job* base, int phase, int total, int nt) {
    pthread_t th[256];
    int made[256];
    mt_job jobs[256];
    if (nt > 256) nt = 256;
    if (nt > total) nt = total > 0 ? total : 1;
    for (int t = 0; t < nt; ++t) {
        jobs[t] = *base;
        jobs[t].phase = phase;
        jobs[t].lo = (int)((int64_t)t * total / nt);
        jobs[t].hi = (int)((int64_t)(t + 1) * total / nt);
    }
    for (int t = 1; t < nt; ++t) {
        made[t] = pthread_create(&th[t], NULL, mt_run, &jobs[t]) == 0;
        if (!made[t]) mt_run(&jobs[t]); /* no thread: run the range here */
    }
    mt_run(&jobs[0]);
    for (int t = 1; t < nt; ++t)
        if (made[t]) pthread_join(th[t], NULL);
}

int orc_layer_step_mt(int d, int F, int r, int blk, const void* wg, const void* wu, const void* wd,
                      const void* bias, const void* p1, const void* p2, int dtype, int act,
                      double thresh, int rms, int k, const float* x, float* scores, int* idx,
                      double* y, float* x_out, int n_threads) {
    int nblk = F / blk;
    double* h = (double*)malloc(sizeof(double) * (size_t)d);
    double* z = (double*)malloc(sizeof(double) * (size_t)r);
    orc_mlp_input(d, x, rms, h);
    mt_job job;
    memset(&job, 0, sizeof job);
    job.d = d; job.F = F; job.r = r; job.dtype = dtype; job.act = act; job.nblk = nblk;
    job.wg = wg; job.wu = wu; job.wd = wd; job.bias = bias; job.p1 = p1; job.p2 = p2;
    job.thresh = thresh; job.h = h; job.z = z; job.scores = scores;
    mt_phase(&job, 0, r, n_threads);
    mt_phase(&job, 1, nblk, n_threads);
    int count = 0;
    if (orc_select(scores, 1, nblk, ORC_SEL_TOPK, k, 0.0f, 0, k, idx, &count) != 0) {
        free(z);
        free(h);
        return -1;
    }
    int n = count * blk;
    int* neurons = (int*)malloc(sizeof(int) * (size_t)n);
    double* a = (double*)malloc(sizeof(double) * (size_t)n);
    for (int p = 0; p < count; ++p)
        for (int q = 0; q < blk; ++q) neurons[p * blk + q] = idx[p] * blk + q;
    job.neurons = neurons; job.a = a; job.y = y; job.n = n;
    mt_phase(&job, 2, n, n_threads);
    mt_phase(&job, 3, d, n_threads);
    for (int m = 0; m < d; ++m) x_out[m] = (float)((double)x[m] + y[m]);
    free(a);
    free(neurons);
    free(z);
    free(h);
    return count;
}

/* ---------------------------------------------------------------------------
 * Stacked learnable hashing, inference (Sec. 3.3.1, Eq. hash_layer and
 * Eq. hashfunc_layer): five hashing layers, tau = 8 hash bits each, binary
 * features of width 256 between them.
 *
 *   layer 1:    c = sign(x W_1), W_1 real [d][8]
 *   layers 2-5: c = sign(x_k W_k), x_k and W_k in {-1,+1}, the product as
 *               XNOR + bitcount: x.w = 256 - 2 * popcount(x XOR w)
 *   index i = phi(c): the code read as an 8-bit number, first hash bit most
 *               significant, +1 -> 1 (the sign-pattern enumeration of the
 *               paper's matrix Z, Eq. hashfunc_mod)
 *   y_k = T_k[i] for k = 1..4; the last layer's index selects a row of the
 *   block-priority head (a reading: a regression output per block, quantised
 *   to 8-bit levels), which gives the block scores.
 * sign(0) = +1.  Bit-packed {-1,+1} vectors: element e is bit (e & 31) of word
 * e >> 5, 1 meaning +1.
 *
 * The first layer is the definition itself: each hash bit is the sign of the
 * real product x . W_1[:, b], summed in double precision in increasing j over
 * exactly represented binary32 operands.  The products are returned, so that a
 * caller comparing with a binary32 evaluation can see which decisions sit
 * within rounding distance of zero; a caller may also impose the first
 * layer's bucket (code0 >= 0) and have only the later, integer layers
 * evaluated from it.
 * ------------------------------------------------------------------------- */
enum { ORC_TAU = 8, ORC_DH = 256, ORC_DHW = ORC_DH / 32, ORC_NLAYERS = 5 };

static int popcount32(uint32_t v) {
    int c = 0;
    while (v) {
        v &= v - 1;
        ++c;
    }
    return c;
}

/* codes[5]: the five bucket indices; scores[nblk] = head[codes[4]][b].
 * prods[8] (may be NULL): the first layer's real products in double.
 * code0 < 0: the first bucket is phi(sign(x W_1)); code0 in [0, 255]: it is
 * code0 (the products are still returned). */
void orc_hash_predict(int d, int nblk, const float* x, const float* w1, const uint32_t* w_bin,
                      const uint32_t* tables, const uint8_t* head, int code0, double* prods,
                      int* codes, float* scores) {
    int idx = 0;
    for (int b = 0; b < ORC_TAU; ++b) {
        double acc = 0.0;
        for (int j = 0; j < d; ++j) acc += (double)x[j] * (double)w1[(size_t)j * ORC_TAU + b];
        if (prods) prods[b] = acc;
        idx = 2 * idx + (acc >= 0.0 ? 1 : 0);
    }
    if (code0 >= 0) idx = code0;
    codes[0] = idx;
    for (int k = 1; k < ORC_NLAYERS; ++k) {
        const uint32_t* y = tables + ((size_t)(k - 1) * ORC_DH + (size_t)idx) * ORC_DHW; /* y_k = T_k[i] */
        int next = 0;
        for (int b = 0; b < ORC_TAU; ++b) {
            const uint32_t* w = w_bin + ((size_t)(k - 1) * ORC_TAU + b) * ORC_DHW;
            int mismatch = 0;
            for (int m = 0; m < ORC_DHW; ++m) mismatch += popcount32(y[m] ^ w[m]);
            const int dot = ORC_DH - 2 * mismatch;
            next = 2 * next + (dot >= 0 ? 1 : 0);
        }
        idx = next;
        codes[k] = idx;
    }
    for (int b = 0; b < nblk; ++b) scores[b] = (float)head[(size_t)idx * nblk + b];
}
