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
void orc_predict(int d, int r, int nblk, const void* p1, const void* p2, int dtype,
                 const double* h, double* z_out, float* scores) {
    double* z = z_out ? z_out : (double*)malloc(sizeof(double) * (size_t)r);
    for (int i = 0; i < r; ++i) {
        double acc = 0.0;
        for (int c = 0; c < d; ++c) acc += orc_decode(p1, dtype, (size_t)i * d + c) * h[c];
        z[i] = acc;
    }
    for (int b = 0; b < nblk; ++b) {
        double acc = 0.0;
        for (int i = 0; i < r; ++i) acc += orc_decode(p2, dtype, (size_t)b * r + i) * z[i];
        scores[b] = (float)acc;
    }
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
void orc_down(int d, int F, const void* wd, int dtype, int n, const int* neurons,
              const double* a, double* y) {
    for (int m = 0; m < d; ++m) {
        double acc = 0.0;
        for (int t = 0; t < n; ++t)
            acc += a[t] * orc_decode(wd, dtype, (size_t)m * F + neurons[t]);
        y[m] = acc;
    }
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
 * The first layer's code is a floating-point decision, so it is taken in the
 * GPU kernel's precision and order (binary32 fused multiply-adds): for each
 * hash bit, 256 partial sums over j = t, t + 256, ... in increasing j, then
 * the pairwise halving sum p[t] += p[t + s] for s = 128, 64, ..., 1.
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

/* codes[5]: the five bucket indices; scores[nblk] = head[codes[4]][b]. */
void orc_hash_predict(int d, int nblk, const float* x, const float* w1, const uint32_t* w_bin,
                      const uint32_t* tables, const uint8_t* head, int* codes, float* scores) {
    int idx = 0;
    for (int b = 0; b < ORC_TAU; ++b) {
        float p[ORC_DH];
        for (int t = 0; t < ORC_DH; ++t) {
            float acc = 0.f;
            for (int j = t; j < d; j += ORC_DH) acc = fmaf(x[j], w1[(size_t)j * ORC_TAU + b], acc);
            p[t] = acc;
        }
        for (int s = ORC_DH / 2; s >= 1; s /= 2)
            for (int t = 0; t < s; ++t) p[t] = p[t] + p[t + s];
        idx = 2 * idx + (p[0] >= 0.f ? 1 : 0);
    }
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
