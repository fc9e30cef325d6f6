/*
 * lsgen.c - seeded, counter-based synthetic input generator.
 *
 * This module holds no arithmetic of the sparse-FFN method.  It only draws
 * random numbers and rounds them to a storage type, so that the CPU oracle and
 * the GPU path consume byte-identical inputs.
 *
 * Definition of element i of stream (seed, tensor_id, layer):
 *   base = splitmix64_mix(seed ^ splitmix64_mix((tensor_id << 32) | layer))
 *   p    = i >> 1  (elements 2p and 2p+1 share one Box-Muller pair)
 *   r1   = splitmix64_mix(base + (2p+1) * GAMMA)      (SplitMix64 output 2p+1)
 *   r2   = splitmix64_mix(base + (2p+2) * GAMMA)      (SplitMix64 output 2p+2)
 *   u1   = ((r1 >> 11) + 1) * 2^-53                   in (0, 1]
 *   u2   =  (r2 >> 11)      * 2^-53                   in [0, 1)
 *   z    = sqrt(-2 ln u1) * (i even ? cos : sin)(2 pi u2)   (Box-Muller, fp64)
 *   v    = mean + std * z, rounded to the storage type with round-to-nearest-even
 * SplitMix64 is the generator of Steele, Lea and Flood (OOPSLA 2014): the n-th
 * output of a generator seeded with s is mix(s + n * GAMMA).
 *
 * Storage types: 0 = IEEE binary32, 1 = IEEE binary16, 2 = bfloat16.
 * The result is independent of the thread count.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

#define GAMMA 0x9E3779B97F4A7C15ULL

static uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static uint64_t stream_base(uint64_t seed, uint32_t tensor_id, uint32_t layer) {
    return mix64(seed ^ mix64(((uint64_t)tensor_id << 32) | (uint64_t)layer));
}

static double normal_at(uint64_t base, uint64_t i) {
    uint64_t p = i >> 1;
    uint64_t r1 = mix64(base + (2 * p + 1) * GAMMA);
    uint64_t r2 = mix64(base + (2 * p + 2) * GAMMA);
    double u1 = (double)((r1 >> 11) + 1) * 0x1.0p-53;
    double u2 = (double)(r2 >> 11) * 0x1.0p-53;
    double rad = sqrt(-2.0 * log(u1));
    double ang = 6.283185307179586476925286766559 * u2;
    return (i & 1) ? rad * sin(ang) : rad * cos(ang);
}

/* Round a double to a binary floating format with `prec` significand bits
 * (implicit bit included), exponent bias `bias` and `ebits` exponent bits,
 * round-to-nearest-even, returning the encoded bits.  nearbyint() honours the
 * default rounding mode, which is round-to-nearest-even. */
static uint32_t encode_rne(double v, int prec, int ebits, int bias) {
    const uint32_t emax_field = (1u << ebits) - 1u;
    const int mbits = prec - 1;
    uint32_t sign = signbit(v) ? 1u : 0u;
    uint32_t out_sign = sign << (ebits + mbits);
    if (isnan(v)) return out_sign | (emax_field << mbits) | (1u << (mbits - 1));
    double a = fabs(v);
    if (isinf(a)) return out_sign | (emax_field << mbits);
    const int emin = 1 - bias; /* exponent of the smallest normal */
    if (a < ldexp(1.0, emin)) {
        /* subnormal range: fixed quantum 2^(emin - mbits) */
        double q = nearbyint(ldexp(a, mbits - emin));
        return out_sign | (uint32_t)q; /* q == 2^mbits encodes the smallest normal */
    }
    int e;
    (void)frexp(a, &e);                  /* a = m * 2^e, m in [0.5, 1) */
    double q = nearbyint(ldexp(a, prec - e)); /* in [2^(prec-1), 2^prec] */
    if (q == ldexp(1.0, prec)) { q = ldexp(1.0, prec - 1); e += 1; }
    int field = (e - 1) + bias;
    if (field >= (int)emax_field) return out_sign | (emax_field << mbits);
    return out_sign | ((uint32_t)field << mbits) | ((uint32_t)q - (1u << mbits));
}

static void store(double v, int dtype, void* out, uint64_t i) {
    if (dtype == 0) {
        ((float*)out)[i] = (float)v; /* C conversion rounds to nearest even */
    } else if (dtype == 1) {
        ((uint16_t*)out)[i] = (uint16_t)encode_rne(v, 11, 5, 15);
    } else {
        ((uint16_t*)out)[i] = (uint16_t)encode_rne(v, 8, 8, 127);
    }
}

typedef struct {
    uint64_t base, offset, lo, hi;
    double mean, std;
    int dtype;
    void* out;
} job_t;

static void* run_job(void* p) {
    job_t* j = (job_t*)p;
    for (uint64_t i = j->lo; i < j->hi; ++i)
        store(j->mean + j->std * normal_at(j->base, j->offset + i), j->dtype, j->out, i);
    return NULL;
}

/* Fill out[0..n) with elements offset..offset+n of the stream, scaled to
 * N(mean, std^2) and rounded to `dtype`.  Returns 0, or -1 on a bad argument. */
int lsgen_normal(uint64_t seed, uint32_t tensor_id, uint32_t layer, uint64_t offset,
                 uint64_t n, double mean, double std, int dtype, void* out, int nthreads) {
    if (dtype < 0 || dtype > 2 || (out == NULL && n > 0)) return -1;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 64) nthreads = 64;
    if ((uint64_t)nthreads > n / 65536 + 1) nthreads = (int)(n / 65536 + 1);
    uint64_t base = stream_base(seed, tensor_id, layer);
    job_t jobs[64];
    pthread_t th[64];
    for (int t = 0; t < nthreads; ++t) {
        jobs[t].base = base;
        jobs[t].offset = offset;
        jobs[t].lo = n * (uint64_t)t / (uint64_t)nthreads;
        jobs[t].hi = n * (uint64_t)(t + 1) / (uint64_t)nthreads;
        jobs[t].mean = mean;
        jobs[t].std = std;
        jobs[t].dtype = dtype;
        jobs[t].out = out;
    }
    int started = 0;
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, run_job, &jobs[t]) != 0) break;
        started = t;
    }
    run_job(&jobs[0]);
    for (int t = started + 1; t < nthreads; ++t) run_job(&jobs[t]); /* threads that failed to start */
    for (int t = 1; t <= started; ++t) pthread_join(th[t], NULL);
    return 0;
}

/* Fill out[0..n) with the constant `value` rounded to `dtype`. */
int lsgen_const(double value, uint64_t n, int dtype, void* out) {
    if (dtype < 0 || dtype > 2 || (out == NULL && n > 0)) return -1;
    for (uint64_t i = 0; i < n; ++i) store(value, dtype, out, i);
    return 0;
}

/* The raw SplitMix64 output n (n >= 1) of a generator seeded with s; exported
 * so tests can check the generator against its published definition. */
uint64_t lsgen_splitmix64(uint64_t s, uint64_t n) { return mix64(s + n * GAMMA); }
