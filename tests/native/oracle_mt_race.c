/* Driver of the oracle's thread-split layer step for ThreadSanitizer builds: one small
 * fp32 layer with deterministic values, the step run on 1 and on 7 threads; exit status 0
 * when both runs give the same list and bitwise the same outputs. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int orc_layer_step(int d, int F, int r, int blk, const void* wg, const void* wu, const void* wd,
                   const void* bias, const void* p1, const void* p2, int dtype, int act,
                   double thresh, int rms, int k, const float* x, float* scores, int* idx,
                   double* y, float* x_out);
int orc_layer_step_mt(int d, int F, int r, int blk, const void* wg, const void* wu, const void* wd,
                      const void* bias, const void* p1, const void* p2, int dtype, int act,
                      double thresh, int rms, int k, const float* x, float* scores, int* idx,
                      double* y, float* x_out, int n_threads);

static float val(uint32_t i) { /* deterministic values in [-1, 1) */
    i = i * 2654435761u + 12345u;
    i ^= i >> 13;
    return (float)(i % 2001u) / 1000.0f - 1.0f;
}

int main(void) {
    enum { D = 64, F = 256, R = 64, BLK = 16, NB = F / BLK, K = 5 };
    float *wg = malloc(sizeof(float) * F * D), *wu = malloc(sizeof(float) * F * D), *wd = malloc(sizeof(float) * D * F);
    float *p1 = malloc(sizeof(float) * R * D), *p2 = malloc(sizeof(float) * NB * R), x[D];
    for (int i = 0; i < F * D; ++i) { wg[i] = val(i); wu[i] = val(i + 100000); wd[i] = val(i + 200000); }
    for (int i = 0; i < R * D; ++i) p1[i] = val(i + 300000);
    for (int i = 0; i < NB * R; ++i) p2[i] = val(i + 400000);
    for (int i = 0; i < D; ++i) x[i] = val(i + 500000);
    float s1[NB], s7[NB], o1[D], o7[D];
    int i1[K], i7[K];
    double y1[D], y7[D];
    int n1 = orc_layer_step(D, F, R, BLK, wg, wu, wd, NULL, p1, p2, 0, 0, 0.0, 1, K, x, s1, i1, y1, o1);
    int n7 = orc_layer_step_mt(D, F, R, BLK, wg, wu, wd, NULL, p1, p2, 0, 0, 0.0, 1, K, x, s7, i7, y7, o7, 7);
    int ok = n1 == K && n7 == K && !memcmp(s1, s7, sizeof s1) && !memcmp(i1, i7, sizeof i1) &&
             !memcmp(y1, y7, sizeof y1) && !memcmp(o1, o7, sizeof o1);
    free(wg); free(wu); free(wd); free(p1); free(p2);
    puts(ok ? "oracle_mt_race ok" : "oracle_mt_race MISMATCH");
    return ok ? 0 : 1;
}
