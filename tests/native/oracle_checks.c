/* The fp64 oracle (oracle/stepq_oracle.c) under the CPU sanitizers
 * (AddressSanitizer and UndefinedBehaviorSanitizer, built by
 * tests/test_sanitizers.py): every entry point on small random tiles of
 * ragged shapes, with pivot rows, both gate forms, both level
 * normalisations and every optional output, plus a pack/unpack round trip.
 * Memory errors and undefined behaviour abort; a failed round trip or a
 * non-finite result exits non-zero. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void orc_fit_absmax(int, int, int, const float *, const double *, const uint8_t *, float *, float *, int);
void orc_quantize(int, int, int, const double *, const float *, const float *, const uint8_t *, int8_t *, double *,
                  uint16_t *, int);
void orc_dequant(int, int, int, const int8_t *, const float *, const float *, const uint8_t *, const uint16_t *,
                 double *, int);
void orc_update_fp(int, int, int, const double *, const double *, const double *, const double *, const double *,
                   int, const double *, double *, double *);
void orc_decode_step(int, int, int, const int8_t *, const float *, const float *, const uint8_t *, const double *,
                     const double *, const double *, const double *, int, const double *, int8_t *, double *,
                     double *, const uint16_t *, uint16_t *, int);
void orc_decode_step_refit(int, int, int, const int8_t *, const float *, const float *, const uint8_t *,
                           const double *, const double *, const double *, const double *, const double *, int,
                           const double *, int8_t *, float *, float *, double *, double *, double *, double *,
                           double, double *, double *, const uint16_t *, uint16_t *, int);
void orc_decode_step_rowmax(int, int, int, const int8_t *, const float *, const float *, const uint8_t *,
                            const double *, const double *, const double *, const double *, int, const double *,
                            int8_t *, float *, float *, double *, double *, const uint16_t *, uint16_t *, int);
void orc_fit_dual_axis(int, int, int, const double *, const uint8_t *, const double *, float *, float *, int8_t *,
                       uint16_t *);
size_t orc_slot_bytes(int, int, int, const uint8_t *);
void orc_pack_pool(int, int, int, int, const uint8_t *, const int8_t *, const uint16_t *, const float *,
                   const float *, uint8_t *);
void orc_unpack_pool(int, int, int, int, const uint8_t *, const uint8_t *, int8_t *, uint16_t *, float *, float *);

static uint64_t rng_s = 12345;
static double unit(void)
{
    rng_s ^= rng_s << 13;
    rng_s ^= rng_s >> 7;
    rng_s ^= rng_s << 17;
    return (double)(rng_s >> 11) * (1.0 / 9007199254740992.0);
}
static double normal(void) { return sqrt(-2.0 * log(unit() + 1e-300)) * cos(6.283185307179586 * unit()); }

static int failures = 0;
static void expect(int ok, const char *what)
{
    if (!ok) {
        fprintf(stderr, "FAILED: %s\n", what);
        ++failures;
    }
}

static void *alloc(size_t n) { return calloc(n ? n : 1, 1); }

static void one_case(int Hv, int dk, int dv, int levels, int with_pivots)
{
    const int n = Hv;   /* one slot: its tiles */
    const size_t N = (size_t)n * dk * dv;
    uint8_t *bits = alloc((size_t)n * dk);
    for (int i = 0; i < n * dk; ++i) bits[i] = (uint8_t)(2 << (int)(unit() * 3));
    if (with_pivots)
        for (int h = 0; h < n; ++h) bits[h * dk + (int)(unit() * dk)] = 16;
    float *S = alloc(N * sizeof(float)), *r = alloc(n * dk * sizeof(float)), *c = alloc(n * dv * sizeof(float));
    double *X = alloc(N * sizeof(double)), *y = alloc(N * sizeof(double)), *y0 = alloc(N * sizeof(double));
    double *w = alloc(n * dk * sizeof(double));
    int8_t *codes = alloc(N), *codes2 = alloc(N);
    uint16_t *pv = alloc(N * 2), *pv2 = alloc(N * 2);
    for (size_t e = 0; e < N; ++e) S[e] = (float)(0.05 * normal());
    for (int i = 0; i < n * dk; ++i) w[i] = exp(0.5 * normal());
    orc_fit_absmax(n, dk, dv, S, w, bits, r, c, levels);
    for (size_t e = 0; e < N; ++e) X[e] = S[e];
    orc_quantize(n, dk, dv, X, r, c, bits, codes, y, pv, levels);
    orc_dequant(n, dk, dv, codes, r, c, bits, pv, X, levels);
    double *q = alloc(n * dk * sizeof(double)), *k = alloc(n * dk * sizeof(double));
    double *v = alloc(n * dv * sizeof(double)), *a = alloc(n * dk * sizeof(double));
    double *b = alloc(n * sizeof(double)), *o = alloc(n * dv * sizeof(double));
    for (int i = 0; i < n * dk; ++i) {
        q[i] = normal() / sqrt(dk);
        k[i] = normal() / sqrt(dk);
        a[i] = 0.9 + 0.1 * unit();
    }
    for (int j = 0; j < n * dv; ++j) v[j] = normal();
    for (int t = 0; t < n; ++t) b[t] = unit();
    double *Xo = alloc(N * sizeof(double)), *lo = alloc(n * dv * sizeof(double)), *hi = alloc(n * dv * sizeof(double));
    float *r2 = alloc(n * dk * sizeof(float)), *c2 = alloc(n * dv * sizeof(float));
    for (int per_row = 0; per_row < 2; ++per_row) {
        orc_update_fp(n, dk, dv, X, q, k, v, a, per_row, b, Xo, o);
        orc_decode_step(n, dk, dv, codes, r, c, bits, q, k, v, a, per_row, b, codes2, o, y, pv, pv2, levels);
        orc_decode_step(n, dk, dv, codes, r, c, bits, q, k, v, a, per_row, b, codes2, o, NULL, pv, pv2, levels);
        orc_decode_step_refit(n, dk, dv, codes, r, c, bits, w, q, k, v, a, per_row, b, codes2, r2, c2, o, y, y0, Xo,
                              2e-3, lo, hi, pv, pv2, levels);
        orc_decode_step_refit(n, dk, dv, codes, r, c, bits, NULL, q, k, v, a, per_row, b, codes2, r2, c2, o, NULL,
                              NULL, NULL, 2e-3, NULL, NULL, pv, pv2, levels);
        orc_decode_step_rowmax(n, dk, dv, codes, r, c, bits, q, k, v, a, per_row, b, codes2, r2, c2, o, y, pv, pv2,
                               levels);
        for (int j = 0; j < n * dv; ++j) expect(isfinite(o[j]), "finite readout");
    }
    orc_fit_dual_axis(n, dk, dv, Xo, bits, w, r2, c2, codes2, pv2);
    /* pack / unpack round trip of one slot */
    const size_t sb = orc_slot_bytes(Hv, dk, dv, bits);
    uint8_t *img = alloc(sb);
    int8_t *cu = alloc(N);
    uint16_t *pu = alloc(N * 2);
    float *ru = alloc(n * dk * sizeof(float)), *cc = alloc(n * dv * sizeof(float));
    for (size_t e = 0; e < N; ++e)
        if (bits[e / dv] == 16) codes[e] = 0;
    orc_pack_pool(1, Hv, dk, dv, bits, codes, pv, r, c, img);
    orc_unpack_pool(1, Hv, dk, dv, bits, img, cu, pu, ru, cc);
    expect(memcmp(cu, codes, N) == 0, "codes round trip");
    expect(memcmp(ru, r, n * dk * sizeof(float)) == 0 && memcmp(cc, c, n * dv * sizeof(float)) == 0,
           "scales round trip");
    for (size_t e = 0; e < N; ++e)
        if (bits[e / dv] == 16) expect(pu[e] == pv[e], "pivot values round trip");
    free(bits); free(S); free(r); free(c); free(X); free(y); free(y0); free(w); free(codes); free(codes2);
    free(pv); free(pv2); free(q); free(k); free(v); free(a); free(b); free(o); free(Xo); free(lo); free(hi);
    free(r2); free(c2); free(img); free(cu); free(pu); free(ru); free(cc);
}

int main(void)
{
    const int shapes[][3] = {{3, 37, 64}, {2, 128, 128}, {1, 1, 64}, {4, 96, 128}};
    for (int s = 0; s < 4; ++s)
        for (int levels = 0; levels < 2; ++levels)
            for (int piv = 0; piv < 2; ++piv) one_case(shapes[s][0], shapes[s][1], shapes[s][2], levels, piv);
    if (failures) {
        fprintf(stderr, "%d failed expectations\n", failures);
        return 1;
    }
    printf("oracle checks ok\n");
    return 0;
}
