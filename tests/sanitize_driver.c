/*
 * sanitize_driver.c -- runs the CPU oracle (oracle/edt_oracle.c) under
 * AddressSanitizer and UndefinedBehaviorSanitizer on seeded masks of rank
 * 1 to 4, unit and anisotropic sampling, with and without indices, one and
 * two threads, and checks on the way what the transform guarantees for any
 * input: zero on background, a reported nearest element that is background
 * and lies at the reported squared distance, and agreement of the
 * separable passes with the brute-force transform on the same input.
 *
 * Built and run by tests/test_oracle_sanitize.py; prints "ok" and exits 0 when
 * every case passes, exits 1 on the first failed check (the sanitizers abort
 * on their own findings).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "edt_oracle.h"

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;

/* splitmix64 (Steele, Lea, Flood 2014) */
static uint64_t next_u64(void) {
    uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

static int fail(const char *what, int ncase, int64_t i) {
    fprintf(stderr, "case %d: %s at element %lld\n", ncase, what, (long long)i);
    return 1;
}

/* Coordinates of flat element e of a sample of rank nd. */
static void coords(int64_t e, int nd, const int64_t *shape, int64_t *c) {
    for (int a = nd - 1; a >= 0; --a) {
        c[a] = e % shape[a];
        e /= shape[a];
    }
}

static int run_case(int ncase, int nd, const int64_t *shape, int64_t batch, double p_bg, const double *sampling,
                    int nthreads) {
    int64_t vox = 1;
    for (int a = 0; a < nd; ++a) vox *= shape[a];
    const int64_t total = vox * batch;
    uint8_t *mask = malloc((size_t)total);
    double *sq_d = malloc(sizeof(double) * (size_t)total);
    int64_t *sq_i = malloc(sizeof(int64_t) * (size_t)total);
    float *dist = malloc(sizeof(float) * (size_t)total);
    int32_t *idx = malloc(sizeof(int32_t) * (size_t)(total * nd));
    double *bf = malloc(sizeof(double) * (size_t)total);
    if (!mask || !sq_d || !sq_i || !dist || !idx || !bf) return fail("host allocation", ncase, -1);
    for (int64_t i = 0; i < total; ++i)
        mask[i] = (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0) < p_bg ? 0 : 1;
    if (ncase % 3 == 0) /* a sample without background */
        for (int64_t i = 0; i < vox; ++i) mask[i] = 1;

    int rc = oracle_edt(mask, nd, shape, batch, sampling, sampling ? NULL : sq_i, sq_d, dist, idx, nthreads);
    if (rc != 0) return fail("oracle_edt returned an error", ncase, rc);
    rc = oracle_dt_bf(mask, nd, shape, batch, 0, sampling, bf, NULL, nthreads);
    if (rc != 0) return fail("oracle_dt_bf returned an error", ncase, rc);

    double w[8];
    for (int a = 0; a < nd; ++a) w[a] = sampling ? sampling[a] * sampling[a] : 1.0;
    int64_t c[8];
    for (int64_t b = 0; b < batch; ++b) {
        int any_bg = 0;
        for (int64_t e = 0; e < vox; ++e) any_bg |= mask[b * vox + e] == 0;
        for (int64_t e = 0; e < vox; ++e) {
            const int64_t i = b * vox + e;
            if (mask[i] == 0 && sq_d[i] != 0.0) return fail("nonzero distance on background", ncase, i);
            if (!sampling && (double)sq_i[i] != sq_d[i]) return fail("integer and double outputs differ", ncase, i);
            /* the reported nearest element: background, at the reported distance */
            double d2 = 0.0;
            coords(e, nd, shape, c);
            int64_t f = 0;
            for (int a = 0; a < nd; ++a) {
                const int64_t y = idx[(b * nd + a) * vox + e];
                const double dd = (double)(c[a] - y);
                d2 += w[a] * dd * dd;
                f = f * shape[a] + y;
            }
            if (any_bg && mask[b * vox + f] != 0) return fail("index of a foreground element", ncase, i);
            if (fabs(d2 - sq_d[i]) > 1e-9 * (1.0 + sq_d[i])) return fail("index not at the distance", ncase, i);
            if (any_bg && fabs(bf[i] - sq_d[i]) > 1e-9 * (1.0 + bf[i])) return fail("differs from brute force", ncase, i);
            if (fabs((double)dist[i] - sqrt(sq_d[i])) > 1e-6 * (1.0 + sqrt(sq_d[i])))
                return fail("distance is not the root of the squared distance", ncase, i);
        }
    }
    free(mask);
    free(sq_d);
    free(sq_i);
    free(dist);
    free(idx);
    free(bf);
    return 0;
}

int main(void) {
    static const int64_t s1[] = {37};
    static const int64_t s2[] = {13, 29};
    static const int64_t s3[] = {7, 9, 11};
    static const int64_t s4[] = {3, 5, 4, 6};
    static const int64_t s5[] = {1, 1};
    static const double samp2[] = {2.5, 0.8};
    static const double samp3[] = {1.5, 0.7, 1.0};
    int ncase = 0;
    for (int th = 1; th <= 2; ++th) {
        if (run_case(++ncase, 1, s1, 3, 0.1, NULL, th)) return 1;
        if (run_case(++ncase, 2, s2, 2, 0.05, NULL, th)) return 1;
        if (run_case(++ncase, 2, s2, 2, 0.2, samp2, th)) return 1;
        if (run_case(++ncase, 3, s3, 2, 0.03, NULL, th)) return 1;
        if (run_case(++ncase, 3, s3, 2, 0.1, samp3, th)) return 1;
        if (run_case(++ncase, 4, s4, 2, 0.02, NULL, th)) return 1;
        if (run_case(++ncase, 2, s5, 4, 0.5, NULL, th)) return 1;
    }
    printf("ok %d cases\n", ncase);
    return 0;
}
