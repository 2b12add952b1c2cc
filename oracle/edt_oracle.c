/*
 * edt_oracle.c -- plain, slow, obviously correct CPU oracle for the exact
 * Euclidean distance transform.
 *
 * TEST INFRASTRUCTURE ONLY: it is called by the tests, by the smoke check and
 * by the benchmark's CPU-baseline leg, never by the GPU library, and it shares
 * no code with it.
 *
 * Method (paper, Section 2.3.2 "Distance-transform kernels", which follows the
 * separable lower-envelope formulation of Felzenszwalb and Huttenlocher, 2012,
 * cited in Section 2.1): the squared distance
 *
 *     D2(x) = min over background y of  sum_a w_a (x_a - y_a)^2,  w_a = s_a^2
 *
 * separates into one-dimensional minimisations, one axis at a time.  Starting
 * from g = 0 on background and g = "no site" elsewhere, each axis a (from the
 * last, contiguous one down to axis 0) replaces every line along a by
 *
 *     g'(q) = min over sites p of the line of  g(p) + w_a (q - p)^2,
 *
 * i.e. the lower envelope of the parabolas rooted at the line's sites.  The
 * envelope is built left to right with a stack of parabola apexes v[] and the
 * abscissae z[] where each one becomes the lowest; then every position reads
 * the parabola whose interval contains it.
 *
 * Ties (our reading; the paper only requires that a returned index is a
 * genuine nearest background element, Section 2.4): a parabola is removed
 * when the new one already undercuts it at or before its interval start, and
 * a query moves to the next parabola only when that parabola's interval
 * starts strictly before the query position.  Each pass therefore keeps the
 * smallest position among equal minimisers, and running the passes from the
 * last axis to axis 0 returns, among all nearest background elements, the
 * one with the smallest row-major flat index.
 *
 * Unit sampling runs in exact int64 arithmetic: a breakpoint is kept as the
 * rational num/den (den > 0) and compared by cross-multiplying in 128 bits.
 * Other samplings run in IEEE double.
 *
 * A sample without any background element (paper, Section 2.3.2: the same
 * virtual out-of-bounds convention as SciPy) is measured against the virtual
 * element (-1, 0, ..., 0).
 */
#include "edt_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define MAXDIM 8
#define NO_SITE_I INT64_MAX /* "no site yet" in the integer field; never added */
#define NO_INDEX (-1)

/* ---------------------------------------------------------------------- */
/* One-dimensional lower envelope, exact integer version (w = 1).          */
/* ---------------------------------------------------------------------- */

/*
 * f[0..n)  : squared distance carried so far, NO_SITE_I where the position
 *            has no background element yet.
 * id[0..n) : flat index of the background element that realises f.
 * g, gid   : results (may not alias f, id).
 * v, zn, zd: work arrays of n entries (apex positions, breakpoint num/den).
 */
static void envelope_int(int64_t n, const int64_t *f, const int64_t *id,
                         int64_t *g, int64_t *gid,
                         int64_t *v, int64_t *zn, int64_t *zd)
{
    int64_t k = -1; /* index of the top parabola; -1 = empty envelope */
    for (int64_t q = 0; q < n; ++q) {
        if (f[q] == NO_SITE_I)
            continue;
        int64_t num = 0, den = 1;
        while (k >= 0) {
            int64_t p = v[k];
            /* The parabolas rooted at p and q meet at num / den. */
            num = (f[q] + q * q) - (f[p] + p * p);
            den = 2 * (q - p);
            /* Parabola k is hidden if q is already at least as low at the
             * start of k's interval (k = 0 starts at minus infinity). */
            if (k >= 1 && (__int128)num * zd[k] <= (__int128)zn[k] * den) {
                --k;
                continue;
            }
            break;
        }
        ++k;
        v[k] = q;
        zn[k] = num; /* unused for k == 0 */
        zd[k] = den;
    }
    if (k < 0) {
        for (int64_t q = 0; q < n; ++q) {
            g[q] = NO_SITE_I;
            gid[q] = NO_INDEX;
        }
        return;
    }
    int64_t j = 0;
    for (int64_t q = 0; q < n; ++q) {
        /* Move on while the next parabola's interval starts before q. */
        while (j < k && (__int128)zn[j + 1] < (__int128)q * zd[j + 1])
            ++j;
        int64_t p = v[j];
        g[q] = f[p] + (q - p) * (q - p);
        gid[q] = id[p];
    }
}

/* ---------------------------------------------------------------------- */
/* One-dimensional lower envelope, double version with weight w = s^2.     */
/* ---------------------------------------------------------------------- */

static void envelope_dbl(int64_t n, double w, const double *f,
                         const int64_t *id, double *g, int64_t *gid,
                         int64_t *v, double *z)
{
    int64_t k = -1;
    for (int64_t q = 0; q < n; ++q) {
        if (isinf(f[q]))
            continue;
        double s = -INFINITY;
        while (k >= 0) {
            int64_t p = v[k];
            double dq = (double)q, dp = (double)p;
            s = ((f[q] + w * dq * dq) - (f[p] + w * dp * dp)) /
                (2.0 * w * (dq - dp));
            if (k >= 1 && s <= z[k]) {
                --k;
                continue;
            }
            break;
        }
        ++k;
        v[k] = q;
        z[k] = s;
    }
    if (k < 0) {
        for (int64_t q = 0; q < n; ++q) {
            g[q] = INFINITY;
            gid[q] = NO_INDEX;
        }
        return;
    }
    int64_t j = 0;
    for (int64_t q = 0; q < n; ++q) {
        while (j < k && z[j + 1] < (double)q)
            ++j;
        int64_t p = v[j];
        double d = (double)(q - p);
        g[q] = f[p] + w * d * d;
        gid[q] = id[p];
    }
}

/* ---------------------------------------------------------------------- */
/* Driver: per sample, per axis (last to first), per line.                 */
/* ---------------------------------------------------------------------- */

int oracle_threads_used(int nthreads)
{
    if (nthreads < 1)
        nthreads = 1;
#ifdef _OPENMP
    int used = 1;
#pragma omp parallel num_threads(nthreads)
    {
#pragma omp single
        used = omp_get_num_threads();
    }
    return used;
#else
    return 1;
#endif
}

/* Run the 1-D pass along `axis` over every line of one sample. */
static int pass_axis(int ndim, const int64_t *shape, int axis, int integer,
                     double w, int64_t *gi, double *gd, int64_t *id,
                     int nthreads)
{
    int64_t n = shape[axis];
    int64_t inner = 1, outer = 1;
    for (int a = axis + 1; a < ndim; ++a)
        inner *= shape[a];
    for (int a = 0; a < axis; ++a)
        outer *= shape[a];
    int64_t lines = outer * inner;
    int failed = 0;

#pragma omp parallel num_threads(nthreads)
    {
        /* Per-thread copies of one line plus the envelope work arrays. */
        int64_t *fi = NULL, *gi2 = NULL, *zn = NULL, *zd = NULL;
        double *fd = NULL, *gd2 = NULL, *z = NULL;
        int64_t *fid = malloc(sizeof(int64_t) * n);
        int64_t *gid = malloc(sizeof(int64_t) * n);
        int64_t *v = malloc(sizeof(int64_t) * n);
        int ok = fid && gid && v;
        if (integer) {
            fi = malloc(sizeof(int64_t) * n);
            gi2 = malloc(sizeof(int64_t) * n);
            zn = malloc(sizeof(int64_t) * n);
            zd = malloc(sizeof(int64_t) * n);
            ok = ok && fi && gi2 && zn && zd;
        } else {
            fd = malloc(sizeof(double) * n);
            gd2 = malloc(sizeof(double) * n);
            z = malloc(sizeof(double) * n);
            ok = ok && fd && gd2 && z;
        }
        if (!ok) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp barrier
        if (!failed) {
#pragma omp for schedule(static)
            for (int64_t line = 0; line < lines; ++line) {
                int64_t o = line / inner, i = line % inner;
                int64_t base = o * n * inner + i;
                for (int64_t q = 0; q < n; ++q) {
                    int64_t e = base + q * inner;
                    fid[q] = id[e];
                    if (integer)
                        fi[q] = gi[e];
                    else
                        fd[q] = gd[e];
                }
                if (integer)
                    envelope_int(n, fi, fid, gi2, gid, v, zn, zd);
                else
                    envelope_dbl(n, w, fd, fid, gd2, gid, v, z);
                for (int64_t q = 0; q < n; ++q) {
                    int64_t e = base + q * inner;
                    id[e] = gid[q];
                    if (integer)
                        gi[e] = gi2[q];
                    else
                        gd[e] = gd2[q];
                }
            }
        }
        free(fi); free(gi2); free(zn); free(zd);
        free(fd); free(gd2); free(z);
        free(fid); free(gid); free(v);
    }
    return failed ? -2 : 0;
}

int oracle_edt(const uint8_t *mask, int ndim, const int64_t *shape,
               int64_t batch, const double *sampling,
               int64_t *out_sq_i, double *out_sq_d, float *out_dist,
               int32_t *out_idx, int nthreads)
{
    if (!mask || !shape || ndim < 1 || ndim > MAXDIM || batch < 1)
        return -1;
    int64_t vox = 1;
    for (int a = 0; a < ndim; ++a) {
        if (shape[a] < 1)
            return -1;
        vox *= shape[a];
    }
    if (vox >= ((int64_t)1 << 31))
        return -1;
    int integer = 1;
    double w[MAXDIM];
    for (int a = 0; a < ndim; ++a) {
        double s = sampling ? sampling[a] : 1.0;
        if (!(s > 0.0) || !isfinite(s))
            return -1;
        if (s != 1.0)
            integer = 0;
        w[a] = s * s;
    }
    if (!integer && out_sq_i)
        return -1;
    if (nthreads < 1)
        nthreads = 1;

    int64_t *gi = NULL;
    double *gd = NULL;
    int64_t *id = malloc(sizeof(int64_t) * vox);
    if (integer)
        gi = malloc(sizeof(int64_t) * vox);
    else
        gd = malloc(sizeof(double) * vox);
    if (!id || (integer && !gi) || (!integer && !gd)) {
        free(id); free(gi); free(gd);
        return -2;
    }

    int rc = 0;
    for (int64_t b = 0; b < batch && rc == 0; ++b) {
        const uint8_t *m = mask + b * vox;
        int any_background = 0;
        for (int64_t e = 0; e < vox; ++e) {
            int bg = (m[e] == 0);
            any_background |= bg;
            id[e] = bg ? e : NO_INDEX;
            if (integer)
                gi[e] = bg ? 0 : NO_SITE_I;
            else
                gd[e] = bg ? 0.0 : INFINITY;
        }
        for (int axis = ndim - 1; axis >= 0 && rc == 0; --axis)
            rc = pass_axis(ndim, shape, axis, integer, w[axis], gi, gd, id,
                           nthreads);
        if (rc)
            break;

        /* Outputs: squared distance, its square root, coordinates. */
        for (int64_t e = 0; e < vox; ++e) {
            int64_t c[MAXDIM], y[MAXDIM];
            int64_t r = e;
            for (int a = ndim - 1; a >= 0; --a) {
                c[a] = r % shape[a];
                r /= shape[a];
            }
            int64_t sq_i = 0;
            double sq_d = 0.0;
            if (!any_background) {
                /* Virtual background element (-1, 0, ..., 0); summed from
                 * the last axis to the first, like the passes. */
                for (int a = 0; a < ndim; ++a)
                    y[a] = 0;
                y[0] = -1;
                for (int a = ndim - 1; a >= 0; --a) {
                    int64_t d = c[a] - y[a];
                    sq_i += d * d;
                    sq_d += w[a] * (double)d * (double)d;
                }
            } else {
                int64_t t = id[e];
                for (int a = ndim - 1; a >= 0; --a) {
                    y[a] = t % shape[a];
                    t /= shape[a];
                }
                if (integer)
                    sq_i = gi[e];
                else
                    sq_d = gd[e];
            }
            if (integer)
                sq_d = (double)sq_i;
            if (out_sq_i)
                out_sq_i[b * vox + e] = sq_i;
            if (out_sq_d)
                out_sq_d[b * vox + e] = sq_d;
            if (out_dist)
                out_dist[b * vox + e] = (float)sqrt(sq_d);
            if (out_idx)
                for (int a = 0; a < ndim; ++a)
                    out_idx[(b * ndim + a) * vox + e] = (int32_t)y[a];
        }
    }
    free(id); free(gi); free(gd);
    return rc;
}

/* ---------------------------------------------------------------------- */
/* Brute-force distance transform under three metrics.                     */
/* ---------------------------------------------------------------------- */

/*
 * The definition written out (paper, Section 2.1 "Distance transforms" for
 * the transform, Section 2.3.2 for the brute-force transform that serves as
 * the exactness check and for the chessboard / taxicab metrics): for every
 * element x, the smallest metric value to a background element y,
 *
 *     euclidean  sum_a w_a (x_a - y_a)^2     (the squared distance, w_a = s_a^2)
 *     taxicab    sum_a s_a |x_a - y_a|
 *     chessboard max_a s_a |x_a - y_a|
 *
 * found by visiting the background elements in row-major order and keeping
 * the first strictly smaller value, so the reported element is the nearest
 * one with the smallest flat index.  A sample without background uses the
 * virtual element (-1, 0, ..., 0), as the exact transform does.
 */
int oracle_dt_bf(const uint8_t *mask, int ndim, const int64_t *shape,
                 int64_t batch, int metric, const double *sampling,
                 double *out_value, int32_t *out_idx, int nthreads)
{
    if (!mask || !shape || ndim < 1 || ndim > MAXDIM || batch < 1 || metric < 0 || metric > 2)
        return -1;
    int64_t vox = 1;
    for (int a = 0; a < ndim; ++a) {
        if (shape[a] < 1)
            return -1;
        vox *= shape[a];
    }
    if (vox >= ((int64_t)1 << 31))
        return -1;
    double s[MAXDIM];
    for (int a = 0; a < ndim; ++a) {
        s[a] = sampling ? sampling[a] : 1.0;
        if (!(s[a] > 0.0) || !isfinite(s[a]))
            return -1;
    }
    if (nthreads < 1)
        nthreads = 1;
    int64_t *zc = malloc(sizeof(int64_t) * (size_t)vox * ndim);   /* background coordinates */
    if (!zc)
        return -2;
    for (int64_t b = 0; b < batch; ++b) {
        const uint8_t *m = mask + b * vox;
        int64_t nz = 0;
        for (int64_t e = 0; e < vox; ++e) {
            if (m[e] != 0)
                continue;
            int64_t r = e;
            for (int a = ndim - 1; a >= 0; --a) {
                zc[nz * ndim + a] = r % shape[a];
                r /= shape[a];
            }
            ++nz;
        }
        if (nz == 0) {
            for (int a = 0; a < ndim; ++a)
                zc[a] = 0;
            zc[0] = -1;
            nz = 1;
        }
#pragma omp parallel for num_threads(nthreads) schedule(static)
        for (int64_t e = 0; e < vox; ++e) {
            int64_t c[MAXDIM];
            int64_t r = e;
            for (int a = ndim - 1; a >= 0; --a) {
                c[a] = r % shape[a];
                r /= shape[a];
            }
            double best = INFINITY;
            int64_t arg = 0;
            for (int64_t k = 0; k < nz; ++k) {
                const int64_t *y = zc + k * ndim;
                double v = 0.0;
                for (int a = 0; a < ndim; ++a) {
                    double d = fabs((double)(c[a] - y[a]));
                    if (metric == 0)
                        v += s[a] * s[a] * d * d;
                    else if (metric == 1)
                        v += s[a] * d;
                    else if (s[a] * d > v)
                        v = s[a] * d;
                }
                if (v < best) {
                    best = v;
                    arg = k;
                }
            }
            if (out_value)
                out_value[b * vox + e] = best;
            if (out_idx)
                for (int a = 0; a < ndim; ++a)
                    out_idx[(b * ndim + a) * vox + e] = (int32_t)zc[arg * ndim + a];
        }
    }
    free(zc);
    return 0;
}
