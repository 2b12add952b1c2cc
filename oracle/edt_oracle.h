/*
 * edt_oracle.h -- C interface of the CPU oracle for the exact Euclidean
 * distance transform (EDT).
 *
 * TEST INFRASTRUCTURE ONLY.  The oracle exists to check the GPU library, and
 * only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load it.  It shares no code, header or table with the GPU library.
 *
 * What it computes (paper, Section 2.1 "Distance transforms" and Section
 * 2.3.2 "Distance-transform kernels"): for every element x of each sample,
 * the distance to the nearest background (zero) element y under the metric
 * sum_a s_a^2 (x_a - y_a)^2 with per-axis sampling s, together with the
 * coordinates of that nearest background element.
 */
#ifndef EDT_ORACLE_H
#define EDT_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * oracle_edt -- exact EDT of `batch` independent samples.
 *
 * mask      [batch][shape[0]]...[shape[ndim-1]] bytes, C order, host memory.
 *           Nonzero = foreground, zero = background.
 * ndim      spatial rank, 1..8.
 * shape     ndim extents, each >= 1.
 * sampling  NULL, or ndim positive finite spacings.  NULL or all-ones selects
 *           the exact integer path (int64 arithmetic, rational breakpoint
 *           tests); anything else runs in IEEE double.
 * out_sq_i  NULL or [batch][voxels] int64: exact squared distance (integer
 *           path only; must be NULL for the double path).
 * out_sq_d  NULL or [batch][voxels] double: squared distance.
 * out_dist  NULL or [batch][voxels] float: sqrt of the squared distance,
 *           correctly rounded to float.
 * out_idx   NULL or [batch][ndim][voxels] int32: coordinates of the chosen
 *           nearest background element (the one with the smallest row-major
 *           flat index among all nearest ones).
 * nthreads  worker threads for the per-line loops (<= 0 means 1).
 *
 * A sample with no background element is measured against the virtual
 * element (-1, 0, ..., 0), whose coordinates are also what out_idx reports.
 *
 * Returns 0 on success, -1 on an invalid argument, -2 if a host allocation
 * failed.  All buffers are owned by the caller.
 */
int oracle_edt(const uint8_t *mask, int ndim, const int64_t *shape,
               int64_t batch, const double *sampling,
               int64_t *out_sq_i, double *out_sq_d, float *out_dist,
               int32_t *out_idx, int nthreads);

/*
 * oracle_dt_bf -- brute-force distance transform under a metric.
 *
 * metric    0 euclidean (value = squared distance sum_a s_a^2 d_a^2),
 *           1 taxicab (sum_a s_a |d_a|), 2 chessboard (max_a s_a |d_a|).
 * sampling  NULL (all ones) or ndim positive finite spacings.
 * out_value NULL or [batch][voxels] double: the metric value to the nearest
 *           background element.
 * out_idx   NULL or [batch][ndim][voxels] int32: its coordinates (the
 *           nearest one with the smallest row-major flat index).
 * Other arguments, the virtual element for samples without background and
 * the return codes are as for oracle_edt.  O(voxels x background) per sample.
 */
int oracle_dt_bf(const uint8_t *mask, int ndim, const int64_t *shape,
                 int64_t batch, int metric, const double *sampling,
                 double *out_value, int32_t *out_idx, int nthreads);

/* Number of threads the OpenMP runtime would actually use for `nthreads`. */
int oracle_threads_used(int nthreads);

#ifdef __cplusplus
}
#endif

#endif /* EDT_ORACLE_H */
