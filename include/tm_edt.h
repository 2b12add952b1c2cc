/*
 * tm_edt.h -- exact Euclidean distance transform on AMD MI355X (gfx950).
 *
 * The operation (paper, Section 2.1 "Distance transforms"; kernels in Section
 * 2.3.2 "Distance-transform kernels"): for each of `batch` independent
 * samples with spatial extents shape[0..ndim), every element x receives the
 * distance to the nearest background (zero) element y of its sample,
 *
 *     D(x) = sqrt( min over background y of  sum_a s_a^2 (x_a - y_a)^2 ),
 *
 * where s is the optional per-axis sampling (paper, Section 2.2.1: the
 * distance transforms take SciPy's `sampling`, `return_distances` and
 * `return_indices` arguments), and optionally the coordinates of that y.
 * Inputs shaped (B, C, spatial...) pass batch = B * C (Section 2.3.2: the
 * passes run over B*C*n^(d-1) independent lines).
 *
 * Conventions shared by every entry point:
 *   - Layout: C order.  in_u8 is [batch][shape[0]]...[shape[ndim-1]] bytes,
 *     nonzero = foreground, zero = background.  Distance-like outputs have
 *     the same layout; out_idx is [batch][ndim][shape...] int32, so each
 *     sample's block matches SciPy's (ndim, *shape) index array.
 *   - Memory: in_u8, out_* are DEVICE pointers owned by the caller; shape
 *     and sampling are HOST pointers read during the call only.  The library
 *     allocates no device memory; intermediate results live in the output
 *     buffers, which are overwritten in full (tm_edt_ws also uses the
 *     caller's workspace).
 *   - Streams: all work is enqueued on `stream` (0 = the null stream) of the
 *     current device and the call returns without waiting for it.  Results
 *     are valid once that stream has been synchronised.  Calls are reentrant;
 *     calls on different streams must not share output buffers.
 *   - Ties: the returned element is the nearest background element with the
 *     smallest row-major flat index (the paper asks only for a genuine
 *     nearest background element, Section 2.4).
 *   - No background: a sample with no zero is measured against the virtual
 *     element (-1, 0, ..., 0), which is also the index reported (paper,
 *     Section 2.3.2: SciPy's virtual out-of-bounds convention).
 *   - Errors: every function returns a tm_status.  Arguments are validated on
 *     the host before any HIP call; a rejected call enqueues nothing.  Nothing
 *     throws or aborts across this interface.
 */
#ifndef TM_EDT_H
#define TM_EDT_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TM_OK = 0,
    TM_ERR_NDIM = -1,        /* ndim outside [1, 8] (paper Section 2.2.1 caps the rank at 8) */
    TM_ERR_SHAPE = -2,       /* shape is NULL or an extent is < 1 */
    TM_ERR_BATCH = -3,       /* batch < 1 */
    TM_ERR_NULL = -4,        /* in_u8 is NULL */
    TM_ERR_NO_OUTPUT = -5,   /* every output pointer is NULL */
    TM_ERR_SAMPLING = -6,    /* a sampling entry is not finite or not > 0 */
    TM_ERR_TOO_LARGE = -7,   /* >= 2^31 elements per sample, batch * elements overflows,
                                or (tm_edt_sq, tm_edt_signed, tm_dt_bf) squared distances
                                may exceed int32 */
    TM_ERR_ALIAS = -8,       /* two of the buffers overlap */
    TM_ERR_UNSUPPORTED = -9, /* a line is longer than the signed or chessboard kernels hold */
    TM_ERR_HIP = -10,        /* the HIP runtime reported an error while enqueuing */
    TM_ERR_METRIC = -11,     /* metric is not one of tm_metric */
    TM_ERR_DTYPE = -12,      /* dtype is not one of tm_dtype */
    TM_ERR_WORKSPACE = -13   /* workspace not 4-byte aligned, or (tm_edt_noalloc) the request's
                                dispatch order needs more than the static workspace holds */
} tm_status;

/*
 * tm_edt -- distances and/or nearest-background indices.
 *
 *   sampling  NULL, or ndim spacings (all finite and > 0).  NULL or all 1.0
 *             runs the exact integer path (squared distances are exact
 *             integers, of any size the shape allows; out_dist is the
 *             correctly rounded float sqrt).  Other spacings run with float32
 *             storage and double breakpoint tests; distances then agree with
 *             an exact evaluation to ~1e-6 relative.
 * Lines of any length along any axis (paper, Section 2.3.2: lines longer
 * than on-chip memory keep their envelope in device memory; here it lives
 * inside the line's own output storage, so nothing is allocated).
 *   out_dist  NULL, or [batch][shape...] float32 distances.
 *   out_idx   NULL, or [batch][ndim][shape...] int32 coordinates of the
 *             nearest background element: with unit sampling the one with
 *             the smallest row-major flat index among equally near ones,
 *             otherwise one of the nearest (paper, Section 2.4: a genuine
 *             nearest element); (-1, 0, ..., 0) for a sample without any.
 * At least one of out_dist and out_idx must be non-NULL.
 */
int tm_edt(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
           const double *sampling, float *out_dist, int32_t *out_idx,
           hipStream_t stream);

/*
 * tm_edt_ws -- tm_edt with a caller-owned device workspace in which the
 * library may keep a dispatch order for one of its passes.
 *
 * The strided passes search each line as far as each element's final
 * distance (paper, Section 2.3.2), so on masks with large foreground
 * regions some groups of lines carry several times the mean work; run last,
 * they set the end of the pass.  With a workspace, a 2-D distance request
 * (unit sampling, no indices) whose column pass runs at least 1024
 * workgroups of 16 columns (rows of at most 512) or of 8 columns (longer
 * rows, ordered in units of four such workgroups) has its row pass estimate
 * each group's work, a one-workgroup kernel order the groups heaviest first,
 * and the column pass dispatch them in that order.  Results are identical to tm_edt's, bit for bit: the order
 * decides only when each group runs.
 *
 *   workspace        NULL, or a DEVICE pointer, 4-byte aligned, owned by the
 *                    caller and not overlapping the input or outputs.
 *   workspace_bytes  its size.  tm_edt_workspace_size() gives the bytes a
 *                    request uses (8 per ordered group of 16 or 32 columns,
 *                    0 when it has no ordered pass); with fewer, or a NULL workspace, the
 *                    call runs exactly as tm_edt.
 * The workspace is read and written on `stream`.  A call that uses it leaves
 * its first half (per-group counters) at zero for the next call; whatever
 * the workspace holds before a call can change only the order, never a
 * result, so it needs no initialisation (zero-filled memory gives the best
 * first order).  Calls that can run at the same time must not share a workspace.
 * Other arguments and errors as tm_edt, plus TM_ERR_WORKSPACE for a
 * misaligned workspace and TM_ERR_ALIAS for one that overlaps a buffer.
 */
int tm_edt_ws(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
              const double *sampling, float *out_dist, int32_t *out_idx, void *workspace,
              size_t workspace_bytes, hipStream_t stream);

/*
 * tm_edt_workspace_size -- bytes of workspace tm_edt_ws uses for a request
 * with these shapes and sampling, with (with_indices != 0) or without index
 * output: 8 per ordered group of 16 or 32 columns for the requests it
 * orders (at most 16384 groups), else 0 (also for arguments tm_edt would
 * reject).  Host-only; no HIP call.  The actual
 * call also needs the input and output pointers 16-byte aligned to use it.
 */
size_t tm_edt_workspace_size(int ndim, const int64_t *shape, int64_t batch, const double *sampling,
                             int with_indices);

/*
 * tm_edt_noalloc -- tm_edt_ws for callers that cannot allocate device
 * memory or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  It allocates nothing: its
 * workspace is a 64 KiB array in the library's own device memory, one per
 * device (each device the library runs on holds it until the process ends),
 * whose address is looked up on the first call on each device.  Requests
 * whose dispatch order needs more (tm_edt_workspace_size() above 65536
 * bytes: more than 8192 ordered groups) are refused with
 * TM_ERR_WORKSPACE before anything is enqueued; requests that need none run
 * as tm_edt.  Every call on a device shares that device's array and leaves
 * its counters at zero: calls on one device that overlap in time (on
 * different streams or threads) race for it.  Results equal tm_edt_ws's.
 * Arguments and other errors as tm_edt.
 */
int tm_edt_noalloc(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
                   const double *sampling, float *out_dist, int32_t *out_idx, hipStream_t stream);

/*
 * tm_edt_sq -- exact integer squared distances (unit sampling).
 *
 *   out_sq    NULL, or [batch][shape...] int32 squared distances.
 *   out_idx   NULL, or [batch][ndim][shape...] int32 coordinates.
 * At least one must be non-NULL.  The sum of squared extents must stay below
 * 2^31 (TM_ERR_TOO_LARGE otherwise).
 */
int tm_edt_sq(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
              int32_t *out_sq, int32_t *out_idx, hipStream_t stream);

/* Static English text for a tm_status value (never NULL). */
const char *tm_strerror(int status);

/*
 * Kernel timing for measurement tools (not needed for computing).
 *
 * tm_prof_enable(n) with n > 0 makes subsequent tm_edt / tm_edt_sq calls
 * from any thread bracket each kernel they launch with a pair of HIP events
 * on the call's stream, for up to n kernels (later kernels go untimed);
 * n = 0 disables timing and releases the events.  tm_prof_count() returns
 * how many kernels were bracketed since enabling; after synchronising the
 * stream, tm_prof_read(i, &name, &ms) returns kernel i's static name and its
 * event-to-event time in milliseconds.  Returns TM_OK, TM_ERR_HIP, or
 * TM_ERR_SHAPE for an index out of range.  Not reentrant with itself.
 */
int tm_prof_enable(int max_kernels);
int tm_prof_count(void);
int tm_prof_read(int i, const char **name, float *ms);
/* Launch shape of timed kernel i: info[0..5] = workgroups, threads per
 * workgroup, dynamic LDS bytes, static LDS bytes, registers per thread and
 * private (scratch) bytes per thread as the HIP runtime reports them (-1 if
 * it cannot).  Returns TM_OK or TM_ERR_SHAPE. */
int tm_prof_launch(int i, int64_t *info);

/* Metrics of the brute-force transform (paper, Section 2.3.2). */
typedef enum {
    TM_METRIC_EUCLIDEAN = 0,   /* sqrt( sum_a (s_a (x_a - y_a))^2 ) */
    TM_METRIC_TAXICAB = 1,     /* sum_a s_a |x_a - y_a| */
    TM_METRIC_CHESSBOARD = 2   /* max_a s_a |x_a - y_a| */
} tm_metric;

/*
 * tm_dt_bf -- brute-force distance transform (paper, Section 2.3.2: the
 * transform that checks the separable ones, templated over metric and rank,
 * and the only route to anisotropic taxicab and chessboard distances).
 *
 * For every element, the nearest background element of its sample under
 * `metric`, found by visiting every background element: O(elements x
 * background elements) per sample, meant for moderate sizes.  out_dist (may
 * be NULL) receives the distance as float32 (euclidean: the correctly
 * rounded square root of the exact squared distance under unit sampling);
 * out_idx (may be NULL) the coordinates, [batch][ndim][shape...].  sampling
 * as for tm_edt (NULL = all ones, exact integer arithmetic; otherwise float).
 * Ties, the virtual element and the other conventions are those above.
 * Errors: as tm_edt, plus TM_ERR_METRIC for an unknown metric.
 */
int tm_dt_bf(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch, int metric,
             const double *sampling, float *out_dist, int32_t *out_idx, hipStream_t stream);

/*
 * tm_edt_signed -- signed Euclidean distance transform, EDT(M) - EDT(not M)
 * (paper, Sections 1 and 2.3.2: the distance field behind boundary-aware
 * losses, which recompute it every training step).
 *
 * For every element of each sample: on foreground (nonzero) elements the
 * distance to the nearest background element, positive; on background
 * elements minus the distance to the nearest foreground element.  Each term
 * follows tm_edt, so a sample holding one class only measures from the
 * virtual element (-1, 0, ..., 0) with that class's sign.  No element is
 * zero.  Unit sampling; float32 results, each the correctly rounded square
 * root of the exact integer squared distance with its sign.  The mask is
 * read once: in every pass an element's own class offers the values found so
 * far and the other class offers sites.  Rank-3 inputs of 128 x 128 planes
 * with an axis-0 extent up to 128 run axis 0 first (class and distance to
 * the other class as one byte per element, kept inside out_dist) and then
 * one workgroup per plane; other shapes carry one field (+F on foreground,
 * -F on background) through whole-line passes.  in_u8, ndim, shape, batch as
 * for tm_edt; out_dist: device
 * float32 [batch][shape...], written completely.  Errors: as tm_edt (no
 * sampling argument), and TM_ERR_UNSUPPORTED for lines longer than about
 * 40 700 elements along an axis other than the last (one whole 32-bit line
 * per workgroup in LDS; squared distances in int32 already cap the extents
 * at 46 340).
 */
int tm_edt_signed(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
                  float *out_dist, hipStream_t stream);

/*
 * tm_cdt -- chamfer distance transform (paper, Section 2.3.2 and Table 1:
 * the taxicab and chessboard transforms, with no sampling argument).
 *
 * For every element of each sample, the distance to the nearest background
 * element under `metric` (TM_METRIC_TAXICAB: sum of |x_a - y_a|;
 * TM_METRIC_CHESSBOARD: max of |x_a - y_a|), on the unit grid.  This is
 * what a chamfer sweep with unit weights over the face neighbours (taxicab)
 * or all 3^ndim - 1 neighbours (chessboard) computes, and the result is
 * exact in int32.  A sample with no background gets -1 everywhere (nothing
 * is reachable).  in_u8, ndim, shape, batch as for tm_edt.  out_dist:
 * device int32 [batch][shape...], written completely, not aliasing in_u8.
 * Errors: as tm_edt_sq (TM_ERR_NO_OUTPUT for a NULL out_dist), plus
 * TM_ERR_METRIC for TM_METRIC_EUCLIDEAN or an unknown metric.  Taxicab
 * lines of any length are taken; chessboard lines along an axis other than
 * the last are held whole in LDS, which takes up to about 81 400 elements
 * while every distance fits 16 bits and about 40 700 otherwise: longer ones
 * give TM_ERR_UNSUPPORTED.
 */
int tm_cdt(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch, int metric,
           int32_t *out_dist, hipStream_t stream);

/*
 * tm_cdt_ws -- tm_cdt with a caller-owned device workspace in which a 2-D
 * chessboard request's column pass (at least 1024 workgroups of 8 columns,
 * ordered in units of four of them) keeps a heaviest-first dispatch order, as
 * tm_edt_ws does for the exact transform; results are identical to tm_cdt's.
 * Taxicab whole-line passes do the same work on every group and take no
 * workspace (size 0).
 * workspace and workspace_bytes as for tm_edt_ws; tm_cdt_workspace_size()
 * gives the bytes a request uses (8 per unit of 32 columns, or 0; host only).
 * Errors: as tm_cdt, plus TM_ERR_WORKSPACE and TM_ERR_ALIAS as for tm_edt_ws.
 */
int tm_cdt_ws(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch, int metric,
              int32_t *out_dist, void *workspace, size_t workspace_bytes, hipStream_t stream);
size_t tm_cdt_workspace_size(int ndim, const int64_t *shape, int64_t batch, int metric);

/* Element types the foreground predicate reads. */
typedef enum {
    TM_DTYPE_U8 = 0,     /* 1-byte integers: uint8, int8, bool */
    TM_DTYPE_I16 = 1,    /* 2-byte integers */
    TM_DTYPE_I32 = 2,    /* 4-byte integers */
    TM_DTYPE_I64 = 3,    /* 8-byte integers */
    TM_DTYPE_F16 = 4,    /* IEEE binary16 */
    TM_DTYPE_BF16 = 5,   /* bfloat16 */
    TM_DTYPE_F32 = 6,    /* IEEE binary32 */
    TM_DTYPE_F64 = 7,    /* IEEE binary64 */
    TM_DTYPE_F8 = 8      /* 1-byte floats (E4M3, E5M2): the top bit is the sign */
} tm_dtype;

/*
 * tm_mask_nonzero -- the byte mask the transforms read, from an input of any
 * element type and any layout (paper, Section 2.2.1: the operators accept
 * what their SciPy counterparts accept, and SciPy counts every nonzero
 * element as foreground, NaN included).
 *
 *   in        DEVICE pointer to the first element of a strided view.
 *   dtype     one of tm_dtype.  Integers are foreground when nonzero;
 *             floating-point values when any bit other than the sign is set,
 *             so +0 and -0 are background and NaN, infinities and subnormals
 *             are foreground.  The test is on bit patterns (no arithmetic).
 *   ndim      dimensions of the view, 1 to 16; shape: HOST pointer to the
 *             extents (each >= 1), outermost first.
 *   strides   HOST pointer to ndim strides in BYTES (each >= 0), or NULL for
 *             a C-contiguous view.
 *   out_u8    DEVICE pointer to prod(shape) bytes, written C-contiguous with
 *             1 for foreground and 0 for background; owned by the caller and
 *             not overlapping the input's footprint.
 * Enqueued on `stream` like the transforms; allocates nothing.  Errors:
 * TM_ERR_NDIM, TM_ERR_SHAPE (NULL shape, an extent < 1 or a negative
 * stride), TM_ERR_NULL (in), TM_ERR_NO_OUTPUT (out_u8), TM_ERR_DTYPE,
 * TM_ERR_TOO_LARGE (2^32 elements or more), TM_ERR_ALIAS, TM_ERR_HIP.
 */
int tm_mask_nonzero(const void *in, int dtype, int ndim, const int64_t *shape,
                    const int64_t *strides, uint8_t *out_u8, hipStream_t stream);

/*
 * tm_selftest_host -- checks the host-side planning arithmetic (the
 * division-by-invariant-integer constants the kernels use to split flat
 * indices) without touching any GPU.  Returns TM_OK or a negative count of
 * failures.
 */
int tm_selftest_host(void);

#ifdef __cplusplus
}
#endif

#endif /* TM_EDT_H */
