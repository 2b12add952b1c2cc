// edt_host.hip -- C-ABI of the MI355X exact Euclidean distance transform:
// argument validation, pass planning and kernel launches (declared in
// include/tm_edt.h).
//
// Pass order (paper, Section 2.3.2: one 1-D pass per axis): the contiguous
// last axis first, as a nearest-zero scan of the mask; then every strided
// axis down to axis 0 as an in-place exact pass; the last pass also writes
// the final outputs (square root, virtual background element, coordinates).
// Running axis 0 last makes the reported index the nearest background
// element with the smallest row-major flat index.  Sampled rank-3 requests
// on the index carrier may take their two strided axes in the other order
// (any nearest element is correct there), and distance-only rank-3 requests
// on 128 x 128 planes run axis 0 first (plane order).
//
// Two carriers: without indices the squared distance itself is carried in
// the distance (or squared-distance) output; with indices the flat index of
// the nearest background element is carried in slice 0 of the index output
// and distances are recomputed from it.

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <array>
#include <atomic>
#include <cmath>
#include <mutex>
#include <vector>

#include "../../include/tm_edt.h"
#include "edt_common.h"
#include "edt_bf.h"
#include "edt_cdt.h"
#include "edt_lsearch.h"
#include "edt_l1scan.h"
#include "edt_fh.h"
#include "edt_tidx.h"
#include "edt_scan.h"
#include "edt_col.h"
#include "edt_small.h"
#include "edt_mask.h"
#include "edt_long.h"
#include "edt_plane.h"
#include "edt_lpair.h"
#include "edt_order.h"

using namespace tmedt;

namespace {

// ---------------------------------------------------------------------------
// Kernel timing (measurement tools only).
// ---------------------------------------------------------------------------
struct Prof {
    std::mutex mu;
    int cap = 0;
    std::atomic<int> next{0};
    std::vector<hipEvent_t> start, stop;
    std::vector<const char *> names;
    // per launch: workgroups, threads per workgroup, dynamic LDS bytes,
    // static LDS bytes, registers per thread, private (scratch) bytes per thread
    std::vector<std::array<int64_t, 6>> info;
};
Prof &prof() {
    static Prof p;
    return p;
}

// A slot for one timed launch (-1: not timing); the launch itself records
// the slot's start and stop events around the kernel (hipExtLaunchKernelGGL),
// so the interval is the kernel's own, without the queue's gaps.
int prof_begin(const char *name) {
    Prof &p = prof();
    if (p.cap <= 0) return -1;
    int slot = p.next.fetch_add(1);
    if (slot >= p.cap) return -1;
    p.names[slot] = name;
    return slot;
}

// ---------------------------------------------------------------------------
// Launch helpers.
// ---------------------------------------------------------------------------
template <typename K>
hipError_t allow_lds(K kernel, size_t bytes) {
    if (bytes <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, int(bytes));
}

template <typename K, typename Args>
int launch(const char *name, K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s,
           const Args &args) {
    if (allow_lds(kernel, lds) != hipSuccess) return TM_ERR_HIP;
    int slot = prof_begin(name);
    if (slot >= 0) {
        hipFuncAttributes fa{};
        const bool ok = hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(kernel)) == hipSuccess;
        prof().info[slot] = {int64_t(grid.x) * grid.y * grid.z, int64_t(block.x) * block.y * block.z,
                             int64_t(lds), ok ? int64_t(fa.sharedSizeBytes) : -1,
                             ok ? int64_t(fa.numRegs) : -1, ok ? int64_t(fa.localSizeBytes) : -1};
    }
    if (slot >= 0)
        hipExtLaunchKernelGGL(kernel, grid, block, uint32_t(lds), s, prof().start[slot], prof().stop[slot], 0u, args);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, s, args);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? TM_OK : TM_ERR_HIP;
}

int bits_for(uint64_t x) {
    int b = 0;
    while (b < 64 && (x >> b) != 0) ++b;
    return b;
}

bool overlaps(const void *a, uint64_t na, const void *b, uint64_t nb) {
    if (!a || !b || na == 0 || nb == 0) return false;
    uintptr_t a0 = uintptr_t(a), b0 = uintptr_t(b);
    return a0 < b0 + nb && b0 < a0 + na;
}

// Lanes per workgroup whose envelope stacks of n entries x eb bytes fit LDS.
uint32_t lanes_for(uint32_t n, uint32_t eb) {
    for (uint32_t l = kWave; l >= 1; l >>= 1)
        if (uint64_t(n) * l * eb <= kLdsBytes) return l;
    return 0;
}

// Unit sampling: int32 suffices for every breakpoint product of a pass over
// lines of length n when the carried squared distance is at most fmax.
bool int32_safe(uint64_t fmax, uint64_t n) {
    const uint64_t lim = (uint64_t(1) << 31) - 1;
    uint64_t key = fmax + (n - 1) * (n - 1);
    uint64_t den = 2 * (n - 1);
    if (key >= lim) return false;
    if (den && key > lim / den) return false;
    if ((n - 1) * den >= lim) return false;
    return true;
}

// ... and every operand also fits in a signed 24-bit multiply.
bool int24_safe(uint64_t fmax, uint64_t n) {
    const uint64_t lim24 = (uint64_t(1) << 23) - 1;
    return int32_safe(fmax, n) && fmax + (n - 1) * (n - 1) < lim24 && 2 * (n - 1) < lim24;
}

struct Request {
    const uint8_t *in;
    int ndim;
    uint32_t shape[kMaxDim];
    uint64_t batch;
    bool unit;
    double w[kMaxDim];
    float *dist;
    int32_t *sq;
    int32_t *idx;
    hipStream_t stream;
    int metric;      // kL2 (exact transform) or kL1 / kLinf (chamfer; output in sq)
    bool sgn;        // signed transform EDT(M) - EDT(not M) (kL2, unit, output in dist)
    bool big;        // unit sampling with squared distances that may pass int32
    uint32_t *ws;    // caller workspace for dispatch orders (may be null), 4-byte aligned
    uint64_t ws_bytes;
};

int validate(const uint8_t *in, int ndim, const int64_t *shape, int64_t batch,
             const double *sampling, const void *o1, const void *o2, const void *o3,
             Request &r, bool squared = true) {
    if (ndim < 1 || ndim > kMaxDim) return TM_ERR_NDIM;
    if (!shape) return TM_ERR_SHAPE;
    for (int a = 0; a < ndim; ++a)
        if (shape[a] < 1) return TM_ERR_SHAPE;
    if (batch < 1) return TM_ERR_BATCH;
    if (!in) return TM_ERR_NULL;
    if (!o1 && !o2 && !o3) return TM_ERR_NO_OUTPUT;
    r.unit = true;
    for (int a = 0; a < ndim; ++a) {
        double s = sampling ? sampling[a] : 1.0;
        if (!(s > 0.0) || !std::isfinite(s)) return TM_ERR_SAMPLING;
        if (s != 1.0) r.unit = false;
        r.w[a] = s * s;
    }
    uint64_t vox = 1, sumsq = 0;
    for (int a = 0; a < ndim; ++a) {
        if (uint64_t(shape[a]) >= (uint64_t(1) << 31)) return TM_ERR_TOO_LARGE;
        vox *= uint64_t(shape[a]);
        if (vox >= (uint64_t(1) << 31)) return TM_ERR_TOO_LARGE;
        sumsq += uint64_t(shape[a]) * uint64_t(shape[a]);
        r.shape[a] = uint32_t(shape[a]);
    }
    if (uint64_t(batch) >= (uint64_t(1) << 32) / vox) return TM_ERR_TOO_LARGE;
    r.big = r.unit && sumsq >= (uint64_t(1) << 31) - 1;
    if (squared && r.big) return TM_ERR_TOO_LARGE;
    r.in = in;
    r.ndim = ndim;
    r.batch = uint64_t(batch);
    return TM_OK;
}

// The paired tile takes 128 lines per workgroup: below this many lines in a
// pass it leaves most of the chip idle, and the whole-line search (8 lines
// per workgroup) is faster.
constexpr uint64_t kPairMinLines = 256 * kPairLines;

// Workgroups of 16 lines below which the packed line pass leaves compute
// units idle (two workgroups of 16 waves fill one): fewer lines take the
// whole-line search with 8 lines per workgroup.
constexpr uint64_t kLpMinGroups = 512;

// Plan of one strided pass.
struct FhPlan {
    uint32_t lpw;
    bool pack;
    int acc;  // 0 int32 with 24-bit multiplies, 1 int32, 2 int64, 3 double
    size_t lds;
    bool tiled16;    // paired 16-bit tile with guard rows (k_tile_pair)
    bool from_mask;  // tiled16 on axis ndim-2, computing the last-axis pass itself
    bool tidx;       // tiled pass on the index carrier (k_tile_idx)
    int ls_lpw;      // whole lines in LDS, windowed search (k_line_search): lines per workgroup (8, 4, 2, 1), 0 = not
    bool ls_w16;     //   with a 16-bit tile
    uint32_t rbits;  // tidx, unit sampling: bits of the row in a key
    bool lng;        // index carrier, envelope in the line's own storage (k_fh_long)
    bool l1long;     // taxicab, two running minima in place (k_cdt_l1_long)
    bool l1scan;     // taxicab, whole lines in LDS, prefix and suffix minima (k_cdt_l1_scan)
    bool lp16;       // 16 lines per workgroup, two per packed 16-bit word (k_line_pair16)
};

// Whole-line windowed search: 8 lines per workgroup (a wave covers 8 rows
// of 8 lines, whose search lengths vary less than those of 64 lines of one
// row), or fewer (down to min_lpw) when the tile of 8 does not fit LDS.
bool plan_line_search(FhPlan &p, uint32_t n, uint64_t total, bool w16, int min_lpw = 4) {
    const int tb = w16 ? 2 : 4;
    const uint64_t lines = total / n;
    int lpw = 0;
    for (int c = 8; c >= min_lpw && !lpw; c /= 2)
        if (line_search_lds(n, c, tb) + 1024 <= kLdsBytes) lpw = c;
    if (!lpw || lines + uint64_t(lpw) >= (uint64_t(1) << 32) || (lines + lpw - 1) / lpw >= (uint64_t(1) << 31))
        return false;
    p.ls_lpw = lpw;
    p.ls_w16 = w16;
    p.lds = line_search_lds(n, lpw, tb);
    return true;
}

// Multiplier of the plane permutation of the plane kernels (workgroup b
// takes plane b * m mod planes): the first of a few primes that does not
// divide the plane count, so m is coprime to it.
uint32_t plane_stride(uint32_t planes) {
    static const uint32_t primes[] = {397, 401, 409, 419, 421, 431, 433, 439};
    for (uint32_t m : primes)
        if (planes % m != 0) return m % planes == 0 ? 1u : m % planes;
    return 1;
}

// Plane order for distance outputs of unit-sampled rank-3 inputs whose last
// two extents are both 128, or both 64 with an even number of planes per
// sample: the axis-0 nearest-zero scan first (k_col_scan, straight from the
// mask), then one workgroup per 128 x 128 plane (k_plane_edt) or per two
// 64 x 64 planes (k_tile_pair with PLANE) for the last two axes.  Axis-0
// distances reach 128 x 128 planes as bytes, 64 x 64 planes as 16-bit
// squares.  (Rank 4 would put the middle axes between the two kernels; on a
// sparse 4-D input that order measured slower than the last-axis-first one,
// whose early passes see fewer empty lines.)  The order of
// the axes does not change any distance (each pass is an exact minimum), and
// no indices are produced on this path.  Returns kNotPlane, before any
// launch, when the input does not qualify.
constexpr int kNotPlane = 1;

// Wavefronts below which the last-axis word scan takes 32-position words
// (one per SIMD).  Measured: 8 x 256^2 6.8 against 8.2 us; at 2048 wavefronts
// (32 x 512^2, 8 x 1024^2) 64-position words stay faster with the int32 field
// (16.7 against 18.0 us).  A unit or chamfer field (written packed to 16 bits
// where the next pass takes it) of rows up to 512 wide takes 32-position
// words below kWord32WavesField: 32 x 512^2 with the cost estimate 14.1 ->
// 11.8 us (HIP events; 8 x 1024^2 unchanged, 15.5 against 15.8 us).
constexpr uint64_t kWord32Waves = 1024;
constexpr uint64_t kWord32WavesField = 4096;

int run_plane(Request &r, uint64_t total, uint64_t vox) {
    const int nd = r.ndim;
    const uint32_t P = r.shape[nd - 1];
    if (nd != 3 || (P != 128 && P != 64) || r.shape[nd - 2] != P || r.shape[0] > 128) return kNotPlane;
    // 64 x 64 planes: a workgroup takes two planes of one sample
    if (P == 64 && (vox / (64 * 64)) % 2 != 0) return kNotPlane;
    int32_t *buf = r.dist ? reinterpret_cast<int32_t *>(r.dist) : r.sq;
    if (uintptr_t(r.in) % 2 != 0 || uintptr_t(buf) % 16 != 0) return kNotPlane;
    const uint64_t S = vox / r.shape[0];                 // a multiple of 128 * 128
    // the column scan addresses a wave's 16 rows with 32-bit offsets 4 * S * j
    if (S >= (uint64_t(1) << 25)) return kNotPlane;
    // Both searches keep the field below "no site" (0xffff): the largest
    // value before a search plus the square of the farthest row it reads,
    // guard rows included.
    const uint64_t fmax = uint64_t(r.shape[0] - 1) * (r.shape[0] - 1);
    const uint64_t reach = uint64_t(P + kGuard16) * (P + kGuard16);
    if (fmax + reach >= uint64_t(kNone16) || fmax + uint64_t(P - 1) * (P - 1) + reach >= uint64_t(kNone16))
        return kNotPlane;

    ColArgs c{};
    c.mask = r.in;
    c.buf = buf;
    c.n0 = r.shape[0];
    c.S = uint32_t(S);
    c.blocks = uint32_t(S / kColBlock);
    c.div_blocks = Div32::make(c.blocks);
    // A 128 x 128 plane pass reads the axis-0 distances as bytes.
    const bool bytes = P == 128;
    const dim3 cgrid(uint32_t(total / (uint64_t(c.n0) * kColBlock))), cblock(kWave * kColWaves);
    int rc = bytes ? launch("col_scan.o8", k_col_scan<true>, cgrid, cblock, 0, r.stream, c)
                   : launch("col_scan.o16", k_col_scan<false>, cgrid, cblock, 0, r.stream, c);
    if (rc != TM_OK) return rc;

    if (P == 64) {
        PairArgs tg{};
        tg.buf = buf;
        tg.total = uint32_t(total);
        tg.dist = r.dist;
        tg.sq = r.sq;
        tg.ndim = nd;
        tg.vox = uint32_t(vox);
        for (int b = 0; b < nd; ++b) {
            tg.shape[b] = r.shape[b];
            tg.wall[b] = 1.0;
        }
        tg.n = P;
        tg.inner = P;
        tg.div_inner = Div32::make(P);
        tg.lines = uint32_t(total / P);
        tg.out_seg = 0;
        tg.in_seg = 1;
        const size_t lds = size_t(P + 2 * kGuard16) * kRowW * 4;
        return launch("plane_final.i16", k_tile_pair<true, false, 8, kL2, 64>, dim3(uint32_t(total / P / kPairLines)),
                      dim3(kWave * kPairWaves), lds, r.stream, tg);
    }
    PlaneEdtArgs pe{};
    pe.bytes = reinterpret_cast<const uint8_t *>(buf);
    pe.dist = r.dist;
    pe.sq = r.sq;
    pe.n0 = r.shape[0];
    pe.planes = uint32_t(total / (kPsN * kPsN));
    pe.mult = plane_stride(pe.planes);
    constexpr int kEdtLut = 1024;
    return launch("plane_final.i8", k_plane_edt<kEdtLut>, dim3(uint32_t(total / (kPsN * kPsN))), dim3(kPsThreads),
                  2 * kPsTile + 4 * kEdtLut, r.stream, pe);
}

// Plane order for the signed transform of rank-3 inputs of 128 x 128 planes
// (n0 <= 128): the axis-0 scan of both classes (k_col_scan_signed, straight
// from the mask), then one workgroup per plane for the last two axes
// (k_plane_signed).  Returns kNotPlane, before any launch, when the input
// does not qualify.
int run_plane_signed(Request &r, uint64_t total, uint64_t vox) {
    if (r.ndim != 3 || r.shape[1] != uint32_t(kPsN) || r.shape[2] != uint32_t(kPsN) || r.shape[0] > 128)
        return kNotPlane;
    if (uintptr_t(r.in) % 2 != 0 || uintptr_t(r.dist) % 16 != 0) return kNotPlane;
    ColArgs c{};
    c.mask = r.in;
    c.buf = reinterpret_cast<int32_t *>(r.dist);
    c.n0 = r.shape[0];
    c.S = uint32_t(vox / r.shape[0]);
    c.blocks = uint32_t(c.S / kColBlock);
    c.div_blocks = Div32::make(c.blocks);
    const dim3 cgrid(uint32_t(total / (uint64_t(c.n0) * kColBlock))), cblock(kWave * kColWaves);
    int rc = launch("col_scan_signed", k_col_scan_signed, cgrid, cblock, 0, r.stream, c);
    if (rc != TM_OK) return rc;
    PlaneSignedArgs ps{};
    ps.out = r.dist;
    ps.n0 = r.shape[0];
    return launch("plane_signed_final", k_plane_signed, dim3(uint32_t(total / (kPsN * kPsN))), dim3(kPsThreads), kPsLds,
                  r.stream, ps);
}

// Plan of every strided pass, axis nd-2 down to 0, before anything is
// launched.  index_path: the index carrier (flat index of the nearest
// background element); otherwise the field carrier (unit squared distances).
// Returns TM_ERR_UNSUPPORTED when a pass has no kernel for its lines.
int plan_passes(const Request &r, uint64_t total, bool index_path, FhPlan *fh) {
    const int nd = r.ndim;
    for (int a = 0; a < kMaxDim; ++a) fh[a] = FhPlan{};
    for (int a = nd - 2; a >= 0; --a) {
        const uint32_t n = r.shape[a];
        uint64_t fmax = 0;
        for (int b = a + 1; b < nd; ++b) fmax += uint64_t(r.shape[b] - 1) * (r.shape[b] - 1);
        FhPlan &p = fh[a];
        if (r.sgn) {
            // signed transform: whole-line search over the signed field
            if (!plan_line_search(p, n, total, false, 1)) return TM_ERR_UNSUPPORTED;
            continue;
        }
        if (r.metric != kL2) {
            // Chamfer transforms: the paired tile with the metric's largest
            // value plus any in-line distance below "no site", else whole
            // lines staged in LDS.
            uint64_t vmax = 0;
            for (int b = a + 1; b < nd; ++b)
                vmax = r.metric == kL1 ? vmax + (r.shape[b] - 1) : std::max<uint64_t>(vmax, r.shape[b] - 1);
            const size_t tp = size_t(n + 2 * kGuard16) * kRowW * 4;
            uint64_t inner = 1;
            for (int b = a + 1; b < nd; ++b) inner *= r.shape[b];
            const bool offsets_fit =
                (uint64_t(n) * inner * 2 + uint64_t(n) * kPairLines) * 4 < (uint64_t(1) << 31);
            if (n <= 256 && vmax + n + 4 < uint64_t(kNone16) && tp + 1024 <= kLdsBytes && offsets_fit &&
                total / n + kPairLines < (uint64_t(1) << 32) && total / n >= kPairMinLines) {
                p.tiled16 = true;
                p.lds = tp;
                const uint32_t n2 = r.shape[nd - 1];
                if (a == nd - 2 && n2 % 32 == 0 && uintptr_t(r.in) % 16 == 0) {
                    uint32_t g = kPairLines;
                    for (uint32_t x = n2; x;) {
                        const uint32_t y = g % x;
                        g = x;
                        x = y;
                    }
                    const uint64_t planes = (uint64_t(n2) - g + kPairLines - 1) / n2 + 1;
                    if (planes * (n2 / 32) * 2 <= uint64_t(kWave)) p.from_mask = true;
                }
                continue;
            }
            const uint64_t cmax = r.metric == kL1 ? vmax + n + 4 : std::max<uint64_t>(vmax, n + 4);
            // taxicab lines whose 8-line groups share rows: prefix and suffix
            // minima, no search
            const void *cfield = r.sq;
            if (r.metric == kL1 && inner % kL1Lines == 0 && n <= kL1MaxN && cmax < (uint64_t(1) << 29) &&
                l1scan_lds(n) + 1024 <= kLdsBytes && total / n / kL1Lines < (uint64_t(1) << 31) &&
                uintptr_t(cfield) % 16 == 0) {
                p.l1scan = true;
                p.lds = l1scan_lds(n);
                continue;
            }
            if (plan_line_search(p, n, total, cmax < uint64_t(kNone16), 1)) continue;
            // taxicab lines of any length: two running minima in place
            if (r.metric == kL1) {
                p.l1long = true;
                continue;
            }
            return TM_ERR_UNSUPPORTED;
        }
        p.acc = !r.unit ? 3 : int24_safe(fmax, n) ? 0 : int32_safe(fmax, n) ? 1 : 2;
        uint32_t eb;
        if (index_path) {
            p.pack = false;
            eb = 4;
        } else {
            int vbits = bits_for(n - 1);
            if (vbits < 1) vbits = 1;
            p.pack = r.unit && vbits + bits_for(fmax) <= 32;
            eb = p.pack ? 4 : 8;
        }
        p.lpw = lanes_for(n, eb);
        if (!index_path && r.unit) {
            // Paired 16-bit tile: every value plus the square of any distance
            // within the line stays below the "no site" code, the tile (with
            // guard rows) fits LDS, and byte offsets within a workgroup's
            // buffer view stay below 2^31.
            const size_t tp = size_t(n + 2 * kGuard16) * kRowW * 4;
            uint64_t inner = 1;
            for (int b = a + 1; b < nd; ++b) inner *= r.shape[b];
            const bool offsets_fit =
                (uint64_t(n) * inner * 2 + uint64_t(n) * kPairLines) * 4 < (uint64_t(1) << 31);
            if (n <= 256 && fmax + uint64_t(n + 4) * (n + 4) < uint64_t(kNone16) && tp + 1024 <= kLdsBytes &&
                total / n >= kPairMinLines &&
                offsets_fit && total / n + kPairLines < (uint64_t(1) << 32)) {
                p.tiled16 = true;
                p.lds = tp;
                // Fold the last-axis pass into this one when it comes right
                // after it, the last extent is whole 32-column mask words, and
                // the mask entries of the planes a workgroup touches fit in a
                // tile row (two words per plane and mask word).
                const uint32_t n2 = r.shape[nd - 1];
                if (a == nd - 2 && n2 % 32 == 0 && uintptr_t(r.in) % 16 == 0) {
                    uint32_t g = kPairLines;
                    for (uint32_t x = n2; x;) {
                        const uint32_t y = g % x;
                        g = x;
                        x = y;
                    }
                    const uint64_t planes = (uint64_t(n2) - g + kPairLines - 1) / n2 + 1;
                    if (planes * (n2 / 32) * 2 <= uint64_t(kWave)) p.from_mask = true;
                }
                continue;
            }
        }
        // Unit sampling without indices, lines of up to 512 rows (a multiple
        // of 16) whose 16 neighbours along the later axes are adjacent in
        // memory: 16 lines per workgroup, two per packed 16-bit word, while
        // that leaves at least two workgroups per compute unit and every
        // exact candidate stays in int32.
        if (!index_path && r.unit && n <= kLpMaxN && n % 16 == 0) {
            uint64_t inner = 1;
            for (int b = a + 1; b < nd; ++b) inner *= r.shape[b];
            const uint64_t groups = total / n / kLpLines;
            const void *field = r.dist ? static_cast<const void *>(r.dist) : static_cast<const void *>(r.sq);
            if (inner % kLpLines == 0 && groups >= kLpMinGroups && groups < (uint64_t(1) << 31) &&
                fmax + uint64_t(n - 1) * (n - 1) < uint64_t(kInfI) && uintptr_t(field) % 16 == 0) {
                p.lp16 = true;
                p.lds = lpair_lds(n);
                continue;
            }
        }
        // Otherwise, unit sampling without indices: whole lines in LDS with
        // the windowed search (32-bit tile) while they fit.
        if (!index_path && r.unit && plan_line_search(p, n, total, false)) continue;
        // Index carrier, lines up to 256 rows: tiled windowed search.  Unit
        // sampling packs (value, row) into one key below 2^31.
        if (index_path && n <= 256) {
            const size_t tb = idx_tile_lds(n, !r.unit);
            int rb = bits_for(n - 1);
            if (rb < 1) rb = 1;
            const uint64_t kv = fmax + uint64_t(n - 1) * (n - 1);
            const bool keys_fit = !r.unit || (rb < 31 && kv < (uint64_t(1) << 31) &&
                                              ((kv << rb) | uint64_t(n - 1)) < (uint64_t(1) << 31));
            if (tb + 2048 <= kLdsBytes && keys_fit && total / n + kIdxLines < (uint64_t(1) << 32)) {
                p.tidx = true;
                p.rbits = uint32_t(rb);
                p.lds = tb;
                continue;
            }
        }
        const uint64_t lines = total / n;
        if (p.lpw == 0 || (lines + p.lpw - 1) / p.lpw >= (uint64_t(1) << 31)) {
            // the field carrier has no kernel for this line; the index
            // carrier keeps the envelope in the line's own storage
            if (!index_path) return TM_ERR_UNSUPPORTED;
            p.lpw = 0;
            p.lng = true;
            continue;
        }
        p.lds = size_t(n) * p.lpw * eb;
    }
    return TM_OK;
}

// Words of the last-axis word scan: 32 positions when 64-position words
// would leave fewer than kWord32Waves wavefronts (twice the wavefronts, and so
// twice the loads and stores, in flight), else 64.
struct WordShape {
    bool w32;
    uint32_t nw;     // words per line
    uint32_t lpw;    // whole lines per wavefront
};

WordShape word_shape(uint32_t nlast, uint64_t lines, bool field) {
    const uint64_t lpw64 = kWave / (nlast / kWave);
    const uint64_t waves64 = (lines + lpw64 - 1) / lpw64;
    const bool w32 = nlast <= uint32_t(32 * kWave) &&
                     (waves64 < kWord32Waves || (field && nlast <= 512u && waves64 < kWord32WavesField));
    const uint32_t nw = nlast / (w32 ? 32 : 64);
    return {w32, nw, uint32_t(kWave) / nw};
}

// Workgroups of the column pass below which no dispatch order is kept: with
// at most two per slot of the chip (two per CU) the heaviest groups start
// early anyway, and the order's own kernel would cost more than it saves.
constexpr uint64_t kOrderMinGroups = 1024;

// The column pass whose dispatch order the workspace carries: a 2-D
// distance request whose row pass is the word scan with the unit field and
// whose column pass is ordered in groups of `width` adjacent columns
// (k_line_pair16: its workgroups' 16; k_line_search with 8 columns per
// workgroup: units of four workgroups, 32), with words per line dividing 64,
// whole workgroups of the scan inside one sample, at most 256 groups per row,
// at least kOrderMinGroups workgroups and at most kOrderMax groups.  groups =
// 0: none.  (On 3-D inputs the packed passes measured no faster in cost
// order.)
struct OrderPlan {
    uint64_t groups;
    uint32_t width;
};

OrderPlan order_groups(const Request &r, const FhPlan *fh, uint64_t total) {
    if (r.ndim != 2 || !r.unit || r.big || r.idx || r.sgn) return {0, 0};
    // k_line_search orders units of four groups of 8 lines (32 columns)
    const uint32_t width = (fh[0].lp16 && r.metric == kL2) ? uint32_t(kLpLines)
                           : (!fh[0].tiled16 && !fh[0].l1long && fh[0].ls_lpw == 8) ? 32u : 0u;
    if (!width) return {0, 0};
    const uint32_t n0 = r.shape[0], nlast = r.shape[1];
    if (nlast % kWave != 0 || nlast > uint32_t(kWave * kWave) || nlast / width > 256) return {0, 0};
    const WordShape wsh = word_shape(nlast, total / nlast, true);
    if (kWave % wsh.nw != 0 || n0 % (4 * wsh.lpw) != 0) return {0, 0};
    const uint64_t groups = total / n0 / width;
    const uint64_t workgroups = total / n0 / (width == 32 ? 8 : width);
    if (workgroups < kOrderMinGroups || workgroups % 32 != 0 || groups > kOrderMax) return {0, 0};
    return {groups, width};
}

int run(Request &r) {
    const int nd = r.ndim;
    uint64_t vox = 1;
    for (int a = 0; a < nd; ++a) vox *= r.shape[a];
    const uint64_t total = r.batch * vox;

    // Buffers must not overlap.
    const uint64_t nin = total, nf = 4 * total, ni = 4 * total * uint64_t(nd);
    if (overlaps(r.in, nin, r.dist, nf) || overlaps(r.in, nin, r.sq, nf) ||
        overlaps(r.in, nin, r.idx, ni) || overlaps(r.dist, nf, r.sq, nf) ||
        overlaps(r.dist, nf, r.idx, ni) || overlaps(r.sq, nf, r.idx, ni))
        return TM_ERR_ALIAS;
    if (r.ws && (overlaps(r.ws, r.ws_bytes, r.in, nin) || overlaps(r.ws, r.ws_bytes, r.dist, nf) ||
                 overlaps(r.ws, r.ws_bytes, r.sq, nf) || overlaps(r.ws, r.ws_bytes, r.idx, ni)))
        return TM_ERR_ALIAS;

    // Small 2-D samples (both extents at most 64): one workgroup per sample
    // runs both passes in LDS, in one launch.
    if (nd == 2 && r.unit && r.metric == kL2 && !r.sgn && r.shape[0] <= uint32_t(kSmallMax) &&
        r.shape[1] <= uint32_t(kSmallMax) && r.batch < (uint64_t(1) << 31)) {
        SmallArgs sa{};
        sa.mask = r.in;
        sa.dist = r.dist;
        sa.sq = r.sq;
        sa.idx = r.idx;
        sa.n0 = r.shape[0];
        sa.n1 = r.shape[1];
        return launch("small2d", k_small2d, dim3(uint32_t(r.batch)), dim3(kWave * kSmallWaves), 0, r.stream, sa);
    }
    if (!r.idx && r.unit && !r.big && r.metric == kL2 && !r.sgn) {
        const int rc = run_plane(r, total, vox);
        if (rc != kNotPlane) return rc;
    }
    if (r.sgn) {
        const int rc = run_plane_signed(r, total, vox);
        if (rc != kNotPlane) return rc;
    }

    // The carrier between passes.  With indices: the flat index of the
    // nearest background element, in slice 0 of out_idx.  Distances only,
    // unit sampling: the squared distance itself, in the output.  Distances
    // only otherwise (sampled, squared distances that may pass int32, or a
    // line no field kernel holds): the flat index again, inside the 32-bit
    // distance output, which the final pass overwrites with the distances.
    FhPlan fh[kMaxDim];
    bool index_path = r.idx != nullptr;
    int prc = TM_OK;
    if (!index_path && r.metric == kL2 && !r.sgn) {
        if (r.unit && !r.big) prc = plan_passes(r, total, false, fh);
        if (!r.unit || r.big || prc != TM_OK) {
            index_path = true;
            prc = plan_passes(r, total, true, fh);
        }
    } else {
        prc = plan_passes(r, total, index_path, fh);
    }
    if (prc != TM_OK) return prc;
    int32_t *const cidx = r.idx ? r.idx : r.dist ? reinterpret_cast<int32_t *>(r.dist) : r.sq;
    const uint64_t cstride = r.idx ? uint64_t(nd) * vox : vox;
    const int coords = r.idx ? 1 : 0;
    // Consecutive paired passes whose rows are whole 128-element runs hand
    // their field over in the 16-bit segment layout.
    bool out_seg[kMaxDim] = {};
    {
        bool seg_ok[kMaxDim] = {};
        for (int a = nd - 2; a >= 0; --a) {
            uint64_t inner = 1;
            for (int b = a + 1; b < nd; ++b) inner *= r.shape[b];
            seg_ok[a] = fh[a].tiled16 && inner % kPairLines == 0;
        }
        for (int a = nd - 2; a >= 1; --a) out_seg[a] = seg_ok[a] && seg_ok[a - 1];
    }
    const uint32_t nlast = r.shape[nd - 1];

    // Dispatch order of the column pass, kept in the workspace (edt_order.h).
    const OrderPlan oplan = r.ws ? order_groups(r, fh, total) : OrderPlan{0, 0};
    uint64_t order_n = oplan.groups;
    if (order_n && r.ws_bytes < order_workspace_bytes(order_n)) order_n = 0;

    int rc;
    // The row scan writes its distances packed to 16 bits, in strips of pkw
    // columns, for a first strided pass on k_line_pair16 (16) or on
    // k_line_search with 8 lines per workgroup (8): half the field's bytes
    // written and read.
    int pkw = 0;
    // ---- pass over the last axis: nearest zero in each contiguous line ----
    // (computed by the next pass itself when that one reads the mask)
    if (r.sgn) {
        SignedScanArgs s{};
        s.in = r.in;
        s.field = reinterpret_cast<int32_t *>(r.dist);
        s.dist = r.dist;
        s.n = nlast;
        s.lines = uint32_t(total / nlast);
        const dim3 grid(uint32_t((uint64_t(s.lines) + 3) / 4)), block(256);
        const bool lng = (nlast + kWave - 1) / kWave > uint32_t(kSignedRegChunks);
        if (nd == 1)
            rc = lng ? launch("scan_signed_final", k_scan_signed<true, true>, grid, block, 0, r.stream, s)
                     : launch("scan_signed_final", k_scan_signed<false, true>, grid, block, 0, r.stream, s);
        else
            rc = lng ? launch("scan_signed", k_scan_signed<true, false>, grid, block, 0, r.stream, s)
                     : launch("scan_signed", k_scan_signed<false, false>, grid, block, 0, r.stream, s);
        if (rc != TM_OK) return rc;
    } else if (!(nd >= 2 && fh[nd - 2].from_mask)) {
        ScanArgs s{};
        s.in = r.in;
        s.n = nlast;
        s.lines = uint32_t(total / nlast);
        s.lps = uint32_t(vox / nlast);
        s.div_n = Div32::make(nlast);
        s.div_lps = Div32::make(s.lps);
        s.vox = uint32_t(vox);
        s.ndim = nd;
        s.w = r.w[nd - 1];
        int mode;
        void *out;
        if (r.metric != kL2) {
            mode = kScanFieldL1;      // |d|, also the whole rank-1 chamfer result
            s.field_i = r.sq;
            out = r.sq;
        } else if (nd == 1) {
            mode = kScanFinal;
            s.dist = r.dist;
            s.sq = r.sq;
            s.idx = r.idx;
            out = nullptr;   // scalar stores: no alignment needed
        } else if (index_path) {
            mode = kScanIndex;
            s.idx = cidx;
            s.cstride = cstride;
            out = cidx;
        } else if (r.unit) {
            mode = kScanFieldInt;
            s.field_i = r.dist ? reinterpret_cast<int32_t *>(r.dist) : r.sq;
            out = s.field_i;
        } else {
            mode = kScanFieldFlt;
            s.field_f = r.dist;
            out = r.dist;
        }
        const bool word_ok = nlast % kWave == 0 && nlast <= uint32_t(kWave * kWave) &&
                             uintptr_t(r.in) % 16 == 0 && uintptr_t(out) % 16 == 0;
        if (!word_ok || (mode != kScanFieldInt && mode != kScanFieldL1)) order_n = 0;
        if (word_ok) {
            WordScanArgs ws{};
            ws.in = r.in;
            ws.n = nlast;
            ws.lines = total / nlast;
            const WordShape wsh = word_shape(nlast, ws.lines, mode == kScanFieldInt || mode == kScanFieldL1);
            const bool w32 = wsh.w32;
            ws.nw = wsh.nw;
            ws.lpw = wsh.lpw;
            ws.lps = uint32_t(vox / nlast);
            ws.vox = uint32_t(vox);
            ws.ndim = nd;
            ws.w = r.w[nd - 1];
            ws.field_i = s.field_i;
            ws.field_f = s.field_f;
            ws.idx = s.idx;
            ws.cstride = s.cstride;
            ws.dist = s.dist;
            ws.sq = s.sq;
            ws.cost = r.ws;
            ws.rows = r.shape[0];
            // packed field: the next pass takes it, and every wave's rows pair
            // up inside one block of that axis's rows
            if (nd >= 2 && wsh.lpw >= 2 && r.shape[nd - 2] % wsh.lpw == 0 && !fh[nd - 2].l1long &&
                !fh[nd - 2].tiled16) {
                const FhPlan &p1 = fh[nd - 2];
                if (mode == kScanFieldInt && p1.lp16) pkw = 16;
                else if ((mode == kScanFieldInt || mode == kScanFieldL1) && !p1.lp16 && (p1.ls_lpw == 8 || p1.l1scan))
                    pkw = 8;
            }
            ws.n1 = nd >= 2 ? r.shape[nd - 2] : 1;
            const uint64_t waves = (ws.lines + ws.lpw - 1) / ws.lpw;
            const dim3 grid(uint32_t((waves + 3) / 4)), block(256);
#define TM_WORD(M)                                                                            \
    (w32 ? launch("scan_word", k_scan_word<M, 32>, grid, block, 0, r.stream, ws)                  \
         : launch("scan_word", k_scan_word<M, 64>, grid, block, 0, r.stream, ws))
#define TM_WORD_X(NM, M, CW, PKW)                                                                          \
    (w32 ? launch(NM, k_scan_word<M, 32, CW, PKW>, grid, block, 0, r.stream, ws)                           \
         : launch(NM, k_scan_word<M, 64, CW, PKW>, grid, block, 0, r.stream, ws))
            // cost widths: 16 with k_line_pair16 (pkw 16 or none), 32 with
            // k_line_search (pkw 8 or none)
            switch (mode) {
                case kScanFieldInt:
                    if (order_n && pkw == 16) rc = TM_WORD_X("scan_word.cost.o16", kScanFieldInt, 16, 16);
                    else if (order_n && pkw == 8) rc = TM_WORD_X("scan_word.cost.o16", kScanFieldInt, 32, 8);
                    else if (order_n && oplan.width == 16) rc = TM_WORD_X("scan_word.cost", kScanFieldInt, 16, 0);
                    else if (order_n) rc = TM_WORD_X("scan_word.cost", kScanFieldInt, 32, 0);
                    else if (pkw == 16) rc = TM_WORD_X("scan_word.o16", kScanFieldInt, 0, 16);
                    else if (pkw == 8) rc = TM_WORD_X("scan_word.o16", kScanFieldInt, 0, 8);
                    else rc = TM_WORD(kScanFieldInt);
                    break;
                case kScanFieldL1:
                    if (order_n && pkw) rc = TM_WORD_X("scan_word.cost.o16", kScanFieldL1, 32, 8);
                    else if (order_n) rc = TM_WORD_X("scan_word.cost", kScanFieldL1, 32, 0);
                    else if (pkw) rc = TM_WORD_X("scan_word.o16", kScanFieldL1, 0, 8);
                    else rc = TM_WORD(kScanFieldL1);
                    break;
                case kScanFieldFlt: rc = TM_WORD(kScanFieldFlt); break;
                case kScanIndex: rc = TM_WORD(kScanIndex); break;
                default: rc = TM_WORD(kScanFinal); break;
            }
#undef TM_WORD_X
#undef TM_WORD
            if (rc == TM_OK && order_n)
                rc = launch("order", k_order, dim3(1), dim3(kOrderThreads), 0, r.stream,
                            OrderArgs{r.ws, uint32_t(order_n)});
        } else if (nlast <= uint32_t(kSpan)) {
            s.span_lines = uint32_t(kSpan) / nlast;
            const uint64_t waves = (uint64_t(s.lines) + s.span_lines - 1) / s.span_lines;
            const dim3 grid(uint32_t((waves + 3) / 4)), block(256);
            const bool vec = mode != kScanFinal && nlast % 4 == 0 && kSpan % nlast == 0 &&
                             uintptr_t(r.in) % 4 == 0 && uintptr_t(out) % 16 == 0;
            switch (mode * 2 + (vec ? 1 : 0)) {
                case kScanFieldInt * 2: rc = launch("scan_span", k_scan_span<kScanFieldInt, false>, grid, block, 0, r.stream, s); break;
                case kScanFieldInt * 2 + 1: rc = launch("scan_span", k_scan_span<kScanFieldInt, true>, grid, block, 0, r.stream, s); break;
                case kScanFieldL1 * 2: rc = launch("scan_span", k_scan_span<kScanFieldL1, false>, grid, block, 0, r.stream, s); break;
                case kScanFieldL1 * 2 + 1: rc = launch("scan_span", k_scan_span<kScanFieldL1, true>, grid, block, 0, r.stream, s); break;
                case kScanFieldFlt * 2: rc = launch("scan_span", k_scan_span<kScanFieldFlt, false>, grid, block, 0, r.stream, s); break;
                case kScanFieldFlt * 2 + 1: rc = launch("scan_span", k_scan_span<kScanFieldFlt, true>, grid, block, 0, r.stream, s); break;
                case kScanIndex * 2: rc = launch("scan_span", k_scan_span<kScanIndex, false>, grid, block, 0, r.stream, s); break;
                case kScanIndex * 2 + 1: rc = launch("scan_span", k_scan_span<kScanIndex, true>, grid, block, 0, r.stream, s); break;
                default: rc = launch("scan_span", k_scan_span<kScanFinal, false>, grid, block, 0, r.stream, s); break;
            }
        } else {
            s.span_lines = 1;
            const dim3 grid(s.lines), block(kWave);
            const size_t lds = 0;
            switch (mode) {
                case kScanFieldInt: rc = launch("scan_long", k_scan_long<kScanFieldInt>, grid, block, lds, r.stream, s); break;
                case kScanFieldL1: rc = launch("scan_long", k_scan_long<kScanFieldL1>, grid, block, lds, r.stream, s); break;
                case kScanFieldFlt: rc = launch("scan_long", k_scan_long<kScanFieldFlt>, grid, block, lds, r.stream, s); break;
                case kScanIndex: rc = launch("scan_long", k_scan_long<kScanIndex>, grid, block, lds, r.stream, s); break;
                default: rc = launch("scan_long", k_scan_long<kScanFinal>, grid, block, lds, r.stream, s); break;
            }
        }
        if (rc != TM_OK) return rc;
        if (nd == 1 && r.metric != kL2) {
            const uint64_t nb = (total + 255) / 256;
            rc = launch("cdt_none", k_cdt_none_to_minus1, dim3(uint32_t(nb)), dim3(256), 0, r.stream,
                        NoneArgs{r.sq, total});
            if (rc != TM_OK) return rc;
        }
    }

    // ---- strided passes, axis nd-2 down to 0 --------------------------------
    // Sampled rank-3 inputs on the index carrier whose two strided passes are
    // both tiled take the axis of the larger sampling first: its searches
    // are short (they stop once s_a^2 d^2 passes the best value found), and
    // the final pass, which its stores bound, takes the longer searches of the
    // other axis (2 x 256^3, sampling (2.5, 0.8, 0.8): middle pass 2.58 ->
    // 1.42 and final pass 1.00 -> 1.94 blocks of four steps per patch).
    // Any order gives the same minimum; unit sampling keeps this one, which
    // fixes the canonical index among equally near elements.
    int order[kMaxDim];
    const int npass = nd - 1;
    for (int i = 0; i < npass; ++i) order[i] = nd - 2 - i;
    if (index_path && !r.unit && nd == 3 && fh[0].tidx && fh[1].tidx && r.w[0] > r.w[1]) {
        order[0] = 0;
        order[1] = 1;
    }
    for (int oi = 0; oi < npass; ++oi) {
        const int a = order[oi];
        const FhPlan &p = fh[a];
        const uint32_t n = r.shape[a];
        uint64_t inner = 1;
        for (int b = a + 1; b < nd; ++b) inner *= r.shape[b];
        const uint64_t lines = total / n;
        const uint32_t lpw = p.lpw ? p.lpw : 1;     // lines per wave of the envelope kernels
        const dim3 grid(uint32_t((lines + lpw - 1) / lpw)), block(kWave);
        const bool fin = oi == npass - 1;
        if (p.l1long) {
            L1LongArgs la{};
            la.buf = r.sq;
            la.lines = lines;
            la.n = n;
            la.inner = uint32_t(inner);
            la.div_inner = Div32::make(la.inner);
            const dim3 lgrid(uint32_t((lines + kWave - 1) / kWave)), lblock(kWave);
            rc = fin ? launch("cdt_l1_long_final", k_cdt_l1_long<true>, lgrid, lblock, 0, r.stream, la)
                     : launch("cdt_l1_long", k_cdt_l1_long<false>, lgrid, lblock, 0, r.stream, la);
        } else if (p.tiled16) {
            PairArgs tg{};
            tg.buf = r.dist ? reinterpret_cast<int32_t *>(r.dist) : r.sq;
            tg.mask = r.in;
            tg.n2 = r.shape[nd - 1];
            tg.div_n2 = Div32::make(tg.n2);
            tg.total = uint32_t(total);
            tg.lines = uint32_t(lines);
            tg.n = n;
            tg.inner = uint32_t(inner);
            tg.div_inner = Div32::make(tg.inner);
            tg.out_seg = out_seg[a] ? 1 : 0;
            tg.in_seg = (a + 1 <= nd - 2 && out_seg[a + 1]) ? 1 : 0;
            tg.dist = r.dist;
            tg.sq = r.sq;
            tg.ndim = nd;
            for (int b = 0; b < nd; ++b) {
                tg.shape[b] = r.shape[b];
                tg.wall[b] = r.w[b];
            }
            const dim3 tgrid(uint32_t((lines + kPairLines - 1) / kPairLines)), tblock(kWave * kPairWaves);
            // Launch names carry the field layout: ".i16" reads and ".o16"
            // writes 16-bit runs (the measurement counts bytes from them).
            static const char *const names[2][2][2][2] = {
                {{{"tile_pair", "tile_pair.o16"}, {"tile_pair.i16", "tile_pair.i16.o16"}},
                 {{"tile_pair_final", "tile_pair_final"}, {"tile_pair_final.i16", "tile_pair_final.i16"}}},
                {{{"plane_pair", "plane_pair.o16"}, {"plane_pair", "plane_pair.o16"}},
                 {{"plane_pair_final", "plane_pair_final"}, {"plane_pair_final", "plane_pair_final"}}}};
            const char *nm = names[p.from_mask][fin][tg.in_seg][tg.out_seg];
            // search results stay in registers: 2 per lane and 16-row block
            if (r.metric != kL2) {
                static const char *const cnames[2][2][2] = {
                    {{"cdt_pair", "cdt_pair.o16"}, {"cdt_pair.i16", "cdt_pair.i16.o16"}},
                    {{"cdt_pair_final", "cdt_pair_final"}, {"cdt_pair_final.i16", "cdt_pair_final.i16"}}};
                nm = p.from_mask ? (fin ? "cdt_plane_final" : tg.out_seg ? "cdt_plane.o16" : "cdt_plane")
                                 : cnames[fin][tg.in_seg][tg.out_seg];
#define TM_CDT_PAIR(M)                                                                                   \
    (p.from_mask ? (fin ? launch(nm, k_tile_pair<true, true, 16, M>, tgrid, tblock, p.lds, r.stream, tg)  \
                        : launch(nm, k_tile_pair<false, true, 16, M>, tgrid, tblock, p.lds, r.stream, tg)) \
                 : (fin ? launch(nm, k_tile_pair<true, false, 16, M>, tgrid, tblock, p.lds, r.stream, tg)  \
                        : launch(nm, k_tile_pair<false, false, 16, M>, tgrid, tblock, p.lds, r.stream, tg)))
                rc = r.metric == kL1 ? TM_CDT_PAIR(kL1) : TM_CDT_PAIR(kLinf);
#undef TM_CDT_PAIR
            } else if (n <= 128) {
                if (p.from_mask)
                    rc = fin ? launch(nm, k_tile_pair<true, true, 8>, tgrid, tblock, p.lds, r.stream, tg)
                             : launch(nm, k_tile_pair<false, true, 8>, tgrid, tblock, p.lds, r.stream, tg);
                else
                    rc = fin ? launch(nm, k_tile_pair<true, false, 8>, tgrid, tblock, p.lds, r.stream, tg)
                             : launch(nm, k_tile_pair<false, false, 8>, tgrid, tblock, p.lds, r.stream, tg);
            } else {
                if (p.from_mask)
                    rc = fin ? launch(nm, k_tile_pair<true, true, 16>, tgrid, tblock, p.lds, r.stream, tg)
                             : launch(nm, k_tile_pair<false, true, 16>, tgrid, tblock, p.lds, r.stream, tg);
                else
                    rc = fin ? launch(nm, k_tile_pair<true, false, 16>, tgrid, tblock, p.lds, r.stream, tg)
                             : launch(nm, k_tile_pair<false, false, 16>, tgrid, tblock, p.lds, r.stream, tg);
            }
        } else if (p.lp16) {
            LinePairArgs lp{};
            lp.buf = r.dist ? reinterpret_cast<int32_t *>(r.dist) : r.sq;
            lp.dist = r.dist;
            lp.sq = r.sq;
            lp.lines = uint32_t(lines);
            lp.n = n;
            lp.inner = uint32_t(inner);
            lp.div_inner = Div32::make(lp.inner);
            lp.mult = plane_stride(uint32_t((lines / kLpLines) & ~uint64_t(31)) / 4u);
            lp.ndim = nd;
            for (int b = 0; b < nd; ++b) {
                lp.shape[b] = r.shape[b];
                lp.wall[b] = r.w[b];
            }
            const dim3 lgrid(uint32_t(lines / kLpLines)), lblock(kPsThreads);
            if (order_n && a == 0 && lgrid.x == order_n) lp.order = r.ws + order_n;
            if (pkw == 16 && a == nd - 2)
                rc = fin ? launch("line_pair_final.i16", k_line_pair16<true, true>, lgrid, lblock, p.lds, r.stream, lp)
                         : launch("line_pair.i16", k_line_pair16<false, true>, lgrid, lblock, p.lds, r.stream, lp);
            else
                rc = fin ? launch("line_pair_final", k_line_pair16<true>, lgrid, lblock, p.lds, r.stream, lp)
                         : launch("line_pair", k_line_pair16<false>, lgrid, lblock, p.lds, r.stream, lp);
        } else if (p.l1scan) {
            LineSearchArgs la{};
            la.buf = r.sq;
            la.lines = uint32_t(lines);
            la.n = n;
            la.inner = uint32_t(inner);
            la.div_inner = Div32::make(la.inner);
            const dim3 lgrid(uint32_t(lines / kL1Lines)), lblock(kWave * kL1Lines);
            const bool lpk = pkw == 8 && a == nd - 2;
            const char *nm = fin ? (lpk ? "cdt_l1_scan_final.i16" : "cdt_l1_scan_final")
                                 : (lpk ? "cdt_l1_scan.i16" : "cdt_l1_scan");
            // 16 rows per lane up to 1024 rows, else 36
            const bool r16 = n <= uint32_t(16 * kWave);
#define TM_L1S(F, PK)                                                                                   \
    (r16 ? launch(nm, k_cdt_l1_scan<F, PK, 16>, lgrid, lblock, p.lds, r.stream, la)                      \
         : launch(nm, k_cdt_l1_scan<F, PK, 36>, lgrid, lblock, p.lds, r.stream, la))
            rc = lpk ? (fin ? TM_L1S(true, true) : TM_L1S(false, true)) : (fin ? TM_L1S(true, false) : TM_L1S(false, false));
#undef TM_L1S
        } else if (p.ls_lpw) {
            LineSearchArgs la{};
            la.buf = r.dist ? reinterpret_cast<int32_t *>(r.dist) : r.sq;
            la.dist = r.dist;
            la.sq = r.sq;
            la.lines = uint32_t(lines);
            la.n = n;
            la.inner = uint32_t(inner);
            la.div_inner = Div32::make(la.inner);
            la.ndim = nd;
            for (int b = 0; b < nd; ++b) {
                la.shape[b] = r.shape[b];
                la.wall[b] = r.w[b];
            }
            if (order_n && a == 0 && p.ls_lpw == 8 && lines == 32 * order_n) la.order = r.ws + order_n;
            const dim3 lgrid(uint32_t((lines + p.ls_lpw - 1) / p.ls_lpw)), lblock(kWave * kLsWaves);
            const char *nm = r.metric == kL2 ? (fin ? "line_search_final" : "line_search")
                                             : (fin ? "cdt_line_final" : "cdt_line");
#define TM_LS4(M, F, W, S)                                                                                 \
    (p.ls_lpw == 8   ? launch(nm, k_line_search<M, F, W, 8, S>, lgrid, lblock, p.lds, r.stream, la)          \
     : p.ls_lpw == 4 ? launch(nm, k_line_search<M, F, W, 4, S>, lgrid, lblock, p.lds, r.stream, la)          \
     : p.ls_lpw == 2 ? launch(nm, k_line_search<M, F, W, 2, S>, lgrid, lblock, p.lds, r.stream, la)          \
                     : launch(nm, k_line_search<M, F, W, 1, S>, lgrid, lblock, p.lds, r.stream, la))
            // lines of the exact transform keep to 8 or 4 per workgroup (the
            // planner sends longer ones to the envelope kernels)
            // lines of at least kLsDirectMinRows take the few-site path
#define TM_LS(M, F, W)                                                                                            \
    (n >= kLsDirectMinRows                                                                                         \
         ? (p.ls_lpw == 8 ? launch(nm, k_line_search<M, F, W, 8, false, true>, lgrid, lblock, p.lds, r.stream, la) \
                          : launch(nm, k_line_search<M, F, W, 4, false, true>, lgrid, lblock, p.lds, r.stream, la)) \
         : (p.ls_lpw == 8 ? launch(nm, k_line_search<M, F, W, 8>, lgrid, lblock, p.lds, r.stream, la)              \
                          : launch(nm, k_line_search<M, F, W, 4>, lgrid, lblock, p.lds, r.stream, la)))
            if (pkw == 8 && a == nd - 2) {
                // the row scan's packed field, in strips of 8 lines (ls_lpw 8)
                nm = r.metric == kL2 ? (fin ? "line_search_final.i16" : "line_search.i16")
                                     : (fin ? "cdt_line_final.i16" : "cdt_line.i16");
#define TM_LSP(M, F, W, D) launch(nm, k_line_search<M, F, W, 8, false, D, true>, lgrid, lblock, p.lds, r.stream, la)
                if (r.metric == kL2)
                    rc = n >= kLsDirectMinRows ? (fin ? TM_LSP(kL2, true, false, true) : TM_LSP(kL2, false, false, true))
                                               : (fin ? TM_LSP(kL2, true, false, false) : TM_LSP(kL2, false, false, false));
                else if (r.metric == kL1)
                    rc = p.ls_w16 ? (fin ? TM_LSP(kL1, true, true, false) : TM_LSP(kL1, false, true, false))
                                  : (fin ? TM_LSP(kL1, true, false, false) : TM_LSP(kL1, false, false, false));
                else
                    rc = p.ls_w16 ? (fin ? TM_LSP(kLinf, true, true, false) : TM_LSP(kLinf, false, true, false))
                                  : (fin ? TM_LSP(kLinf, true, false, false) : TM_LSP(kLinf, false, false, false));
#undef TM_LSP
            } else if (r.sgn) {
                nm = fin ? "line_search_signed_final" : "line_search_signed";
                rc = fin ? TM_LS4(kL2, true, false, true) : TM_LS4(kL2, false, false, true);
            } else if (r.metric == kL2) rc = fin ? TM_LS(kL2, true, false) : TM_LS(kL2, false, false);
            else if (r.metric == kL1 && p.ls_w16) rc = fin ? TM_LS4(kL1, true, true, false) : TM_LS4(kL1, false, true, false);
            else if (r.metric == kL1) rc = fin ? TM_LS4(kL1, true, false, false) : TM_LS4(kL1, false, false, false);
            else if (p.ls_w16) rc = fin ? TM_LS4(kLinf, true, true, false) : TM_LS4(kLinf, false, true, false);
            else rc = fin ? TM_LS4(kLinf, true, false, false) : TM_LS4(kLinf, false, false, false);
#undef TM_LS
#undef TM_LS4
        } else if (!index_path) {
            FieldArgs f{};
            f.buf = r.dist ? static_cast<void *>(r.dist) : static_cast<void *>(r.sq);
            f.lines = lines;
            f.n = n;
            f.inner = uint32_t(inner);
            f.lpw = p.lpw;
            int vbits = bits_for(n - 1);
            f.vbits = uint32_t(vbits < 1 ? 1 : vbits);
            f.w = r.w[a];
            f.dist = r.dist;
            f.sq = r.sq;
            f.ndim = nd;
            for (int b = 0; b < nd; ++b) {
                f.shape[b] = r.shape[b];
                f.wall[b] = r.w[b];
            }
            const char *nm = fin ? "fh_field_final" : "fh_field";
#define TM_FIELD(M, PK, FN) launch(nm, k_fh_field<M, PK, FN>, grid, block, p.lds, r.stream, f)
            if (p.acc == 0 && p.pack) rc = fin ? TM_FIELD(ArI24, true, true) : TM_FIELD(ArI24, true, false);
            else if (p.acc == 0) rc = fin ? TM_FIELD(ArI24, false, true) : TM_FIELD(ArI24, false, false);
            else if (p.acc == 1 && p.pack) rc = fin ? TM_FIELD(ArI32, true, true) : TM_FIELD(ArI32, true, false);
            else if (p.acc == 1) rc = fin ? TM_FIELD(ArI32, false, true) : TM_FIELD(ArI32, false, false);
            else if (p.pack) rc = fin ? TM_FIELD(ArI64, true, true) : TM_FIELD(ArI64, true, false);
            else rc = fin ? TM_FIELD(ArI64, false, true) : TM_FIELD(ArI64, false, false);
#undef TM_FIELD
        } else if (p.tidx) {
            IdxTileArgs x{};
            x.idx = cidx;
            x.cstride = cstride;
            x.coords = coords;
            x.lines = uint32_t(lines);
            x.lps = uint32_t(vox / n);
            x.n = n;
            x.inner = uint32_t(inner);
            x.vox = uint32_t(vox);
            x.rbits = p.rbits;
            x.ndim = nd;
            x.axis = a;
            x.div_inner = Div32::make(uint32_t(inner));
            x.div_lps = Div32::make(x.lps);
            for (int b = 0; b < nd; ++b) {
                x.div_shape[b] = Div32::make(r.shape[b]);
                x.wall[b] = r.w[b];
                x.shape[b] = r.shape[b];
            }
            x.dist = fin ? r.dist : nullptr;
            x.sq = fin ? r.sq : nullptr;
            const dim3 igrid(uint32_t((lines + kIdxLines - 1) / kIdxLines)), iblock(kWave * kIdxWaves);
            // Ranks 2 and 3 take kernels with the rank and axis built in;
            // FAST ones when every extent after axis 0 is a power of two, the
            // line length a multiple of 32 and every buffer below 2 GiB.
            bool fast = (nd == 2 || nd == 3) && n % 32 == 0;
            {
                uint32_t shb = 0;
                for (int b = nd - 1; b >= 0; --b) {
                    const uint32_t e = r.shape[b];
                    if (b > 0 && (e & (e - 1)) != 0) fast = false;
                    x.sh[b] = shb;
                    x.msk[b] = b > 0 ? e - 1 : 0xffffffffu;
                    if (b > 0) shb += uint32_t(__builtin_ctz(e));
                }
                const uint64_t cb = r.batch * cstride * 4, db = r.batch * vox * 4;
                if (cb >= (uint64_t(1) << 31) || db >= (uint64_t(1) << 31)) fast = false;
                x.cbytes = uint32_t(cb);
                x.dbytes = uint32_t(db);
            }
            const char *nm = fin ? "tile_idx_final" : "tile_idx";
#define TM_TIDX_ND(S, F)                                                                          \
    (nd == 2             ? launch(nm, k_tile_idx<S, true, 2, 0, F>, igrid, iblock, p.lds, r.stream, x)  \
     : a == 1 && !fin    ? launch(nm, k_tile_idx<S, false, 3, 1, F>, igrid, iblock, p.lds, r.stream, x) \
     : a == 0 && fin     ? launch(nm, k_tile_idx<S, true, 3, 0, F>, igrid, iblock, p.lds, r.stream, x)  \
     : !S                ? int(TM_ERR_UNSUPPORTED) /* unit sampling keeps the default order */   \
     : a == 0            ? launch(nm, k_tile_idx<true, false, 3, 0, F>, igrid, iblock, p.lds, r.stream, x) \
                         : launch(nm, k_tile_idx<true, true, 3, 1, F>, igrid, iblock, p.lds, r.stream, x))
#define TM_TIDX(S)                                                                                \
    (nd == 2 || nd == 3 ? (fast ? TM_TIDX_ND(S, true) : TM_TIDX_ND(S, false))                      \
     : fin              ? launch(nm, k_tile_idx<S, true>, igrid, iblock, p.lds, r.stream, x)      \
                        : launch(nm, k_tile_idx<S, false>, igrid, iblock, p.lds, r.stream, x))
            rc = r.unit ? TM_TIDX(false) : TM_TIDX(true);
#undef TM_TIDX
#undef TM_TIDX_ND
        } else {
            IndexArgs x{};
            x.idx = cidx;
            x.cstride = cstride;
            x.coords = coords;
            x.lines = lines;
            x.lps = uint32_t(vox / n);
            x.n = n;
            x.inner = uint32_t(inner);
            x.lpw = p.lpw;
            x.vox = uint32_t(vox);
            x.ndim = nd;
            x.axis = a;
            x.div_inner = Div32::make(uint32_t(inner));
            for (int b = 0; b < nd; ++b) {
                x.div_shape[b] = Div32::make(r.shape[b]);
                x.wall[b] = r.w[b];
            }
            x.dist = fin ? r.dist : nullptr;
            x.sq = fin ? r.sq : nullptr;
            if (p.lng) {
                const dim3 lgrid(uint32_t((lines + kWave - 1) / kWave)), lblock(kWave);
                const char *ln = fin ? "fh_long_final" : "fh_long";
                if (r.unit)
                    rc = fin ? launch(ln, k_fh_long<false, true>, lgrid, lblock, 0, r.stream, x)
                             : launch(ln, k_fh_long<false, false>, lgrid, lblock, 0, r.stream, x);
                else
                    rc = fin ? launch(ln, k_fh_long<true, true>, lgrid, lblock, 0, r.stream, x)
                             : launch(ln, k_fh_long<true, false>, lgrid, lblock, 0, r.stream, x);
                if (rc != TM_OK) return rc;
                continue;
            }
            const char *nm = fin ? "fh_index_final" : "fh_index";
#define TM_INDEX(M, FN) launch(nm, k_fh_index<M, FN>, grid, block, p.lds, r.stream, x)
            if (p.acc == 3) rc = fin ? TM_INDEX(ArF64, true) : TM_INDEX(ArF64, false);
            else if (p.acc == 0) rc = fin ? TM_INDEX(ArI24, true) : TM_INDEX(ArI24, false);
            else if (p.acc == 1) rc = fin ? TM_INDEX(ArI32, true) : TM_INDEX(ArI32, false);
            else rc = fin ? TM_INDEX(ArI64, true) : TM_INDEX(ArI64, false);
#undef TM_INDEX
        }
        if (rc != TM_OK) return rc;
    }
    return TM_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C-ABI
// ---------------------------------------------------------------------------
extern "C" int tm_edt(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
                      const double *sampling, float *out_dist, int32_t *out_idx,
                      hipStream_t stream) {
    Request r{};
    // float outputs: exact squared distances of any size are carried in
    // 64-bit arithmetic (flat-index carrier), so no int32 bound applies
    int rc = validate(in_u8, ndim, shape, batch, sampling, out_dist, out_idx, nullptr, r, false);
    if (rc != TM_OK) return rc;
    r.dist = out_dist;
    r.sq = nullptr;
    r.idx = out_idx;
    r.stream = stream;
    return run(r);
}

extern "C" int tm_edt_ws(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
                         const double *sampling, float *out_dist, int32_t *out_idx, void *workspace,
                         size_t workspace_bytes, hipStream_t stream) {
    Request r{};
    int rc = validate(in_u8, ndim, shape, batch, sampling, out_dist, out_idx, nullptr, r, false);
    if (rc != TM_OK) return rc;
    if (workspace && uintptr_t(workspace) % 4 != 0) return TM_ERR_WORKSPACE;
    r.dist = out_dist;
    r.sq = nullptr;
    r.idx = out_idx;
    r.ws = workspace_bytes ? static_cast<uint32_t *>(workspace) : nullptr;
    r.ws_bytes = workspace ? workspace_bytes : 0;
    r.stream = stream;
    return run(r);
}

extern "C" size_t tm_edt_workspace_size(int ndim, const int64_t *shape, int64_t batch, const double *sampling,
                                        int with_indices) {
    Request r{};
    // any non-null device addresses: only the shapes matter here
    const void *dummy = reinterpret_cast<const void *>(uintptr_t(4096));
    if (validate(static_cast<const uint8_t *>(dummy), ndim, shape, batch, sampling, dummy,
                 with_indices ? dummy : nullptr, nullptr, r, false) != TM_OK)
        return 0;
    r.dist = reinterpret_cast<float *>(uintptr_t(4096));
    r.idx = with_indices ? reinterpret_cast<int32_t *>(uintptr_t(4096)) : nullptr;
    if (r.idx || !r.unit || r.big || r.ndim != 2) return 0;
    uint64_t vox = 1;
    for (int a = 0; a < r.ndim; ++a) vox *= r.shape[a];
    const uint64_t total = r.batch * vox;
    // the fused small 2-D kernel takes both extents up to kSmallMax
    if (r.shape[0] <= uint32_t(kSmallMax) && r.shape[1] <= uint32_t(kSmallMax)) return 0;
    FhPlan fh[kMaxDim];
    if (plan_passes(r, total, false, fh) != TM_OK) return 0;
    const uint64_t g = order_groups(r, fh, total).groups;
    return g ? size_t(order_workspace_bytes(g)) : 0;
}

namespace {

// ---------------------------------------------------------------------------
// Allocation-free workspace of tm_edt_noalloc: one static array per device
// (each device that loads the library holds its own copy, zero at load, until
// the process ends).  In host code `scratch` names a host-side stand-in, not
// the device array: its device address comes from hipGetSymbolAddress, once
// per device with that device current, and only that address is passed on.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = 64 * 1024;     // the dispatch order of up to 8192 groups
static __device__ __align__(256) uint32_t scratch[kScratchBytes / 4];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint32_t *g_scratch_ptr[kMaxDevices] = {};

int scratch_address(uint32_t **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TM_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TM_ERR_HIP;
        g_scratch_ptr[dev] = static_cast<uint32_t *>(p);
    }
    *out = g_scratch_ptr[dev];
    return TM_OK;
}

}  // namespace

extern "C" int tm_edt_noalloc(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
                              const double *sampling, float *out_dist, int32_t *out_idx, hipStream_t stream) {
    Request r{};
    int rc = validate(in_u8, ndim, shape, batch, sampling, out_dist, out_idx, nullptr, r, false);
    if (rc != TM_OK) return rc;
    const size_t need = tm_edt_workspace_size(ndim, shape, batch, sampling, out_idx != nullptr);
    if (need > kScratchBytes) return TM_ERR_WORKSPACE;
    uint32_t *ws = nullptr;
    if (need) {
        rc = scratch_address(&ws);
        if (rc != TM_OK) return rc;
    }
    r.dist = out_dist;
    r.sq = nullptr;
    r.idx = out_idx;
    r.ws = ws;
    r.ws_bytes = ws ? kScratchBytes : 0;
    r.stream = stream;
    return run(r);
}

extern "C" int tm_edt_sq(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
                         int32_t *out_sq, int32_t *out_idx, hipStream_t stream) {
    Request r{};
    int rc = validate(in_u8, ndim, shape, batch, nullptr, out_sq, out_idx, nullptr, r);
    if (rc != TM_OK) return rc;
    r.dist = nullptr;
    r.sq = out_sq;
    r.idx = out_idx;
    r.stream = stream;
    return run(r);
}

extern "C" int tm_dt_bf(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch, int metric,
                        const double *sampling, float *out_dist, int32_t *out_idx, hipStream_t stream) {
    Request r{};
    int rc = validate(in_u8, ndim, shape, batch, sampling, out_dist, out_idx, nullptr, r);
    if (rc != TM_OK) return rc;
    if (metric < TM_METRIC_EUCLIDEAN || metric > TM_METRIC_CHESSBOARD) return TM_ERR_METRIC;
    uint64_t vox = 1;
    for (int a = 0; a < ndim; ++a) vox *= r.shape[a];
    const uint64_t total = r.batch * vox;
    if (overlaps(in_u8, total, out_dist, 4 * total) || overlaps(in_u8, total, out_idx, 4 * total * ndim) ||
        overlaps(out_dist, 4 * total, out_idx, 4 * total * ndim))
        return TM_ERR_ALIAS;
    BfArgs x{};
    x.in = in_u8;
    x.dist = out_dist;
    x.idx = out_idx;
    x.vox = uint32_t(vox);
    x.bps = uint32_t((vox + kBfOut - 1) / kBfOut);
    if (uint64_t(x.bps) * r.batch >= (uint64_t(1) << 31)) return TM_ERR_TOO_LARGE;
    x.ndim = ndim;
    for (int a = 0; a < ndim; ++a) {
        x.div_shape[a] = Div32::make(r.shape[a]);
        x.sd[a] = sampling ? sampling[a] : 1.0;
        x.s[a] = float(x.sd[a]);
    }
    const dim3 grid(uint32_t(x.bps * r.batch)), block(kBfThreads);
    const bool samp = !r.unit;
#define TM_BF(M, S)                                                                               \
    (ndim == 2   ? launch("dt_bf", k_dt_bf<M, S, 2>, grid, block, 0, stream, x)                   \
     : ndim == 3 ? launch("dt_bf", k_dt_bf<M, S, 3>, grid, block, 0, stream, x)                   \
                 : launch("dt_bf", k_dt_bf<M, S, 0>, grid, block, 0, stream, x))
    if (metric == TM_METRIC_EUCLIDEAN) rc = samp ? TM_BF(0, true) : TM_BF(0, false);
    else if (metric == TM_METRIC_TAXICAB) rc = samp ? TM_BF(1, true) : TM_BF(1, false);
    else rc = samp ? TM_BF(2, true) : TM_BF(2, false);
#undef TM_BF
    return rc;
}

extern "C" int tm_edt_signed(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch,
                             float *out_dist, hipStream_t stream) {
    Request r{};
    int rc = validate(in_u8, ndim, shape, batch, nullptr, out_dist, nullptr, nullptr, r);
    if (rc != TM_OK) return rc;
    r.dist = out_dist;
    r.sq = nullptr;
    r.idx = nullptr;
    r.stream = stream;
    r.sgn = true;
    return run(r);
}

extern "C" int tm_cdt_ws(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch, int metric,
                         int32_t *out_dist, void *workspace, size_t workspace_bytes, hipStream_t stream) {
    Request r{};
    int rc = validate(in_u8, ndim, shape, batch, nullptr, nullptr, out_dist, nullptr, r, false);
    if (rc != TM_OK) return rc;
    if (metric != TM_METRIC_TAXICAB && metric != TM_METRIC_CHESSBOARD) return TM_ERR_METRIC;
    if (workspace && uintptr_t(workspace) % 4 != 0) return TM_ERR_WORKSPACE;
    r.dist = nullptr;
    r.sq = out_dist;
    r.idx = nullptr;
    r.ws = workspace_bytes ? static_cast<uint32_t *>(workspace) : nullptr;
    r.ws_bytes = workspace ? workspace_bytes : 0;
    r.stream = stream;
    r.metric = metric == TM_METRIC_TAXICAB ? kL1 : kLinf;
    return run(r);
}

extern "C" int tm_cdt(const uint8_t *in_u8, int ndim, const int64_t *shape, int64_t batch, int metric,
                      int32_t *out_dist, hipStream_t stream) {
    return tm_cdt_ws(in_u8, ndim, shape, batch, metric, out_dist, nullptr, 0, stream);
}

extern "C" size_t tm_cdt_workspace_size(int ndim, const int64_t *shape, int64_t batch, int metric) {
    Request r{};
    const void *dummy = reinterpret_cast<const void *>(uintptr_t(4096));
    if (validate(static_cast<const uint8_t *>(dummy), ndim, shape, batch, nullptr, nullptr, dummy, nullptr, r,
                 false) != TM_OK)
        return 0;
    if (metric != TM_METRIC_TAXICAB && metric != TM_METRIC_CHESSBOARD) return 0;
    r.sq = reinterpret_cast<int32_t *>(uintptr_t(4096));
    r.metric = metric == TM_METRIC_TAXICAB ? kL1 : kLinf;
    if (r.ndim != 2) return 0;
    uint64_t vox = 1;
    for (int a = 0; a < r.ndim; ++a) vox *= r.shape[a];
    const uint64_t total = r.batch * vox;
    FhPlan fh[kMaxDim];
    if (plan_passes(r, total, false, fh) != TM_OK) return 0;
    const uint64_t g = order_groups(r, fh, total).groups;
    return g ? size_t(order_workspace_bytes(g)) : 0;
}

extern "C" int tm_mask_nonzero(const void *in, int dtype, int ndim, const int64_t *shape,
                               const int64_t *strides, uint8_t *out_u8, hipStream_t stream) {
    if (ndim < 1 || ndim > kMaskMaxDim) return TM_ERR_NDIM;
    if (!shape) return TM_ERR_SHAPE;
    if (!in) return TM_ERR_NULL;
    if (!out_u8) return TM_ERR_NO_OUTPUT;
    if (dtype < TM_DTYPE_U8 || dtype > TM_DTYPE_F8) return TM_ERR_DTYPE;
    static const int esize[] = {1, 2, 4, 8, 2, 2, 4, 8, 1};
    const int E = esize[dtype];
    const bool flt = dtype >= TM_DTYPE_F16;
    uint64_t n = 1, span = uint64_t(E);   // elements, and bytes from `in` to the end of the last one
    bool contig = true;
    uint64_t want = uint64_t(E);          // C-order stride of the current axis
    for (int b = ndim - 1; b >= 0; --b) {
        if (shape[b] < 1) return TM_ERR_SHAPE;
        const int64_t st = strides ? strides[b] : int64_t(want);
        if (st < 0) return TM_ERR_SHAPE;
        if (uint64_t(shape[b]) >= (uint64_t(1) << 32)) return TM_ERR_TOO_LARGE;
        n *= uint64_t(shape[b]);
        if (n >= (uint64_t(1) << 32)) return TM_ERR_TOO_LARGE;
        if (shape[b] > 1 && uint64_t(st) != want) contig = false;
        span += uint64_t(shape[b] - 1) * uint64_t(st);
        if (span >= (uint64_t(1) << 62)) return TM_ERR_TOO_LARGE;
        want *= uint64_t(shape[b]);
    }
    if (overlaps(in, span, out_u8, n)) return TM_ERR_ALIAS;
    MaskArgs m{};
    m.in = static_cast<const uint8_t *>(in);
    m.out = out_u8;
    m.n = uint32_t(n);
    m.ndim = ndim;
    for (int b = 0; b < ndim; ++b) {
        m.div_shape[b] = Div32::make(uint32_t(shape[b]));
        m.stride[b] = strides ? strides[b] : 0;
    }
    const uint64_t per = uint64_t(kMaskThreads) * kMaskPer;
    const dim3 grid(uint32_t((n + per - 1) / per)), block(kMaskThreads);
#define TM_MASK(EB, F)                                                                                  \
    (contig ? launch("mask_nonzero", k_mask_nonzero<EB, F, true>, grid, block, 0, stream, m)            \
            : launch("mask_nonzero", k_mask_nonzero<EB, F, false>, grid, block, 0, stream, m))
    switch (E * 2 + (flt ? 1 : 0)) {
        case 2: return TM_MASK(1, false);
        case 3: return TM_MASK(1, true);
        case 4: return TM_MASK(2, false);
        case 5: return TM_MASK(2, true);
        case 8: return TM_MASK(4, false);
        case 9: return TM_MASK(4, true);
        case 16: return TM_MASK(8, false);
        default: return TM_MASK(8, true);
    }
#undef TM_MASK
}

extern "C" const char *tm_strerror(int status) {
    switch (status) {
        case TM_OK: return "success";
        case TM_ERR_NDIM: return "spatial rank must be between 1 and 8";
        case TM_ERR_SHAPE: return "shape is missing or has an extent below 1";
        case TM_ERR_BATCH: return "batch must be at least 1";
        case TM_ERR_NULL: return "input pointer is null";
        case TM_ERR_NO_OUTPUT: return "at least one output must be requested";
        case TM_ERR_SAMPLING: return "sampling entries must be finite and positive";
        case TM_ERR_TOO_LARGE: return "input too large for 32-bit indices or int32 squared distances";
        case TM_ERR_ALIAS: return "input and output buffers overlap";
        case TM_ERR_UNSUPPORTED: return "a line is longer than the signed or chessboard kernels hold in LDS";
        case TM_ERR_HIP: return "HIP runtime error while enqueuing kernels";
        case TM_ERR_METRIC: return "metric must be euclidean, taxicab or chessboard";
        case TM_ERR_DTYPE: return "element type is not one of tm_dtype";
        case TM_ERR_WORKSPACE: return "workspace is not 4-byte aligned, or the request needs more than the static workspace";
        default: return "unknown status";
    }
}

extern "C" int tm_prof_enable(int max_kernels) {
    Prof &p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    for (size_t k = 0; k < p.start.size(); ++k) {
        (void)hipEventDestroy(p.start[k]);
        (void)hipEventDestroy(p.stop[k]);
    }
    p.start.clear();
    p.stop.clear();
    p.names.clear();
    p.cap = 0;
    p.next = 0;
    if (max_kernels <= 0) return TM_OK;
    p.start.resize(max_kernels);
    p.stop.resize(max_kernels);
    p.names.assign(max_kernels, nullptr);
    p.info.assign(max_kernels, {});
    for (int k = 0; k < max_kernels; ++k) {
        if (hipEventCreate(&p.start[k]) != hipSuccess || hipEventCreate(&p.stop[k]) != hipSuccess) {
            p.start.resize(k);
            p.stop.resize(k);
            return TM_ERR_HIP;
        }
    }
    p.cap = max_kernels;
    return TM_OK;
}

extern "C" int tm_prof_count(void) {
    Prof &p = prof();
    int c = p.next.load();
    return c < p.cap ? c : p.cap;
}

extern "C" int tm_prof_read(int i, const char **name, float *ms) {
    Prof &p = prof();
    if (i < 0 || i >= tm_prof_count()) return TM_ERR_SHAPE;
    if (name) *name = p.names[i];
    if (ms && hipEventElapsedTime(ms, p.start[i], p.stop[i]) != hipSuccess) return TM_ERR_HIP;
    return TM_OK;
}

extern "C" int tm_prof_launch(int i, int64_t *info) {
    Prof &p = prof();
    if (i < 0 || i >= tm_prof_count() || !info) return TM_ERR_SHAPE;
    for (int k = 0; k < 6; ++k) info[k] = p.info[i][k];
    return TM_OK;
}

extern "C" int tm_selftest_host(void) {
    int bad = 0;
    const uint32_t divs[] = {1u, 2u, 3u, 5u, 7u, 64u, 100u, 127u, 128u, 255u, 256u, 1000u,
                             4096u, 65535u, 65536u, 1u << 20, 16777215u, 2147483647u,
                             2147483648u, 4294967295u};
    uint64_t state = 0x9e3779b97f4a7c15ull;
    for (uint32_t d : divs) {
        Div32 q = Div32::make(d);
        for (int t = 0; t < 20000; ++t) {
            state = state * 6364136223846793005ull + 1442695040888963407ull;
            uint32_t x = uint32_t(state >> 32);
            if (t < 8) x = (t < 4) ? uint32_t(t) : 0xffffffffu - uint32_t(t - 4);
            if (t == 8) x = d;
            if (t == 9) x = d - 1;
            if (q.div(x) != x / d) ++bad;
        }
    }
    return bad ? -bad : TM_OK;
}
