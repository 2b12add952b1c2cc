// Tiled pass on the index carrier: nearest background elements (and, on the
// last pass, distances and coordinates) for unit or anisotropic sampling.
//
// A workgroup owns 32 adjacent lines of one pass (two workgroups fit a
// compute unit at 256 rows, so one stages while the other searches).  It
// stages, per line and row, the carried site (the in-sample flat index of the
// nearest background element found by the earlier passes, -1 for none) and
// the site's squared distance over the axes already processed, recomputed
// from the site's coordinates.  Each element then runs the windowed exact
// search over the rows of its line: examine rows at growing distance d and
// stop once w d^2 exceeds the best value found; a lane searches two adjacent
// rows of one line, which share every row read.  The winner's site comes from
// the staged copy, so the pass can overwrite its lines in place.  The axes
// already processed are those after the pass axis (passes from the last axis
// down), or, with the rank built in, the last axis and, in the final pass,
// every other axis (rank 3 may take its two strided axes in either order).
//
// Unit sampling: values are exact integers and a candidate is the key
// (value << RB) | row, so one integer minimum picks the smallest value and,
// among equal values, the smallest row: the canonical choice of the
// separable method (smallest flat index among nearest elements).
// Sampled: values are float, w = s_a^2.  Each step keeps only the smaller
// of its two rows' candidates (min(f(q-e), f(q+e)) + w e^2, which rounds to
// the smaller of the two sums), and each block of four steps only its
// minimum, the first block that reached the best value and that block's four
// candidates; the row is found once at the end (any nearest element is
// correct there).
#pragma once

#include "edt_fh.h"

namespace tmedt {

constexpr int kIdxWaves = 16;
constexpr int kIdxLines = 32;     // lines per workgroup
constexpr int kIdxGuard = 5;       // guard rows of "no site" per side (a block reads 5 rows per side)
constexpr int kIdxRowW = kIdxLines + 4;  // padded row stride (words)

struct IdxTileArgs {
    int32_t *idx;            // the carrier of the sites: slice 0 of [batch][ndim][vox], or a
                             // distance output holding flat indices (cstride = vox)
    uint64_t cstride;        // carrier elements per sample
    int32_t coords;          // final pass: write the ndim coordinate slices at idx
    float *dist;             // final pass outputs (each may be null; may be the carrier)
    int32_t *sq;
    uint32_t lines;          // batch * lps
    uint32_t lps;            // lines per sample
    uint32_t n;              // line length
    uint32_t inner;          // element stride of the line
    uint32_t vox;            // elements per sample
    uint32_t rbits;          // unit: bits of the row in a key
    int32_t ndim;
    int32_t axis;
    Div32 div_inner;
    Div32 div_lps;
    Div32 div_shape[kMaxDim];
    double wall[kMaxDim];    // squared sampling per axis
    uint32_t shape[kMaxDim];
    // FAST kernels only: every extent after axis 0 is a power of two and
    // every buffer below 2 GiB.  Coordinate b of an in-sample flat index y
    // is (y >> sh[b]) & msk[b]; rc / rd / rs span the carrier buffer (from
    // idx), dist and sq.
    uint32_t sh[kMaxDim];
    uint32_t msk[kMaxDim];
    uint32_t cbytes, dbytes;
};

// LDS words of the two tile arrays for lines of n rows, and of the table of
// w k^2 for k = 0 .. n + 7 (sampled searches; three leading words align the
// blocks' reads).
__host__ __device__ constexpr uint32_t idx_tile_words(uint32_t n) { return (n + 2 * kIdxGuard) * kIdxRowW; }
__host__ __device__ constexpr uint32_t idx_step_words(uint32_t n) { return (n + 12 + 3) & ~3u; }
__host__ __device__ constexpr size_t idx_tile_lds(uint32_t n, bool samp) {
    return size_t(2 * idx_tile_words(n) + (samp ? idx_step_words(n) : 0u)) * 4u;
}

// ND, AX: rank and axis of the pass fixed at compile time (ND = 0: taken
// from the arguments), so the coordinate loops unroll without tests.
// FAST (ND > 0 only): coordinates by shifts and masks, and every global
// access through a buffer resource with a 32-bit byte offset, the row and
// slice parts of which are wave-uniform scalar offsets.
// Lines of a search patch (a lane takes two adjacent rows of one line, so a
// patch has 128 / lines rows).  FAST passes take 32 lines, so each store
// instruction writes two whole 128-byte segments (2 x 256^3 sampled with
// indices, one row per lane: final pass 171 -> 145 us, middle pass 117 ->
// 109 us against 8 x 8 patches); the others take 8.
__host__ __device__ constexpr int idx_patch_lines(bool fast) { return fast ? 32 : 8; }

template <bool SAMP, bool FINAL, int ND = 0, int AX = 0, bool FAST = false>
__global__ void __launch_bounds__(kWave * kIdxWaves) k_tile_idx(IdxTileArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    constexpr int kGroups = kWave * kIdxWaves / kIdxLines;   // staging row groups
    static_assert(kIdxLines == 32, "staging: lanes l and l + 32 of a wave take line l");
    __shared__ __attribute__((aligned(16))) uint32_t wave_has[kIdxWaves];   // per wave: bit l set when line l has a site in its rows
    // per line: sample and base of row 0 in slice 0 (FAST: byte offsets of
    // row 0 in the carrier and in the outputs), position i, live
    __shared__ uint4 line_info[kIdxLines];
    __shared__ uint32_t line_pos0[kIdxLines];  // per line: position o along the earlier axes
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(t / kWave);
    const int n = int(a.n);
    const int nd = ND ? ND : a.ndim;
    const int ax = ND ? AX : a.axis;
    const uint32_t tw = idx_tile_words(uint32_t(n));
    uint32_t *val0 = lds + kIdxGuard * kIdxRowW;             // row 0 of the values / keys
    int32_t *site0 = reinterpret_cast<int32_t *>(lds + tw) + kIdxGuard * kIdxRowW;   // row 0 of the sites
    float *const step = reinterpret_cast<float *>(lds + 2 * tw) + 3;   // sampled: step[k] = w k^2
    const uint32_t L0 = blockIdx.x * uint32_t(kIdxLines);

    // Line j of the workgroup: sample, base of the line in slice 0, position
    // along the later axes.
    struct Line {
        bool live;
        uint32_t s, base, i, o;
    };
    auto line_of = [&](int j) {
        Line l;
        const uint32_t L = L0 + uint32_t(j);
        l.live = L < a.lines;
        const uint32_t LL = l.live ? L : L0;
        l.s = a.div_lps.div(LL);
        const uint32_t r = LL - l.s * a.lps;
        const uint32_t o = a.div_inner.div(r);
        l.i = r - o * a.inner;
        l.o = o;                                // position along the earlier axes
        l.base = o * a.n * a.inner + l.i;       // in-sample flat of row 0
        return l;
    };
    // Axes whose distances the carried sites already hold.  In the generic
    // kernel the passes run from the last axis to axis 0, so those are the
    // axes after `ax`.  With the rank built in, a pass along axis AX follows
    // the last-axis scan, and the final pass every other axis: for rank 3 a
    // non-final pass along either strided axis has the last axis behind it.
    auto proc = [&](int b) -> bool {
        if constexpr (ND > 0) return b != AX && (b == ND - 1 || FINAL);
        else return b > ax && b < nd;
    };
    // Coordinates of this lane's line along the processed axes (staging),
    // computed once: those after `ax` from its position i along them, those
    // before from its position o along them (rank 3: o is the coordinate
    // along axis 0).
    int xc[kMaxDim] = {};
    float wf[kMaxDim] = {};
    auto line_coords = [&](uint32_t xi, uint32_t xo) {
#pragma unroll
        for (int b = kMaxDim - 1; b >= 0; --b) {
            if (b > ax && b < nd) {
                const uint32_t qx = a.div_shape[b].div(xi);
                xc[b] = int(xi - qx * a.div_shape[b].d);
                xi = qx;
            }
            if (b < nd && proc(b)) wf[b] = float(a.wall[b]);
        }
        if constexpr (ND == 3 && AX == 1) xc[0] = int(xo);
    };
    // squared distance over the processed axes between this lane's line and
    // site y (in-sample flat; its coordinate along axis b is its remainder by
    // extent b after dividing by the later extents), or "none" (sampled:
    // float sum of the exact integer squares times the squared sampling)
    auto carried = [&](int32_t y, uint32_t &key_or_bits, int q) {
        if (y < 0) {
            key_or_bits = SAMP ? __builtin_bit_cast(uint32_t, __builtin_inff()) : uint32_t(kInfI);
            return;
        }
        uint32_t yi = uint32_t(y);
        float accf = 0.0f;
        uint32_t acci = 0;
#pragma unroll
        for (int b = kMaxDim - 1; b >= 0; --b) {
            // (rank 3, final pass along axis 1: axis 0 is the quotient left)
            const bool need = b < nd && (ND == 3 && AX == 1 && FINAL ? true : b > ax);
            if (need) {
                const uint32_t qy = b > 0 ? a.div_shape[b].div(yi) : 0u;
                const int dy = int(yi - qy * a.div_shape[b].d) - xc[b];
                yi = qy;
                if (proc(b)) {
                    if (SAMP) accf += wf[b] * float(dy * dy);
                    else acci += uint32_t(dy * dy);
                }
            }
        }
        key_or_bits = SAMP ? __builtin_bit_cast(uint32_t, accf) : ((acci << a.rbits) | uint32_t(q));
    };

    // Squared distance from element (row q of a line at positions i, o) to
    // the virtual background element (-1, 0, ..., 0), for samples without
    // background (double when sampled, exact integers otherwise).
    auto virtual_d2 = [&](int q, uint32_t i, uint32_t o) -> double {
        if constexpr (ND == 3 && AX == 1) {
            // x0 = o, x1 = q, x2 = i
            if (SAMP)
                return a.wall[0] * double(o + 1) * double(o + 1) + a.wall[1] * double(q) * double(q) +
                       a.wall[2] * double(i) * double(i);
            return double(int64_t(o + 1) * (o + 1) + int64_t(q) * q + int64_t(i) * i);
        } else {
            return SAMP ? virtual_sq<double>(q, i, nd, a.shape, a.wall)
                        : double(virtual_sq<int64_t>(q, i, nd, a.shape, a.wall));
        }
    };

    // ---- guard rows, step table and staging ---------------------------------
    for (int k = t; k < kIdxGuard * kIdxRowW; k += kWave * kIdxWaves) {
        const uint32_t none = SAMP ? __builtin_bit_cast(uint32_t, __builtin_inff()) : uint32_t(kInfI);
        lds[k] = none;
        val0[n * kIdxRowW + k] = none;
    }
    if constexpr (SAMP) {
        const float w = float(a.wall[ax]);
        for (int k = t; k <= n + 7; k += kWave * kIdxWaves) step[k] = w * float(k * k);
    }
    // thread t stages line t % kIdxLines, rows t / kIdxLines + kGroups j
    const int sl = t & (kIdxLines - 1), sg = t / kIdxLines;
    const Line me = line_of(sl);
    const uint32_t cvo = (me.s * uint32_t(a.cstride) + me.base) * 4u;   // FAST: carrier byte offset of row 0
    if (t < kIdxLines)
        line_info[sl] = FAST ? uint4{cvo, (me.s * a.vox + me.base) * 4u, me.i, me.live ? 1u : 0u}
                             : uint4{me.s, me.base, me.i, me.live ? 1u : 0u};
    line_coords(me.i, me.o);
    if (t < kIdxLines) line_pos0[sl] = me.o;
    const int32_t *src = a.idx + uint64_t(me.s) * a.cstride + me.base;
    // FAST only (a null resource elsewhere)
    const __amdgpu_buffer_rsrc_t rc = make_rsrc(a.idx, FAST ? a.cbytes : 0u);
    const __amdgpu_buffer_rsrc_t rd = make_rsrc(a.dist, FAST && a.dist ? a.dbytes : 0u);
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.sq, FAST && a.sq ? a.dbytes : 0u);
    uint32_t seen = 0;
    constexpr int SB = 8;
    const uint32_t svo = cvo + uint32_t(sg) * a.inner * 4u;
    if constexpr (FAST) {
        // n is a multiple of 32 = kGroups, so every row test is uniform, and
        // the values are computed without branches ("none" selected at the end)
        const int32_t dead = me.live ? 0 : -1;
        int32_t ymax = -1;
        uint32_t *const vrow = val0 + sg * kIdxRowW + sl;
        int32_t *const srow = site0 + sg * kIdxRowW + sl;
        for (int it = 0; it * kGroups * SB < n; ++it) {
            int32_t y[SB];
#pragma unroll
            for (int j = 0; j < SB; ++j) {
                const int u = it * kGroups * SB + j * kGroups;
                y[j] = u < n ? int32_t(__builtin_amdgcn_raw_buffer_load_b32(rc, svo, uint32_t(u) * a.inner * 4u, 0))
                             : -1;
            }
#pragma unroll
            for (int j = 0; j < SB; ++j) {
                const int u = it * kGroups * SB + j * kGroups;
                if (u < n) {
                    const int32_t yy = y[j] | dead;
                    float accf = 0.0f;
                    uint32_t acci = 0;
#pragma unroll
                    for (int b = ND - 1; b >= 0; --b) {
                        if (proc(b)) {
                            const int dy = int((uint32_t(yy) >> a.sh[b]) & a.msk[b]) - xc[b];
                            if (SAMP) accf += wf[b] * float(dy * dy);
                            else acci += uint32_t(dy * dy);
                        }
                    }
                    const uint32_t v = SAMP ? __builtin_bit_cast(uint32_t, accf) : ((acci << a.rbits) | uint32_t(sg + u));
                    const uint32_t none = SAMP ? __builtin_bit_cast(uint32_t, __builtin_inff()) : uint32_t(kInfI);
                    ymax = max(ymax, yy);
                    vrow[u * kIdxRowW] = yy < 0 ? none : v;
                    srow[u * kIdxRowW] = yy;
                }
            }
        }
        seen = ymax >= 0 ? 1u : 0u;
    } else {
        for (int it = 0; it * kGroups * SB < n; ++it) {
            const int q0 = sg + it * kGroups * SB;
            int32_t y[SB];
#pragma unroll
            for (int j = 0; j < SB; ++j) y[j] = src[uint64_t(min(q0 + j * kGroups, n - 1)) * a.inner];
#pragma unroll
            for (int j = 0; j < SB; ++j) {
                const int q = q0 + j * kGroups;
                if (q < n) {
                    const int32_t yy = me.live ? y[j] : -1;
                    uint32_t v;
                    carried(yy, v, q);
                    seen |= yy >= 0 ? 1u : 0u;
                    val0[q * kIdxRowW + sl] = v;
                    site0[q * kIdxRowW + sl] = yy;
                }
            }
        }
    }
    {
        // lanes l and l + 32 of a wave stage line l
        const uint64_t bal = __ballot(seen != 0u);
        if (lane == 0) wave_has[wv] = uint32_t(bal) | uint32_t(bal >> 32);
    }
    __syncthreads();
    uint32_t has_mask = 0;
#pragma unroll
    for (int k = 0; k < kIdxWaves; k += 4) {
        const uint4 h = *reinterpret_cast<const uint4 *>(&wave_has[k]);
        has_mask |= h.x | h.y | h.z | h.w;
    }

    // ---- output of element (row qr, line ln) --------------------------------
    const uint32_t rmask = (1u << a.rbits) - 1u;
    int32_t *slice0 = nullptr;
    auto output = [&](int qr, int ln, bool has, uint32_t best, int r_best) {
        const uint4 li = line_info[ln];
        if (!li.w) return;
        int32_t site = -1;
        if (has) {
            const int rw = SAMP ? r_best : int(best & rmask);
            site = site0[rw * kIdxRowW + ln];
        }
        if constexpr (FAST) {
            const uint32_t ro = uint32_t(qr) * a.inner * 4u;   // byte offset of row qr
            const uint32_t co = li.x + ro;                     // the element in slice 0 of the carrier
            if (!FINAL) {
                __builtin_amdgcn_raw_buffer_store_b32(uint32_t(site), rc, co, 0, 0);
                return;
            }
            const float fbest = __builtin_bit_cast(float, best);
            double d2;
            if (site >= 0) {
                d2 = SAMP ? double(fbest) : double(best >> a.rbits);
                if (a.coords) {
#pragma unroll
                    for (int b = 0; b < ND; ++b)
                        __builtin_amdgcn_raw_buffer_store_b32((uint32_t(site) >> a.sh[b]) & a.msk[b], rc, co,
                                                              uint32_t(b) * a.vox * 4u, 0);
                }
            } else {
                // no background in the sample: the virtual element (-1, 0, ..., 0)
                d2 = virtual_d2(qr, li.z, line_pos0[ln]);
                if (a.coords) {
#pragma unroll
                    for (int b = 0; b < ND; ++b)
                        __builtin_amdgcn_raw_buffer_store_b32(b == 0 ? 0xffffffffu : 0u, rc, co,
                                                              uint32_t(b) * a.vox * 4u, 0);
                }
            }
            const float dist = (SAMP && site >= 0)                ? sqrtf(fbest)
                               : (!SAMP && d2 < 16777216.0) ? sqrt_rn_int(uint32_t(d2))
                                                            : float(sqrt(d2));
            if (a.dist) __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, dist), rd, li.y + ro, 0, 0);
            if (a.sq) __builtin_amdgcn_raw_buffer_store_b32(uint32_t(int32_t(d2)), rs, li.y + ro, 0, 0);
            return;
        }
        Line l;
        l.s = li.x;
        l.base = li.y;
        l.i = li.z;
        slice0 = a.idx + uint64_t(l.s) * a.cstride;
        const uint64_t e = uint64_t(l.base) + uint64_t(qr) * a.inner;   // in-sample flat
        if (!FINAL) {
            slice0[e] = site;
            return;
        }
        // final pass: coordinates, distance, squared distance (with the
        // carrier in a distance output, the distance replaces the carried
        // site in place: this workgroup staged every row of its lines)
        const float fbest = __builtin_bit_cast(float, best);
        double d2;
        if (site >= 0) {
            if (SAMP) d2 = double(fbest);
            else d2 = double(best >> a.rbits);
            if (a.coords) {
                uint32_t t2 = uint32_t(site);
#pragma unroll
                for (int b = kMaxDim - 1; b >= 0; --b) {
                    if (b < nd) {
                        if (b > 0) {
                            const uint32_t qd = a.div_shape[b].div(t2);
                            slice0[uint64_t(b) * a.vox + e] = int32_t(t2 - qd * a.div_shape[b].d);
                            t2 = qd;
                        } else {
                            slice0[e] = int32_t(t2);
                        }
                    }
                }
            }
        } else {
            // no background in the sample: the virtual element (-1, 0, ..., 0)
            d2 = virtual_d2(qr, l.i, line_pos0[ln]);
            if (a.coords) {
                slice0[e] = -1;
                for (int b = 1; b < nd; ++b) slice0[uint64_t(b) * a.vox + e] = 0;
            }
        }
        // A found site's sampled value is a float, and its correctly rounded
        // float root (sqrtf) equals the double root rounded to float, since
        // 53 >= 2 * 24 + 2; the virtual element's value takes the double root.
        const float dist = (SAMP && site >= 0)                ? sqrtf(fbest)
                           : (!SAMP && d2 < 16777216.0) ? sqrt_rn_int(uint32_t(d2))
                                                        : float(sqrt(d2));
        if (a.dist) a.dist[uint64_t(l.s) * a.vox + e] = dist;
        if (a.sq) a.sq[uint64_t(l.s) * a.vox + e] = int32_t(d2);
    };

    // ---- search and output, patch by patch ----------------------------------
    // Patch p = (row block rb = p / L, line block (p + rb) % L), with PL
    // lines (L = kIdxLines / PL line blocks) and PR = 128 / PL rows: lane l
    // takes rows PR rb + 2 (l / PL) and the next one of line PL cb + l % PL.
    //
    // The search runs in blocks of four steps d .. d+3.  For the lane's two
    // rows q and q + 1 a block reads rows q-d-3 .. q-d+1 and q+d .. q+d+4 at
    // fixed offsets from two LDS byte addresses that step by four rows per
    // block and are clamped to the first guard row above and the first one
    // below the line: a clamped block lies wholly past that end of the line,
    // where every candidate is "none" and the guard rows it then reads are
    // "none" too.  The candidate of step e is the smaller of the two rows at
    // distance e plus the weight of e (for unit keys the minimum of the two
    // keys, whose low bits keep the row).
    constexpr int kRB = kIdxRowW * 4;              // row stride in bytes
    constexpr int PL = idx_patch_lines(FAST);      // lines of a patch
    constexpr int PR = 2 * kWave / PL;             // rows of a patch
    const int pr = 2 * (lane / PL);
    constexpr int kLB = kIdxLines / PL;            // line blocks
    const int npatch = kLB * ((n + PR - 1) / PR);
    for (int p = wv; p < npatch; p += kIdxWaves) {
        const int rbk = p / kLB;
        const int ln = PL * ((p + rbk) % kLB) + (lane % PL);
        const bool has = (has_mask >> ln) & 1u;
        const int qr = PR * rbk + pr;                          // the lane's rows qr, qr + 1
        const int q = min(qr, n - 1);
        const int cb = int(lds_byte_addr(val0 + ln));          // row 0 of this lane's line
        const int lo_min = cb - kIdxGuard * kRB;               // first guard row above the line
        const uint32_t hi_max = uint32_t(cb + n * kRB);        // first guard row below it
        // best values (sampled: float bits, ordered as unsigned integers for
        // values >= 0) or keys of rows q and q + 1; nothing to find, or a row
        // past the line: 0, which stops at once
        uint32_t best[2];
        best[0] = has && qr < n ? lds_word(uint32_t(cb + q * kRB)) : 0u;
        best[1] = has && qr + 1 < n ? lds_word(uint32_t(cb + (q + 1) * kRB)) : 0u;
        int bd[2] = {0, 0};                                    // sampled: block of the best (0: own row)
        uint32_t cbk[2][4] = {};                               // sampled: that block's four candidates
        int lo = cb + (q - 4) * kRB;                           // row q - d - 3 at d = 1
        uint32_t hi = uint32_t(cb + (q + 1) * kRB);            // row q + d at d = 1
        // One block of four steps d .. d+3; true when the search is over.
        // Sampled: `cur` holds the block's weights, and `nxt` receives the
        // next block's (read one block early; the two registers alternate).
        auto block = [&](int d, const float4 &cur, float4 &nxt) -> bool {
            bool done;
            const uint32_t bmax = max(best[0], best[1]);
            if (SAMP) done = cur.x > __builtin_bit_cast(float, bmax);
            else done = (uint64_t(uint32_t(d) * uint32_t(d)) << a.rbits) > uint64_t(bmax);
            if (d > n || __all(done)) return true;
            const uint32_t lb = uint32_t(max(lo, lo_min)), hb = min(hi, hi_max);
            uint32_t U[5], W[5];
#pragma unroll
            for (int k = 0; k < 5; ++k) {
                U[k] = lds_word(lb + k * kRB);                 // row q - d - 3 + k
                W[k] = lds_word(hb + k * kRB);                 // row q + d + k
            }
            if constexpr (SAMP) {
                const float adk[4] = {cur.x, cur.y, cur.z, cur.w};
                nxt = *reinterpret_cast<const float4 *>(step + d + 4);
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    uint32_t c[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        c[k] = __builtin_bit_cast(uint32_t,
                                                  __builtin_bit_cast(float, min(U[3 + h - k], W[k + h])) + adk[k]);
                    const uint32_t m = min(min(c[0], c[1]), min(c[2], c[3]));
                    const bool imp = m < best[h];
                    bd[h] = imp ? d : bd[h];
#pragma unroll
                    for (int k = 0; k < 4; ++k) cbk[h][k] = imp ? c[k] : cbk[h][k];
                    best[h] = min(best[h], m);
                }
            } else {
                // "none" keys (0x7fffffff) plus a weight stay above every real
                // key, which is below 2^31 with its weight (no wrap: the
                // weights are below 2^31)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    uint32_t c[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        c[k] = min(U[3 + h - k], W[k + h]) + (uint32_t((d + k) * (d + k)) << a.rbits);
                    best[h] = min(best[h], min(min(c[0], c[1]), min(c[2], c[3])));
                }
            }
            lo -= 4 * kRB;
            hi += 4 * kRB;
            return false;
        };
        float4 adA = SAMP ? *reinterpret_cast<const float4 *>(step + 1) : float4{}, adB{};
        for (int d = 1;; d += 8) {
            if (block(d, adA, adB)) break;
            if (block(d + 4, adB, adA)) break;
        }
        for (int h = 0; h < 2; ++h) {
            const int qh = q + h;
            // sampled: the row of the best value.  Its step e = bd + k is the
            // first of the block's candidates equal to it; the row is qh - e
            // when that row's own candidate equals it (same operands, same
            // sum), else qh + e.  A row qh - e above the first guard row reads
            // that guard row ("none").
            int r_best = qh;
            if (SAMP && bd[h] > 0) {
                int k = 3;
#pragma unroll
                for (int j = 2; j >= 0; --j) k = cbk[h][j] == best[h] ? j : k;
                const int e = bd[h] + k;
                const float ce =
                    __builtin_bit_cast(float, lds_word(uint32_t(max(cb + (qh - e) * kRB, lo_min)))) + step[e];
                r_best = __builtin_bit_cast(uint32_t, ce) == best[h] ? qh - e : qh + e;
            }
            if (qr + h >= n) continue;
            output(qr + h, ln, has, best[h], r_best);
        }
    }
}

}  // namespace tmedt
