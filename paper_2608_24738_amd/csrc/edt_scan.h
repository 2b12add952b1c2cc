// edt_scan.h -- first pass of the separable EDT, along the contiguous last
// axis (paper, Section 2.3.2: one 1-D pass per axis; this one starts from a
// binary mask, so the lower envelope degenerates to "nearest zero in the
// line").
//
// Each wavefront owns a span of up to 1024 consecutive mask bytes.  Lane l
// holds the 16 positions 256k + 4l + j (k, j < 4), so every load instruction
// of the wave reads 256 contiguous bytes and every store writes 1 KiB
// contiguous.  The nearest zero on each side comes from per-lane 4-bit zero
// masks, a wave-wide inclusive prefix-max (last zero so far) and suffix-min
// (first zero from here), and carries across the four groups.  Ties between
// an equally distant left and right zero go to the left (smaller) one.
#pragma once

#include "edt_common.h"

namespace tmedt {

enum ScanMode : int {
    kScanFieldInt = 0,   // int32 squared distance, kInfI if the line has no zero
    kScanFieldFlt = 1,   // float w * squared distance, +inf if none
    kScanIndex = 2,      // int32 in-sample flat index of the zero, -1 if none
    kScanFinal = 3,      // rank-1 input: the line is the sample; final outputs
    kScanFieldL1 = 4     // int32 distance (taxicab / chessboard first pass), kInfI if none
};

struct ScanArgs {
    const uint8_t *in;
    uint32_t n;            // line length
    uint32_t lines;        // lines in the batch (batch * voxels / n)
    uint32_t span_lines;   // whole lines per wavefront span (n <= 1024)
    uint32_t lps;          // lines per sample
    Div32 div_n;           // span-relative position -> line
    Div32 div_lps;         // line -> sample
    uint32_t vox;          // elements per sample
    int32_t ndim;
    double w;              // squared sampling of the last axis
    int32_t *field_i;      // kScanFieldInt output (batch-flat)
    float *field_f;        // kScanFieldFlt output (batch-flat)
    int32_t *idx;          // kScanIndex: the carrier, cstride elements per sample (slice 0 of
                           // [batch][ndim][vox], or a distance output holding flat indices);
                           // kScanFinal: coords
    uint64_t cstride;      // kScanIndex: carrier elements per sample
    float *dist;           // kScanFinal outputs (each may be null)
    int32_t *sq;
};

constexpr int kBig = 0x3fffffff;

// Left/right zero candidates for the 16 positions a lane holds in one 1024-
// position chunk.  zb[k] bit j marks a zero at chunk position 256k + 4l + j.
// cl / cr: last zero before / first zero after the chunk (chunk-relative,
// -kBig / kBig when none).  Outputs chunk-relative candidates (-kBig / kBig
// when none).
__device__ inline void chunk_candidates(const uint32_t zb[4], int cl, int cr, int lane,
                                        int left[4][4], int right[4][4]) {
    int pl[4], sf[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        int base = 256 * k + 4 * lane;
        pl[k] = zb[k] ? base + 31 - __clz(zb[k]) : -kBig;
        sf[k] = zb[k] ? base + __ffs(zb[k]) - 1 : kBig;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            int t = __shfl_up(pl[k], d, kWave);
            if (lane >= d) pl[k] = max(pl[k], t);
            int u = __shfl_down(sf[k], d, kWave);
            if (lane + d < kWave) sf[k] = min(sf[k], u);
        }
    }
    int exl[4], exr[4];
    int carry = cl;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        int t = __shfl_up(pl[k], 1, kWave);
        exl[k] = max(lane == 0 ? -kBig : t, carry);
        carry = max(carry, __shfl(pl[k], kWave - 1, kWave));
    }
    carry = cr;
#pragma unroll
    for (int k = 3; k >= 0; --k) {
        int t = __shfl_down(sf[k], 1, kWave);
        exr[k] = min(lane == kWave - 1 ? kBig : t, carry);
        carry = min(carry, __shfl(sf[k], 0, kWave));
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        int base = 256 * k + 4 * lane;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t lo = zb[k] & ((2u << j) - 1u);
            left[k][j] = lo ? base + 31 - __clz(lo) : exl[k];
            uint32_t hi = zb[k] >> j;
            right[k][j] = hi ? base + j + __ffs(hi) - 1 : exr[k];
        }
    }
}

// Zero masks of one chunk: positions >= valid read as foreground.
template <bool VEC>
__device__ inline void load_zero_bits(const uint8_t *p, int valid, int lane, uint32_t zb[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        int base = 256 * k + 4 * lane;
        uint32_t bits = 0;
        if (VEC) {
            uint32_t word = *reinterpret_cast<const uint32_t *>(p + base);
#pragma unroll
            for (int j = 0; j < 4; ++j) bits |= ((word >> (8 * j)) & 0xffu) == 0 ? (1u << j) : 0u;
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (base + j < valid && p[base + j] == 0) bits |= 1u << j;
        }
        zb[k] = bits;
    }
}

// Writes the results of four consecutive positions (x0 .. x0+3 of one line,
// line-relative; y[j] = line-relative zero or -1) for line `gline`.
template <int MODE, bool VEC>
__device__ inline void scan_store4(const ScanArgs &a, uint32_t gline, int x0, const int y[4],
                                   int count) {
    const uint64_t lbase = uint64_t(gline) * a.n;  // batch-flat start of the line
    if (MODE == kScanFieldInt || MODE == kScanFieldL1) {
        int32_t v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int d = x0 + j - y[j];
            if (MODE == kScanFieldL1) d = d < 0 ? -d : d;
            v[j] = y[j] >= 0 ? (MODE == kScanFieldL1 ? d : d * d) : kInfI;
        }
        int32_t *o = a.field_i + lbase + x0;
        if (VEC) {
            *reinterpret_cast<int4 *>(o) = make_int4(v[0], v[1], v[2], v[3]);
        } else {
            for (int j = 0; j < count; ++j) o[j] = v[j];
        }
    } else if (MODE == kScanFieldFlt) {
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            double d = double(x0 + j - y[j]);
            v[j] = y[j] >= 0 ? float(a.w * (d * d)) : __builtin_inff();
        }
        float *o = a.field_f + lbase + x0;
        if (VEC) {
            *reinterpret_cast<float4 *>(o) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
            for (int j = 0; j < count; ++j) o[j] = v[j];
        }
    } else if (MODE == kScanIndex) {
        uint32_t s = a.div_lps.div(gline);
        uint32_t lline = gline - s * a.lps;
        uint64_t local = uint64_t(lline) * a.n;
        int32_t v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = y[j] >= 0 ? int32_t(local + y[j]) : kNoIdx;
        int32_t *o = a.idx + uint64_t(s) * a.cstride + local + x0;
        if (VEC) {
            *reinterpret_cast<int4 *>(o) = make_int4(v[0], v[1], v[2], v[3]);
        } else {
            for (int j = 0; j < count; ++j) o[j] = v[j];
        }
    } else {  // kScanFinal: rank 1, the line is the whole sample
        for (int j = 0; j < count; ++j) {
            int x = x0 + j;
            double d = y[j] >= 0 ? double(x - y[j]) : double(x + 1);  // virtual zero at -1
            if (a.dist) a.dist[lbase + x] = float(sqrt(a.w * (d * d)));
            if (a.sq) {
                int64_t di = y[j] >= 0 ? int64_t(x - y[j]) : int64_t(x + 1);
                a.sq[lbase + x] = int32_t(di * di);
            }
            if (a.idx) a.idx[lbase + x] = y[j] >= 0 ? y[j] : -1;
        }
    }
}

// Lines of length n <= 1024: each wavefront scans `span_lines` whole lines.
template <int MODE, bool VEC>
__global__ void __launch_bounds__(256) k_scan_span(ScanArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const uint32_t wave = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    const uint64_t line0 = uint64_t(wave) * a.span_lines;
    if (line0 >= a.lines) return;  // whole wavefront exits together
    const uint32_t nl = uint32_t(min<uint64_t>(a.span_lines, a.lines - line0));
    const int valid = int(nl * a.n);
    const uint8_t *src = a.in + line0 * a.n;
    const bool full = VEC && valid == kSpan;

    uint32_t zb[4];
    if (full) load_zero_bits<true>(src, valid, lane, zb);
    else load_zero_bits<false>(src, valid, lane, zb);
    int left[4][4], right[4][4];
    chunk_candidates(zb, -kBig, kBig, lane, left, right);

#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int p0 = 256 * k + 4 * lane;  // span position of the group's first element
        if (p0 >= valid) continue;
        // With n % 4 == 0 (vector path) the four positions share one line.
        int y[4];
        uint32_t line_of[4];
        int xs[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int p = p0 + j;
            uint32_t l = a.div_n.div(uint32_t(p));
            int ls = int(l * a.n);
            int le = ls + int(a.n);
            bool hl = left[k][j] >= ls;
            bool hr = right[k][j] < le && right[k][j] < valid;
            int yy = -1;
            if (hl && (!hr || p - left[k][j] <= right[k][j] - p)) yy = left[k][j] - ls;
            else if (hr) yy = right[k][j] - ls;
            y[j] = yy;
            line_of[j] = l;
            xs[j] = p - ls;
        }
        if (full) {
            scan_store4<MODE, true>(a, uint32_t(line0) + line_of[0], xs[0], y, 4);
        } else {
            for (int j = 0; j < 4; ++j) {
                if (p0 + j >= valid) break;
                int yy[4] = {y[j], -1, -1, -1};
                scan_store4<MODE, false>(a, uint32_t(line0) + line_of[j], xs[j], yy, 1);
            }
        }
    }
}

// The 32-bit output word of position x of line `gline` (the first output
// present in the rank-1 case).
template <int MODE>
__device__ inline uint32_t *scan_slot(const ScanArgs &a, uint32_t gline, int x) {
    const uint64_t lbase = uint64_t(gline) * a.n;
    if (MODE == kScanFieldInt || MODE == kScanFieldL1) return reinterpret_cast<uint32_t *>(a.field_i + lbase + x);
    if (MODE == kScanFieldFlt) return reinterpret_cast<uint32_t *>(a.field_f + lbase + x);
    if (MODE == kScanIndex) {
        const uint32_t s = a.div_lps.div(gline);
        const uint64_t local = uint64_t(gline - s * a.lps) * a.n;
        return reinterpret_cast<uint32_t *>(a.idx + uint64_t(s) * a.cstride + local + x);
    }
    if (a.dist) return reinterpret_cast<uint32_t *>(a.dist + lbase + x);
    if (a.sq) return reinterpret_cast<uint32_t *>(a.sq + lbase + x);
    return reinterpret_cast<uint32_t *>(a.idx + lbase + x);
}

// Lines longer than 1024: one wavefront per line, two sweeps over 1024-
// position chunks.  The first (right to left) finds, per chunk, the first
// zero at or after the chunk start and parks it in the output word of the
// chunk's first position (every lane writes the same value there, and reads
// it back itself); the second (left to right) carries the last zero seen and
// reads the right carry of the next chunk before this chunk's results are
// stored.  Lines of any length, no workspace.
template <int MODE>
__global__ void __launch_bounds__(64) k_scan_long(ScanArgs a) {
    const int lane = threadIdx.x;
    const uint32_t gline = blockIdx.x;
    const uint8_t *src = a.in + uint64_t(gline) * a.n;
    const int n = int(a.n);
    const int chunks = (n + kSpan - 1) / kSpan;
    int carry = kBig;
    for (int c = chunks - 1; c >= 0; --c) {
        const int valid = min(kSpan, n - c * kSpan);
        uint32_t zb[4];
        load_zero_bits<false>(src + c * kSpan, valid, lane, zb);
        int m = kBig;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (zb[k]) m = min(m, c * kSpan + 256 * k + 4 * lane + __ffs(zb[k]) - 1);
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) m = min(m, __shfl_xor(m, d, kWave));
        carry = min(carry, m);
        if (c >= 1) *scan_slot<MODE>(a, gline, c * kSpan) = uint32_t(carry);
    }
    int last = -kBig;  // last zero before the current chunk (line-relative)
    for (int c = 0; c < chunks; ++c) {
        const int valid = min(kSpan, n - c * kSpan);
        const int off = c * kSpan;
        uint32_t zb[4];
        load_zero_bits<false>(src + off, valid, lane, zb);
        const int cl = last == -kBig ? -kBig : last - off;
        const int nxt = c + 1 < chunks ? int(*scan_slot<MODE>(a, gline, (c + 1) * kSpan)) : kBig;
        const int cr = nxt == kBig ? kBig : nxt - off;
        int left[4][4], right[4][4];
        chunk_candidates(zb, cl, cr, lane, left, right);
        int m = -kBig;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (zb[k]) m = max(m, off + 256 * k + 4 * lane + 31 - __clz(zb[k]));
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) m = max(m, __shfl_xor(m, d, kWave));
        last = max(last, m);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int p0 = 256 * k + 4 * lane;
            for (int j = 0; j < 4; ++j) {
                const int p = p0 + j;
                if (p >= valid) break;
                const int l = left[k][j], r = right[k][j];
                const bool hl = l > -kBig;
                const bool hr = r < kBig;
                int yy = -1;
                if (hl && (!hr || p - l <= r - p)) yy = l + off;
                else if (hr) yy = r + off;
                int ys[4] = {yy, -1, -1, -1};
                scan_store4<MODE, false>(a, gline, p + off, ys, 1);
            }
        }
    }
}

}  // namespace tmedt

namespace tmedt {

// ---------------------------------------------------------------------------
// Lines whose length is a multiple of WB (64, or 32 to run twice as many
// wavefronts on short batches): one lane per WB-position word.  A wavefront
// holds 64 / words-per-line whole lines (lanes past them idle).  Each lane
// loads its WB mask bytes (16-byte loads), builds the zero mask, takes the
// last zero of the earlier words and the first zero of the later words of
// its line from two segmented wave scans, then walks its WB positions left
// to right (distance to the last zero) and right to left (distance to the
// next zero), keeping the left zero on ties.
//
// COST = CW > 0 (unit or chamfer field output, when the next pass is the
// final column pass of a 2-D input, dispatched in an order kept in a
// workspace: k_line_pair16, whose groups are 16 columns, or k_line_search,
// whose units are four workgroups of 8 columns, 32): the scan also estimates that pass's work per
// group of CW columns, as the sum over every fourth element of the group of
// min(d, 128), d the distance just found along the row.  The
// column search from an element runs as far as its final distance, which d
// bounds from above, so groups crossing large foreground regions sum high.
// Words per line divide 64 and the four waves of a workgroup hold rows of one
// sample (the host checks both),
// reduce their sums in LDS after their stores, and add them to the group's
// counter with one relaxed device-scope atomic per group (k_order, next,
// turns the counters into the column pass's order).
// ---------------------------------------------------------------------------
struct WordScanArgs {
    const uint8_t *in;
    uint32_t n;            // line length, a multiple of the word size WB
    uint32_t nw;           // words per line = n / WB (<= 64)
    uint32_t lpw;          // whole lines per wavefront = 64 / nw
    uint64_t lines;        // lines in the batch
    uint32_t lps;          // lines per sample
    uint32_t vox;          // elements per sample
    int32_t ndim;
    double w;              // squared sampling of the last axis
    int32_t *field_i;      // kScanFieldInt output
    float *field_f;        // kScanFieldFlt output
    int32_t *idx;          // kScanIndex: the carrier (see ScanArgs); kScanFinal: coords
    uint64_t cstride;      // kScanIndex: carrier elements per sample
    float *dist;           // kScanFinal outputs (each may be null)
    int32_t *sq;
    uint32_t *cost;        // CW > 0: one counter per group of CW columns, [sample][n / CW]
    uint32_t rows;         // CW > 0: rows per sample, a multiple of 4 lpw
    uint32_t n1;           // PKW > 0: extent of the next axis (rows of a strip), a multiple of lpw
};

template <int MODE, int WB, int CW = 0, int PKW = 0>
__global__ void __launch_bounds__(256) k_scan_word(WordScanArgs a) {
    constexpr bool COST = CW > 0;
    constexpr bool PK = PKW > 0;
    static_assert(!PK || MODE == kScanFieldInt || MODE == kScanFieldL1,
                  "the packed field holds distances along the row (unit or chamfer)");
    static_assert(PKW == 0 || PKW == 8 || PKW == 16, "strips of 8 or 16 columns");
    static_assert(!COST || MODE == kScanFieldInt || MODE == kScanFieldL1,
                  "the cost estimate comes with the unit field or the chamfer field");
    static_assert(CW == 0 || CW == 16 || CW == 32, "groups of 16 or 32 columns");
    constexpr int kCG = COST ? WB / CW : 1;     // groups per lane word
    static_assert(WB == 32 || WB == 64, "a word holds 32 or 64 positions");
    const int lane = threadIdx.x & (kWave - 1);
    const uint64_t wave = uint64_t(blockIdx.x) * (blockDim.x / kWave) + threadIdx.x / kWave;
    const int nw = int(a.nw);
    const int lw = lane / nw;                 // line within the wavefront
    const int w = lane - lw * nw;             // word within the line
    const uint64_t line = wave * a.lpw + lw;
    const bool live = lw < int(a.lpw) && line < a.lines;
    if (wave * a.lpw >= a.lines) return;      // whole wavefront exits together
    // kScanIndex: sample of the line and the line's first in-sample position
    // (the 64-bit division runs here, while few registers are live)
    const uint64_t smp = MODE == kScanIndex ? line / a.lps : 0;
    const uint32_t local = MODE == kScanIndex ? uint32_t(line - smp * a.lps) * a.n : 0;

    // ---- zero mask of this lane's WB positions ---------------------------
    const uint64_t pos0 = line * a.n + uint64_t(w) * WB;   // batch-flat first position
    uint64_t mask = 0;
    if (live) {
        const uint4 *src = reinterpret_cast<const uint4 *>(a.in + pos0);
        uint4 v[WB / 16];
#pragma unroll
        for (int k = 0; k < WB / 16; ++k) v[k] = src[k];
#pragma unroll
        for (int k = 0; k < WB / 16; ++k) {
            const uint32_t d4[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                // 0x80 in every zero byte (exact: no carries between bytes)
                const uint32_t x = d4[c];
                const uint32_t zb = ~(((x & 0x7f7f7f7fu) + 0x7f7f7f7fu) | x | 0x7f7f7f7fu);
                // gather bits 7, 15, 23, 31 into a nibble
                const uint32_t nib = ((zb >> 7) & 1u) | ((zb >> 14) & 2u) | ((zb >> 21) & 4u) | ((zb >> 28) & 8u);
                mask |= uint64_t(nib) << (16 * k + 4 * c);
            }
        }
    }

    // ---- nearest zero in the other words of the line ---------------------
    // Keys carry the line within the wavefront in their high bits so that a
    // plain wave-wide max / min never mixes two lines.
    const int base = w * WB;
    const uint32_t hi = uint32_t(lw) << 16;
    const uint32_t own_last = mask ? hi | uint32_t(base + 63 - __clzll(mask) + 1) : hi;
    const uint32_t own_first = mask ? hi | uint32_t(base + __ffsll((unsigned long long)mask) - 1) : hi | 0xffffu;
    uint32_t pm = own_last, sm = own_first;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t u = __shfl_up(pm, d, kWave);
        if (lane >= d) pm = max(pm, u);
        const uint32_t v = __shfl_down(sm, d, kWave);
        if (lane + d < kWave) sm = min(sm, v);
    }
    uint32_t before = __shfl_up(pm, 1, kWave);   // words < w of the line
    uint32_t after = __shfl_down(sm, 1, kWave);  // words > w of the line
    if (w == 0 || (before >> 16) != uint32_t(lw)) before = hi;
    if (w == nw - 1 || (after >> 16) != uint32_t(lw)) after = hi | 0xffffu;
    constexpr int kFar = 1 << 20;
    int last = (before & 0xffffu) ? int(before & 0xffffu) - 1 : -kFar;  // line-relative
    int next = (after & 0xffffu) != 0xffffu ? int(after & 0xffffu) : kFar;

    // ---- per-position distances -------------------------------------------
    int dl[WB];
#pragma unroll
    for (int p = 0; p < WB; ++p) {
        if ((mask >> p) & 1ull) last = base + p;
        dl[p] = last;             // last zero at or before base + p
    }
    int32_t out[WB];
    uint32_t csum[kCG] = {};          // COST: this lane's share of its groups' sums
#pragma unroll
    for (int p = WB - 1; p >= 0; --p) {
        if ((mask >> p) & 1ull) next = base + p;
        const int x = base + p;
        const int l = x - dl[p], r = next - x;   // l, r >= 0
        const bool left = l <= r;
        const int dd = left ? l : r;
        if (COST && p % 4 == 0) csum[p / (COST ? CW : 1)] += uint32_t(min(dd, 128));
        const int y = left ? dl[p] : next;        // line-relative zero, valid if dd < kFar / 2
        const bool none = dd >= kFar / 2;
        if (PK) {
            out[p] = none ? 0xffff : dd;
        } else if (MODE == kScanFieldInt || MODE == kScanFieldL1) {
            out[p] = none ? kInfI : (MODE == kScanFieldL1 ? dd : dd * dd);
        } else if (MODE == kScanFieldFlt) {
            const double df = double(dd);
            out[p] = none ? __builtin_bit_cast(int32_t, __builtin_inff())
                          : __builtin_bit_cast(int32_t, float(a.w * (df * df)));
        } else if (MODE == kScanIndex) {
            out[p] = none ? kNoIdx : int32_t(local + y);
        } else {
            out[p] = none ? -1 : y;   // kScanFinal: the line is the sample
        }
    }
    // ---- stores -------------------------------------------------------------
    if (MODE != kScanFinal) {
        // A lane's WB results are 4 WB contiguous bytes.  Written straight
        // from registers, each store instruction of the wave would touch 64
        // separate 16-byte pieces; instead they pass through LDS in halves
        // of 32 results, so that each store instruction writes 8 whole
        // 128-byte segments (a half of each of 8 lanes).  The destinations of the
        // lanes' results go through LDS as well: index slices of different
        // samples are not adjacent.
        constexpr int kPad = 9;                                   // int4 per lane row: 8 + 1 pad
        __shared__ int4 stage[256 / kWave][kWave * kPad];
        __shared__ uint64_t dest[256 / kWave][kWave];
        int4 *st = stage[threadIdx.x / kWave];
        uint64_t *ds = dest[threadIdx.x / kWave];
        int32_t *db;
        uint64_t own;
        if (MODE == kScanIndex) {
            db = a.idx;
            own = smp * a.cstride + local + uint64_t(w) * WB;
        } else {
            db = MODE == kScanFieldFlt ? reinterpret_cast<int32_t *>(a.field_f) : a.field_i;
            own = pos0;
        }
        if constexpr (PK) {
            // Packed field: per strip of PKW columns, row R of the int32
            // layout (4 PKW bytes) holds the distances of rows 2R and 2R + 1
            // (0xffff: no zero in the line) as 16-bit pairs of adjacent
            // columns, row 2R in its first half.  The wave's lpw rows (even,
            // inside one block of n1 rows) fill lpw / 2 int32 rows, one
            // contiguous run of 32 WB words; a lane's four-word pieces go to LDS
            // at their place in the run (one pad piece per eight) and each
            // store instruction then writes 1 KiB of it.
            const uint32_t rb = uint32_t(lw >> 1) * a.n + uint32_t(w) * WB + uint32_t(PKW / 2) * uint32_t(lw & 1);
#pragma unroll
            for (int k = 0; k < (PK ? WB / PKW : 0); ++k) {
#pragma unroll
                for (int j = 0; j < PKW / 8; ++j) {
                    const int p0 = PKW * k + 8 * j;
                    auto pair = [&](int q) { return int32_t(uint32_t(out[q]) | (uint32_t(out[q + 1]) << 16)); };
                    const int4 v = make_int4(pair(p0), pair(p0 + 2), pair(p0 + 4), pair(p0 + 6));
                    const uint32_t c = (rb + uint32_t(PKW * k + 4 * j)) / 4u;  // strip k: PKW words
                    st[c + c / 8] = v;
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const uint64_t l0 = wave * a.lpw;
            const uint64_t blk = l0 / a.n1;
            int4 *dst = reinterpret_cast<int4 *>(a.field_i + (blk * a.n1 + (l0 - blk * a.n1) / 2) * a.n);
#pragma unroll
            for (int i = 0; i < WB / 8; ++i) {
                const int c = lane + kWave * i;
                dst[c] = st[c + c / 8];
            }
        }
        if (!PK) ds[lane] = live ? own : ~0ull;
        const int src = lane >> 3, piece = lane & 7;
#pragma unroll
        for (int h = PK ? -1 : WB / 32 - 1; h >= 0; --h) {      // the later half is ready first
#pragma unroll
            for (int i = 0; i < 8; ++i)
                st[lane * kPad + i] = make_int4(out[32 * h + 4 * i], out[32 * h + 4 * i + 1],
                                                out[32 * h + 4 * i + 2], out[32 * h + 4 * i + 3]);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int sl = 8 * k + src;                       // source lane
                const uint64_t o = ds[sl];
                const int4 v = st[sl * kPad + piece];
                if (o != ~0ull) *reinterpret_cast<int4 *>(db + o + 32 * h + 4 * piece) = v;
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        if (COST) {
            // sums over the wave's lines (lanes w, w + nw, ...), then over the
            // workgroup's waves, all of one sample: one atomic per group
            __shared__ uint32_t cs[256 / kWave][kWave * 4];
#pragma unroll
            for (int k = 0; k < kCG; ++k) {
                uint32_t v = live ? csum[k] : 0u;
                for (int d = nw; d < kWave; d <<= 1) v += __shfl_xor(v, d, kWave);
                if (lw == 0) cs[threadIdx.x / kWave][w * kCG + k] = v;
            }
            __syncthreads();
            const uint32_t ng = a.n / uint32_t(COST ? CW : 1), t = threadIdx.x;
            if (t < ng) {
                const uint32_t smp_c = uint32_t(uint64_t(blockIdx.x) * (256 / kWave) * a.lpw / a.rows);
                __hip_atomic_fetch_add(a.cost + uint64_t(smp_c) * ng + t, cs[0][t] + cs[1][t] + cs[2][t] + cs[3][t],
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    } else {
        if (!live) return;
        // rank 1: a line without any zero measures from the virtual zero at -1
#pragma unroll
        for (int p = 0; p < WB; ++p) {
            const int x = base + p;
            const int y = out[p];
            const int64_t dd = y >= 0 ? int64_t(x - y) : int64_t(x + 1);
            const uint64_t g = pos0 + p;
            if (a.dist) a.dist[g] = float(sqrt(a.w * double(dd * dd)));
            if (a.sq) a.sq[g] = int32_t(dd * dd);
            if (a.idx) a.idx[g] = y;
        }
    }
}

}  // namespace tmedt

namespace tmedt {

// ---------------------------------------------------------------------------
// First pass of the signed transform EDT(M) - EDT(not M): every element
// measures to the nearest element of the other class along its line, and
// the field keeps one signed squared distance per element, +F for
// foreground (distance to background) and -F for background (distance to
// foreground), +-kInfI when the line has no element of the other class.
// Zero never occurs, since an element is never a site of its own field.
//
// One wavefront per line, in 64-position chunks: two ballots mark the
// chunk's background and foreground positions; a forward sweep carries the
// last position of each class, a backward sweep the next one.  Lines of up
// to kSignedRegChunks chunks keep the ballots and left candidates in
// registers; longer lines park the left candidate in the output between the
// sweeps (each lane rereads only what it wrote).
// Rank 1 (FINAL): the line is the sample; the outputs are float distances
// with the class sign, from the virtual element (-1) when the sample holds
// one class only.
// ---------------------------------------------------------------------------
constexpr int kSignedRegChunks = 16;

struct SignedScanArgs {
    const uint8_t *in;
    int32_t *field;        // signed squared distances (intermediate output)
    float *dist;           // rank 1: signed distances
    uint32_t n;            // line length
    uint32_t lines;
};

template <bool LONG, bool FINAL>
__global__ void __launch_bounds__(256) k_scan_signed(SignedScanArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const uint32_t line = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (line >= a.lines) return;                       // whole wavefront exits together
    const int n = int(a.n);
    const uint8_t *src = a.in + uint64_t(line) * a.n;
    int32_t *fld = a.field + uint64_t(line) * a.n;
    constexpr int kFar = 1 << 30;
    const int nc = (n + kWave - 1) / kWave;
    const uint64_t le = lane == kWave - 1 ? ~0ull : (2ull << lane) - 1ull;   // positions <= lane
    constexpr int RC = LONG ? 1 : kSignedRegChunks;
    uint64_t zs[RC], os[RC];
    int lcand[RC];
    auto chunk = [&](int c, uint64_t &z, uint64_t &o, bool &fg) {
        const int pos = c * kWave + lane;
        const bool valid = pos < n;
        const uint8_t b = valid ? src[pos] : 0;
        z = __ballot(valid && b == 0);
        o = __ballot(valid && b != 0);
        fg = valid && b != 0;
    };
    // ---- forward: last element of the other class at or before each position
    int lz = -kFar, lo = -kFar;                        // last background / foreground so far
    auto forward = [&](int c, uint64_t &z, uint64_t &o) {
        bool fg;
        chunk(c, z, o, fg);
        const uint64_t opp = (fg ? z : o) & le;
        const int left = opp ? c * kWave + 63 - __clzll(opp) : (fg ? lz : lo);
        if (z) lz = c * kWave + 63 - __clzll(z);
        if (o) lo = c * kWave + 63 - __clzll(o);
        return left;
    };
    if (LONG) {
        for (int c = 0; c < nc; ++c) {
            uint64_t z, o;
            const int left = forward(c, z, o);
            if (c * kWave + lane < n) fld[c * kWave + lane] = left;
        }
    } else {
#pragma unroll
        for (int c = 0; c < RC; ++c)
            if (c < nc) lcand[c] = forward(c, zs[c], os[c]);
    }
    // ---- backward: next element of the other class, then the values
    int nz = kFar, no = kFar;                          // next background / foreground
    auto finish = [&](int c, uint64_t z, uint64_t o, int left) {
        const int pos = c * kWave + lane;
        const bool fg = (o >> lane) & 1ull;
        const uint64_t opp = (fg ? z : o) >> lane;
        const int right = opp ? pos + __ffsll((unsigned long long)opp) - 1 : (fg ? nz : no);
        if (z) nz = c * kWave + __ffsll((unsigned long long)z) - 1;
        if (o) no = c * kWave + __ffsll((unsigned long long)o) - 1;
        if (pos >= n) return;
        const int dl = left > -kFar ? pos - left : kFar, dr = right < kFar ? right - pos : kFar;
        const int d = min(dl, dr);
        if (!FINAL) {
            const int32_t v = d < kFar ? d * d : kInfI;
            fld[pos] = fg ? v : -v;
        } else {
            const float dv = d < kFar ? float(d) : float(pos + 1);   // virtual element at -1
            a.dist[uint64_t(line) * a.n + pos] = fg ? dv : -dv;
        }
    };
    if (LONG) {
        for (int c = nc - 1; c >= 0; --c) {
            uint64_t z, o;
            bool fg;
            chunk(c, z, o, fg);
            const int left = c * kWave + lane < n ? fld[c * kWave + lane] : 0;
            finish(c, z, o, left);
        }
    } else {
#pragma unroll
        for (int c = RC - 1; c >= 0; --c)
            if (c < nc) finish(c, zs[c], os[c], lcand[c]);
    }
}

}  // namespace tmedt
