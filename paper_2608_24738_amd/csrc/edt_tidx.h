// Tiled pass on the index carrier: nearest background elements (and, on the
// last pass, distances and coordinates) for unit or anisotropic sampling.
//
// A workgroup owns 64 adjacent lines of one pass.  It stages, per line and
// row, the carried site (the in-sample flat index of the nearest background
// element found by the earlier passes, -1 for none) and the site's squared
// distance over the axes already processed, recomputed from the site's
// coordinates.  Each element then runs the windowed exact search over the
// rows of its line: examine rows at growing distance d and stop once
// w d^2 exceeds the best value found.  The winner's site comes from the
// staged copy, so the pass can overwrite its lines in place.
//
// Unit sampling: values are exact integers and a candidate is the key
// (value << RB) | row, so one integer minimum picks the smallest value and,
// among equal values, the smallest row: the canonical choice of the
// separable method (smallest flat index among nearest elements).
// Sampled: values are float, w = s_a^2; ties keep the first candidate met
// (any nearest element is correct there).
#pragma once

#include "edt_fh.h"

namespace tmedt {

constexpr int kIdxWaves = 16;
constexpr int kIdxGuard = 4;       // guard rows of "no site" per side
constexpr int kIdxRowW = kWave + 8;  // padded row stride (words)
constexpr int kIdxPatch = 8;       // patch: 8 rows x 8 lines

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
};

// LDS words of the two tile arrays for lines of n rows.
__host__ __device__ constexpr uint32_t idx_tile_words(uint32_t n) { return (n + 2 * kIdxGuard) * kIdxRowW; }

// Sampled search blocks BLK .. NBLK-1 (four steps each, unrolled at compile
// time): candidates f(q -+ d) + w d^2 at immediate LDS offsets from `pb`,
// the word of row q - 4 NBLK (every read stays in the tile).  Keeps the
// first strictly smaller candidate and its row offset; ends early once every
// lane of the wave has w d^2 above its best value.
template <int BLK, int NBLK>
__device__ __forceinline__ void search_samp(const uint32_t *pb, float w, float &fbest, int &roff, int &dnext) {
    if constexpr (BLK < NBLK) {
        constexpr int d = 1 + 4 * BLK;
        constexpr int R = 4 * NBLK;
        if (__all(w * float(d * d) > fbest)) return;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int dd = d + s;
            const float add = w * float(dd * dd);
            const float cu = __builtin_bit_cast(float, pb[(R - dd) * kIdxRowW]) + add;
            const float cv = __builtin_bit_cast(float, pb[(R + dd) * kIdxRowW]) + add;
            if (cu < fbest) {
                fbest = cu;
                roff = -dd;
            }
            if (cv < fbest) {
                fbest = cv;
                roff = dd;
            }
        }
        dnext = d + 4;
        search_samp<BLK + 1, NBLK>(pb, w, fbest, roff, dnext);
    }
}

template <bool SAMP, bool FINAL>
__global__ void __launch_bounds__(kWave * kIdxWaves) k_tile_idx(IdxTileArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    __shared__ __attribute__((aligned(16))) uint8_t any_site[kWave][kIdxWaves];   // [line][wave]
    __shared__ uint4 line_info[kWave];     // per line: sample, base of row 0, position i, live
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(t / kWave);
    const int n = int(a.n);
    const int nd = a.ndim;
    const int ax = a.axis;
    const uint32_t tw = idx_tile_words(uint32_t(n));
    uint32_t *val0 = lds + kIdxGuard * kIdxRowW;             // row 0 of the values / keys
    int32_t *site0 = reinterpret_cast<int32_t *>(lds + tw) + kIdxGuard * kIdxRowW;   // row 0 of the sites
    const uint32_t L0 = blockIdx.x * uint32_t(kWave);

    // Line j of the workgroup: sample, base of the line in slice 0, position
    // along the later axes.
    struct Line {
        bool live;
        uint32_t s, base, i;
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
        l.base = o * a.n * a.inner + l.i;       // in-sample flat of row 0
        return l;
    };
    // Coordinates along the axes after `ax` of the position i of this lane's
    // line (staging), computed once.
    int xc[kMaxDim] = {};
    float wf[kMaxDim] = {};
    auto line_coords = [&](uint32_t xi) {
#pragma unroll
        for (int b = kMaxDim - 1; b >= 0; --b) {
            if (b > ax && b < nd) {
                const uint32_t qx = a.div_shape[b].div(xi);
                xc[b] = int(xi - qx * a.div_shape[b].d);
                wf[b] = float(a.wall[b]);
                xi = qx;
            }
        }
    };
    // squared distance over the axes after `ax` between this lane's line and
    // site y (in-sample flat), or "none" (sampled: float sum of the exact
    // integer squares times the squared sampling)
    auto carried = [&](int32_t y, uint32_t &key_or_bits, int q) {
        if (y < 0) {
            key_or_bits = SAMP ? __builtin_bit_cast(uint32_t, __builtin_inff()) : uint32_t(kInfI);
            return;
        }
        uint32_t yi = a.div_inner.div(uint32_t(y));
        yi = uint32_t(y) - yi * a.inner;               // site position along the later axes
        float accf = 0.0f;
        uint32_t acci = 0;
#pragma unroll
        for (int b = kMaxDim - 1; b >= 0; --b) {
            if (b > ax && b < nd) {
                const uint32_t qy = a.div_shape[b].div(yi);
                const int dy = int(yi - qy * a.div_shape[b].d) - xc[b];
                yi = qy;
                if (SAMP) accf += wf[b] * float(dy * dy);
                else acci += uint32_t(dy * dy);
            }
        }
        key_or_bits = SAMP ? __builtin_bit_cast(uint32_t, accf) : ((acci << a.rbits) | uint32_t(q));
    };

    // ---- guard rows and staging ---------------------------------------------
    for (int k = t; k < kIdxGuard * kIdxRowW; k += kWave * kIdxWaves) {
        const uint32_t none = SAMP ? __builtin_bit_cast(uint32_t, __builtin_inff()) : uint32_t(kInfI);
        lds[k] = none;
        val0[n * kIdxRowW + k] = none;
    }
    const Line me = line_of(lane);
    if (wv == 0) line_info[lane] = uint4{me.s, me.base, me.i, me.live ? 1u : 0u};
    line_coords(me.i);
    const int32_t *src = a.idx + uint64_t(me.s) * a.cstride + me.base;
    uint32_t seen = 0;
    constexpr int SB = 8;
    for (int q0 = wv; q0 < n; q0 += kIdxWaves * SB) {
        int32_t y[SB];
#pragma unroll
        for (int j = 0; j < SB; ++j) y[j] = src[uint64_t(min(q0 + j * kIdxWaves, n - 1)) * a.inner];
#pragma unroll
        for (int j = 0; j < SB; ++j) {
            const int q = q0 + j * kIdxWaves;
            if (q < n) {
                const int32_t yy = me.live ? y[j] : -1;
                uint32_t v;
                carried(yy, v, q);
                seen |= yy >= 0 ? 1u : 0u;
                val0[q * kIdxRowW + lane] = v;
                site0[q * kIdxRowW + lane] = yy;
            }
        }
    }
    any_site[lane][wv] = uint8_t(seen);
    __syncthreads();

    // ---- search and output, patch by patch ----------------------------------
    // Patch p = (row block p / 8, line block (p + p / 8) % 8); lane l takes
    // row 8 rb + l / 8 of line 8 cb + l % 8.
    const int pr = lane >> 3;
    const float w = float(a.wall[ax]);
    const uint32_t rmask = (1u << a.rbits) - 1u;
    const int npatch = 8 * ((n + kIdxPatch - 1) / kIdxPatch);
    int32_t *slice0 = nullptr;
    for (int p = wv; p < npatch; p += kIdxWaves) {
        const int rbk = p >> 3;
        const int ln = kIdxPatch * ((p + rbk) & 7) + (lane & 7);
        const uint4 hv = *reinterpret_cast<const uint4 *>(&any_site[ln][0]);
        const bool has = (hv.x | hv.y | hv.z | hv.w) != 0u;
        const int qr = kIdxPatch * rbk + pr;
        const int q = min(qr, n - 1);
        const uint32_t *col = val0 + ln;
        int r_best = q;
        uint32_t kbest = col[q * kIdxRowW];
        float fbest = __builtin_bit_cast(float, kbest);
        if (!has) {                                   // nothing to find: stop at once
            kbest = 0;
            fbest = 0.0f;
        }
        int d0 = 1;
        if constexpr (SAMP) {
            // Unrolled blocks while every read of the patch stays in the tile
            // (guard rows included); the loop below takes over from d0.
            const int q_lo = kIdxPatch * rbk, q_hi = min(q_lo + kIdxPatch - 1, n - 1);
            const int room = min(q_lo + kIdxGuard, n - 1 + kIdxGuard - q_hi);
            int roff = 0;
            if (room >= 16) search_samp<0, 4>(col + (q - 16) * kIdxRowW, w, fbest, roff, d0);
            else if (room >= 12) search_samp<0, 3>(col + (q - 12) * kIdxRowW, w, fbest, roff, d0);
            else if (room >= 8) search_samp<0, 2>(col + (q - 8) * kIdxRowW, w, fbest, roff, d0);
            else if (room >= 4) search_samp<0, 1>(col + (q - 4) * kIdxRowW, w, fbest, roff, d0);
            r_best = q + roff;
        }
        for (int d = d0;; d += 4) {
            bool done;
            if (SAMP) done = w * float(d) * float(d) > fbest;
            else done = (uint64_t(uint32_t(d) * uint32_t(d)) << a.rbits) > uint64_t(kbest);
            if (__all(done) || d > n) break;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int dd = d + s;
                const int lo = max(q - dd, -kIdxGuard), hi = min(q + dd, n + kIdxGuard - 1);
                const uint32_t u = col[lo * kIdxRowW], v = col[hi * kIdxRowW];
                if (SAMP) {
                    const float add = w * float(dd) * float(dd);
                    const float cu = __builtin_bit_cast(float, u) + add;
                    const float cv = __builtin_bit_cast(float, v) + add;
                    if (cu < fbest) {
                        fbest = cu;
                        r_best = q - dd;
                    }
                    if (cv < fbest) {
                        fbest = cv;
                        r_best = q + dd;
                    }
                } else {
                    // keys of "no site" stay above every real key
                    const uint32_t add = uint32_t(dd * dd) << a.rbits;
                    const uint32_t cu = u == uint32_t(kInfI) ? u : u + add;
                    const uint32_t cv = v == uint32_t(kInfI) ? v : v + add;
                    kbest = min(kbest, min(cu, cv));
                }
            }
        }
        if (qr >= n) continue;
        // ---- output of element (row qr, line ln) ----------------------------
        const uint4 li = line_info[ln];
        if (!li.w) continue;
        Line l;
        l.s = li.x;
        l.base = li.y;
        l.i = li.z;
        slice0 = a.idx + uint64_t(l.s) * a.cstride;
        const uint64_t e = uint64_t(l.base) + uint64_t(qr) * a.inner;   // in-sample flat
        int32_t site = -1;
        if (has) {
            const int rw = SAMP ? r_best : int(kbest & rmask);
            site = site0[rw * kIdxRowW + ln];
        }
        if (!FINAL) {
            slice0[e] = site;
            continue;
        }
        // final pass: coordinates, distance, squared distance (with the
        // carrier in a distance output, the distance replaces the carried
        // site in place: this workgroup staged every row of its lines)
        double d2;
        if (site >= 0) {
            if (SAMP) d2 = double(fbest);
            else d2 = double(kbest >> a.rbits);
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
            d2 = virtual_sq<double>(qr, l.i, nd, a.shape, a.wall);
            if (!SAMP) d2 = double(virtual_sq<int64_t>(qr, l.i, nd, a.shape, a.wall));
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
    }
}

}  // namespace tmedt
